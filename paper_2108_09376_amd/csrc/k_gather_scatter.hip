// Standalone halo gather and block scatter (Section 3.1: blocks padded from their
// neighbours; stored representations written back at executed blocks only).
//
// Both are pure HBM streams. With channels-last storage a tile row of the halo is
// one contiguous run of tw*C elements in the source and in the packed tile, and a
// block row of the destination is one contiguous run of bw*C elements, so whenever
// C*esize is a multiple of 16 the copies use 16-byte vectors, a fixed-size chunk of a
// tile per workgroup. Channels-first sources are transposed element by element (the
// fp32 correctness path). Workgroups beyond the device-side active count exit at
// once; destination elements outside active blocks are never touched.
#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 256;

struct RowGeom {
    int gh, gw, bh, bw, stride, pad, kh, kw;
    int h, w, c;             // source (gather) / destination (scatter) image
    int th, tw;              // tile rows/cols (gather: halo tile; scatter: block)
    int total_blocks;
};

__device__ __forceinline__ int active_count(const int32_t *count, int total)
{
    return count ? *count : total;
}

__device__ __forceinline__ void block_origin(const int32_t *idx, int k, const RowGeom &g,
                                             int &img, int &gy, int &gx)
{
    const int bid = idx ? idx[k] : k;
    img = bid / (g.gh * g.gw);
    const int rem = bid - img * g.gh * g.gw;
    gy = rem / g.gw;
    gx = rem - gy * g.gw;
}

// ---------------------------------------------------------------- channels last

// Channels last, 16-byte vectors: a packed tile is th*tw*vpp contiguous vectors, and a
// workgroup copies one chunk of kVecPerWG of them; each thread issues all of its loads
// before any store, so the whole chunk is in flight at once.
constexpr int kVecPerThread = 4;
constexpr int kVecPerWG = kThreads * kVecPerThread;

__global__ __launch_bounds__(kThreads) void k_gather_nhwc16(const uint4 *__restrict__ src,
                                                            uint4 *__restrict__ packed, RowGeom g,
                                                            int vpp, int chunks, uint4 padv,
                                                            const int32_t *__restrict__ idx,
                                                            const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / chunks;
    const int chunk = blockIdx.x - k * chunks;
    if (k >= active_count(count, g.total_blocks)) return;
    int img, gy, gx;
    block_origin(idx, k, g, img, gy, gx);
    const int rowv = g.tw * vpp;
    const int nv = g.th * rowv;
    const int x0 = gx * g.bw * g.stride - g.pad;
    const int y0 = gy * g.bh * g.stride - g.pad;
    uint4 *out = packed + (size_t)k * nv;
    // Every load reads a valid address (indices clamped into the image) and the padding
    // is selected afterwards: no load sits under a branch, so all of them are in flight
    // together instead of each waiting for the previous one.
    uint4 val[kVecPerThread];
    bool in_img[kVecPerThread];
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u) {
        const int v = min(chunk * kVecPerWG + u * kThreads + (int)threadIdx.x, nv - 1);
        const int r = v / rowv;
        const int t = v - r * rowv;
        const int tx = t / vpp;
        const int iy = y0 + r, ix = x0 + tx;
        in_img[u] = iy >= 0 && iy < g.h && ix >= 0 && ix < g.w;
        const int cy = min(max(iy, 0), g.h - 1), cx = min(max(ix, 0), g.w - 1);
        val[u] = src[(((size_t)img * g.h + cy) * g.w + cx) * vpp + (t - tx * vpp)];
    }
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u)
        if (!in_img[u]) val[u] = padv;
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u) {
        const int v = chunk * kVecPerWG + u * kThreads + threadIdx.x;
        if (v < nv) out[v] = val[u];
    }
}

// Raw buffer resource (no swizzle, dword format): stores at byte offsets at or beyond
// num_records are dropped, which lets the ragged end of a chunk store unconditionally.
constexpr int kBufferFlags = 0x00020000;
constexpr int kOutOfRange = 0x7FFFFF00;

__global__ __launch_bounds__(kThreads) void k_scatter_nhwc16(const uint4 *__restrict__ packed,
                                                             uint4 *__restrict__ dst, RowGeom g,
                                                             int vpp, int chunks,
                                                             const int32_t *__restrict__ idx,
                                                             const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / chunks;
    const int chunk = blockIdx.x - k * chunks;
    if (k >= active_count(count, g.total_blocks)) return;
    int img, gy, gx;
    block_origin(idx, k, g, img, gy, gx);
    const int rowv = g.bw * vpp;
    const int nv = g.bh * rowv;
    const int pitch = g.w * vpp;                 // vectors per destination image row
    const uint4 *in = packed + (size_t)k * nv;
    uint4 *out = dst + (((size_t)img * g.h + (size_t)gy * g.bh) * g.w + (size_t)gx * g.bw) * vpp;
    // The block's footprint in dst: bh rows of rowv vectors, pitch apart (below 2 GiB,
    // checked by the launcher).
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        (void *)out, (short)0, ((g.bh - 1) * pitch + rowv) * 16, kBufferFlags);
    uint4 val[kVecPerThread];
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u)     // clamped: unconditional loads, all in flight
        val[u] = in[min(chunk * kVecPerWG + u * kThreads + (int)threadIdx.x, nv - 1)];
#pragma unroll
    for (int u = 0; u < kVecPerThread; ++u) {
        const int v = chunk * kVecPerWG + u * kThreads + threadIdx.x;
        const int row = v / rowv;
        const int off = v < nv ? (row * pitch + (v - row * rowv)) * 16 : kOutOfRange;
        const uint4 x = val[u];
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(__attribute__((ext_vector_type(4))) int, x), r, off, 0, 0);
    }
}

// Element-wise channels-last fallback (C * esize not a multiple of 16): one tile row per
// workgroup.
template <typename V>
__global__ __launch_bounds__(kThreads) void k_gather_nhwc(const V *__restrict__ src,
                                                          V *__restrict__ packed, RowGeom g,
                                                          int vpp, V padv,
                                                          const int32_t *__restrict__ idx,
                                                          const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / g.th;
    const int ty = blockIdx.x - k * g.th;
    if (k >= active_count(count, g.total_blocks)) return;
    int img, gy, gx;
    block_origin(idx, k, g, img, gy, gx);
    const int iy = gy * g.bh * g.stride - g.pad + ty;
    const int x0 = gx * g.bw * g.stride - g.pad;
    const bool row_in = iy >= 0 && iy < g.h;
    V *out = packed + ((size_t)k * g.th + ty) * (size_t)g.tw * vpp;
    const V *in = src + ((size_t)img * g.h + (row_in ? iy : 0)) * (size_t)g.w * vpp;
    const int nv = g.tw * vpp;
    for (int v = threadIdx.x; v < nv; v += kThreads) {
        const int tx = v / vpp;
        const int ix = x0 + tx;
        V val = padv;
        if (row_in && ix >= 0 && ix < g.w) val = in[(size_t)ix * vpp + (v - tx * vpp)];
        out[v] = val;
    }
}

template <typename V>
__global__ __launch_bounds__(kThreads) void k_scatter_nhwc(const V *__restrict__ packed,
                                                           V *__restrict__ dst, RowGeom g,
                                                           int vpp,
                                                           const int32_t *__restrict__ idx,
                                                           const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / g.bh;
    const int py = blockIdx.x - k * g.bh;
    if (k >= active_count(count, g.total_blocks)) return;
    int img, gy, gx;
    block_origin(idx, k, g, img, gy, gx);
    const V *in = packed + ((size_t)k * g.bh + py) * (size_t)g.bw * vpp;
    V *out = dst + (((size_t)img * g.h + gy * g.bh + py) * g.w + (size_t)gx * g.bw) * vpp;
    const int nv = g.bw * vpp;
    for (int v = threadIdx.x; v < nv; v += kThreads) out[v] = in[v];
}

// ---------------------------------------------------------------- channels first

template <typename E>
__global__ __launch_bounds__(kThreads) void k_gather_nchw(const E *__restrict__ src,
                                                          E *__restrict__ packed, RowGeom g,
                                                          E padv,
                                                          const int32_t *__restrict__ idx,
                                                          const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / g.th;
    const int ty = blockIdx.x - k * g.th;
    if (k >= active_count(count, g.total_blocks)) return;
    int img, gy, gx;
    block_origin(idx, k, g, img, gy, gx);
    const int iy = gy * g.bh * g.stride - g.pad + ty;
    const int x0 = gx * g.bw * g.stride - g.pad;
    const bool row_in = iy >= 0 && iy < g.h;
    E *out = packed + ((size_t)k * g.th + ty) * (size_t)g.tw * g.c;
    const int ne = g.tw * g.c;
    for (int e = threadIdx.x; e < ne; e += kThreads) {
        const int tx = e / g.c;
        const int c = e - tx * g.c;
        const int ix = x0 + tx;
        E val = padv;
        if (row_in && ix >= 0 && ix < g.w)
            val = src[(((size_t)img * g.c + c) * g.h + iy) * (size_t)g.w + ix];
        out[e] = val;
    }
}

template <typename E>
__global__ __launch_bounds__(kThreads) void k_scatter_nchw(const E *__restrict__ packed,
                                                           E *__restrict__ dst, RowGeom g,
                                                           const int32_t *__restrict__ idx,
                                                           const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / g.bh;
    const int py = blockIdx.x - k * g.bh;
    if (k >= active_count(count, g.total_blocks)) return;
    int img, gy, gx;
    block_origin(idx, k, g, img, gy, gx);
    const E *in = packed + ((size_t)k * g.bh + py) * (size_t)g.bw * g.c;
    const int oy = gy * g.bh + py;
    const int ne = g.bw * g.c;
    for (int e = threadIdx.x; e < ne; e += kThreads) {
        const int c = e / g.bw;
        const int px = e - c * g.bw;
        dst[(((size_t)img * g.c + c) * g.h + oy) * (size_t)g.w + gx * g.bw + px] =
            in[(size_t)px * g.c + c];
    }
}

RowGeom row_geom(const LayerGeom &L, bool gather)
{
    RowGeom g;
    g.gh = L.gh; g.gw = L.gw; g.bh = L.bh; g.bw = L.bw;
    g.stride = L.stride; g.pad = L.pad; g.kh = L.kh; g.kw = L.kw;
    g.total_blocks = L.total_blocks;
    if (gather) {
        g.h = L.hin; g.w = L.win; g.c = L.cin;
        g.th = (L.bh - 1) * L.stride + L.kh;
        g.tw = (L.bw - 1) * L.stride + L.kw;
    } else {
        g.h = L.hout; g.w = L.wout; g.c = L.cout;
        g.th = L.bh; g.tw = L.bw;
    }
    return g;
}

}  // namespace

hipError_t launch_gather_halo(const void *src, int esize, bool nhwc, const LayerGeom &L,
                              uint32_t pad_bits, void *packed, hipStream_t s)
{
    const RowGeom g = row_geom(L, true);
    const dim3 grid((unsigned)L.total_blocks * g.th), block(kThreads);
    if (nhwc && (g.c * esize) % 16 == 0) {
        const uint32_t p = esize == 2 ? (pad_bits & 0xFFFFu) * 0x10001u : pad_bits;
        const uint4 padv = make_uint4(p, p, p, p);
        const int vpp = g.c * esize / 16;
        const int chunks = (g.th * g.tw * vpp + kVecPerWG - 1) / kVecPerWG;
        hipLaunchKernelGGL(k_gather_nhwc16, dim3((unsigned)L.total_blocks * chunks), block, 0, s,
                           (const uint4 *)src, (uint4 *)packed, g, vpp, chunks, padv, L.idx,
                           L.count);
    } else if (nhwc && esize == 2) {
        hipLaunchKernelGGL(k_gather_nhwc<uint16_t>, grid, block, 0, s, (const uint16_t *)src,
                           (uint16_t *)packed, g, g.c, (uint16_t)pad_bits, L.idx, L.count);
    } else if (nhwc) {
        hipLaunchKernelGGL(k_gather_nhwc<uint32_t>, grid, block, 0, s, (const uint32_t *)src,
                           (uint32_t *)packed, g, g.c, pad_bits, L.idx, L.count);
    } else if (esize == 2) {
        hipLaunchKernelGGL(k_gather_nchw<uint16_t>, grid, block, 0, s, (const uint16_t *)src,
                           (uint16_t *)packed, g, (uint16_t)pad_bits, L.idx, L.count);
    } else {
        hipLaunchKernelGGL(k_gather_nchw<uint32_t>, grid, block, 0, s, (const uint32_t *)src,
                           (uint32_t *)packed, g, pad_bits, L.idx, L.count);
    }
    return hipGetLastError();
}

hipError_t launch_scatter_blocks(const void *packed, int esize, bool nhwc, const LayerGeom &L,
                                 void *dst, hipStream_t s)
{
    const RowGeom g = row_geom(L, false);
    const dim3 grid((unsigned)L.total_blocks * g.bh), block(kThreads);
    const int64_t span = nhwc ? ((int64_t)(g.bh - 1) * g.w + g.bw) * g.c * esize : 0;
    if (nhwc && (g.c * esize) % 16 == 0 && span < kOutOfRange) {
        const int vpp = g.c * esize / 16;
        const int chunks = (g.bh * g.bw * vpp + kVecPerWG - 1) / kVecPerWG;
        hipLaunchKernelGGL(k_scatter_nhwc16, dim3((unsigned)L.total_blocks * chunks), block, 0, s,
                           (const uint4 *)packed, (uint4 *)dst, g, vpp, chunks, L.idx, L.count);
    } else if (nhwc && esize == 2) {
        hipLaunchKernelGGL(k_scatter_nhwc<uint16_t>, grid, block, 0, s, (const uint16_t *)packed,
                           (uint16_t *)dst, g, g.c, L.idx, L.count);
    } else if (nhwc) {
        hipLaunchKernelGGL(k_scatter_nhwc<uint32_t>, grid, block, 0, s, (const uint32_t *)packed,
                           (uint32_t *)dst, g, g.c, L.idx, L.count);
    } else if (esize == 2) {
        hipLaunchKernelGGL(k_scatter_nchw<uint16_t>, grid, block, 0, s, (const uint16_t *)packed,
                           (uint16_t *)dst, g, L.idx, L.count);
    } else {
        hipLaunchKernelGGL(k_scatter_nchw<uint32_t>, grid, block, 0, s, (const uint32_t *)packed,
                           (uint32_t *)dst, g, L.idx, L.count);
    }
    return hipGetLastError();
}

}  // namespace bc
