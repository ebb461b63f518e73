// Block-sparse decoder merge of SwiftNet-style segmentation networks (Section 4, the
// paper's semantic segmentation model): out = up2(coarse) (+ skip) (ReLU) on the
// executed output blocks, every other block of out untouched (feature transfer).
//
// up2 is bilinear upsampling by two with pixel centres aligned and edges replicated:
// output row y = 2i takes 3/4 of coarse row i and 1/4 of row i-1, row 2i+1 takes 3/4 of
// row i and 1/4 of row i+1 (a row outside the image is replaced by the edge row); the
// same for columns. An output block reads a one-pixel coarse halo, taken from the
// coarse buffer as it is (fresh where that block ran this frame, transferred else).
//
// Channels last (bf16/fp16, C % 8 == 0): one thread makes 8 channels of one output pixel
// from four 16-byte coarse loads and a skip load, all issued before any use, and one
// 16-byte store; arithmetic in fp32, one round to the storage format. Channels first
// (fp32): one thread per element.
#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 256;
constexpr int kBufferFlags = 0x00020000;     // raw buffer, dword format
constexpr int kOutOfRange = 0x7FFFFF00;      // loads return 0, stores are dropped

typedef int i32x4 __attribute__((ext_vector_type(4)));

template <bool BF16>
__device__ __forceinline__ float h16_to_f32(uint32_t h)
{
    if constexpr (BF16) return __uint_as_float(h << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// fp32 -> storage format, round to nearest even; NaN stays NaN.
template <bool BF16>
__device__ __forceinline__ uint32_t f32_to_h16(float z)
{
    if constexpr (BF16) {
        const uint32_t u = __float_as_uint(z);
        if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
        return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    } else {
        return __builtin_bit_cast(uint16_t, (_Float16)z);
    }
}

struct UpGeom {
    int hc, wc;        // coarse size (output is 2hc x 2wc)
    int gh, gw, bh, bw, total_blocks;
    int vpp;           // 16-byte vectors per pixel (C / 8)
    int relu;
};

// Two coarse indices and the weight of the second for output index o (coarse size n).
__device__ __forceinline__ void taps(int o, int n, int &i0, int &i1)
{
    const int i = o >> 1;
    i0 = i;
    i1 = (o & 1) ? min(i + 1, n - 1) : max(i - 1, 0);
}

template <bool BF16, bool SKIP>
__global__ __launch_bounds__(kThreads) void k_upsample_add_nhwc16(
    const uint4 *__restrict__ coarse, const uint4 *__restrict__ skip, uint4 *__restrict__ out,
    UpGeom g, int chunks, int coarse_bytes, int out_bytes, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ count)
{
    const int k = blockIdx.x / chunks;
    const int chunk = blockIdx.x - k * chunks;
    // the block id with the active count, one round trip (k < total_blocks: a valid read)
    const int bid = idx ? idx[k] : k;
    const int cnt = count ? *count : g.total_blocks;
    if (k >= cnt) return;
    const int img = bid / (g.gh * g.gw);
    const int rem = bid - img * g.gh * g.gw;
    const int gy = rem / g.gw, gx = rem - gy * g.gw;
    const int nv = g.bh * g.bw * g.vpp;
    const int v = chunk * kThreads + threadIdx.x;
    const int vv = min(v, nv - 1);                     // clamped: every load is in range
    const int pix = vv / g.vpp, cv = vv - pix * g.vpp;
    const int r = pix / g.bw, c = pix - r * g.bw;
    const int y = gy * g.bh + r, x = gx * g.bw + c;
    const int ho = 2 * g.hc, wo = 2 * g.wc;
    int y0, y1, x0, x1;
    taps(y, g.hc, y0, y1);
    taps(x, g.wc, x0, x1);
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)coarse, (short)0, coarse_bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void *)out, (short)0, out_bytes, kBufferFlags);
    auto coff = [&](int yy, int xx) { return ((((img * g.hc + yy) * g.wc + xx) * g.vpp) + cv) * 16; };
    const i32x4 a00 = __builtin_amdgcn_raw_buffer_load_b128(rc, coff(y0, x0), 0, 0);
    const i32x4 a01 = __builtin_amdgcn_raw_buffer_load_b128(rc, coff(y0, x1), 0, 0);
    const i32x4 a10 = __builtin_amdgcn_raw_buffer_load_b128(rc, coff(y1, x0), 0, 0);
    const i32x4 a11 = __builtin_amdgcn_raw_buffer_load_b128(rc, coff(y1, x1), 0, 0);
    const int ooff = v < nv ? ((((img * ho + y) * wo + x) * g.vpp) + cv) * 16 : kOutOfRange;
    i32x4 sk = {0, 0, 0, 0};                           // not read without a skip input
    if constexpr (SKIP) {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)skip, (short)0, out_bytes, kBufferFlags);
        sk = __builtin_amdgcn_raw_buffer_load_b128(rs, ooff, 0, 0);
    }
    i32x4 res;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        uint32_t o = 0;
#pragma unroll
        for (int hhalf = 0; hhalf < 2; ++hhalf) {
            const int sh = 16 * hhalf;
            const float p00 = h16_to_f32<BF16>(((uint32_t)a00[t] >> sh) & 0xFFFFu);
            const float p01 = h16_to_f32<BF16>(((uint32_t)a01[t] >> sh) & 0xFFFFu);
            const float p10 = h16_to_f32<BF16>(((uint32_t)a10[t] >> sh) & 0xFFFFu);
            const float p11 = h16_to_f32<BF16>(((uint32_t)a11[t] >> sh) & 0xFFFFu);
            const float top = 0.75f * p00 + 0.25f * p01;
            const float bot = 0.75f * p10 + 0.25f * p11;
            float z = 0.75f * top + 0.25f * bot;
            if constexpr (SKIP) z += h16_to_f32<BF16>(((uint32_t)sk[t] >> sh) & 0xFFFFu);
            if (g.relu) z = (z > 0.f || z != z) ? z : 0.f;
            o |= f32_to_h16<BF16>(z) << sh;
        }
        res[t] = (int)o;
    }
    __builtin_amdgcn_raw_buffer_store_b128(res, ro, ooff, 0, 0);
}

__global__ __launch_bounds__(kThreads) void k_upsample_add_nchw32(
    const float *__restrict__ coarse, const float *__restrict__ skip, float *__restrict__ out,
    UpGeom g, int c, const int32_t *__restrict__ idx, const int32_t *__restrict__ count)
{
    const int per_block = c * g.bh * g.bw;
    const int cnt = count ? *count : g.total_blocks;
    const int ho = 2 * g.hc, wo = 2 * g.wc;
    for (long long e = blockIdx.x * (long long)kThreads + threadIdx.x; e < (long long)cnt * per_block;
         e += (long long)gridDim.x * kThreads) {
        const int k = (int)(e / per_block);
        int rem = (int)(e - (long long)k * per_block);
        const int bid = idx ? idx[k] : k;
        const int img = bid / (g.gh * g.gw);
        const int r2 = bid - img * g.gh * g.gw;
        const int gy = r2 / g.gw, gx = r2 - gy * g.gw;
        const int xx = rem % g.bw;
        rem /= g.bw;
        const int yy = rem % g.bh;
        const int ch = rem / g.bh;
        const int y = gy * g.bh + yy, x = gx * g.bw + xx;
        int y0, y1, x0, x1;
        taps(y, g.hc, y0, y1);
        taps(x, g.wc, x0, x1);
        const float *cp = coarse + ((size_t)img * c + ch) * g.hc * g.wc;
        const float top = 0.75f * cp[y0 * g.wc + x0] + 0.25f * cp[y0 * g.wc + x1];
        const float bot = 0.75f * cp[y1 * g.wc + x0] + 0.25f * cp[y1 * g.wc + x1];
        const size_t o = (((size_t)img * c + ch) * ho + y) * wo + x;
        float z = 0.75f * top + 0.25f * bot;
        if (skip) z += skip[o];
        if (g.relu) z = (z > 0.f || z != z) ? z : 0.f;
        out[o] = z;
    }
}

}  // namespace

hipError_t launch_upsample_add(const void *coarse, const void *skip, void *out, int n, int c,
                               int hc, int wc, int esize, bool nhwc, bool bf16, int gh, int gw,
                               const int32_t *idx, const int32_t *count, int relu, hipStream_t s)
{
    UpGeom g;
    g.hc = hc; g.wc = wc; g.gh = gh; g.gw = gw;
    g.bh = 2 * hc / gh; g.bw = 2 * wc / gw;
    g.total_blocks = n * gh * gw;
    g.relu = relu;
    if (nhwc) {
        g.vpp = c * esize / 16;
        const int nv = g.bh * g.bw * g.vpp;
        const int chunks = (nv + kThreads - 1) / kThreads;
        const int cb = (int)((size_t)n * hc * wc * c * esize);
        const int ob = (int)((size_t)n * 4 * hc * wc * c * esize);
        const dim3 grid((unsigned)g.total_blocks * chunks), block(kThreads);
        auto go = [&](auto kern) {
            hipLaunchKernelGGL(kern, grid, block, 0, s, (const uint4 *)coarse, (const uint4 *)skip,
                               (uint4 *)out, g, chunks, cb, ob, idx, count);
        };
        if (bf16) {
            if (skip) go(k_upsample_add_nhwc16<true, true>);
            else go(k_upsample_add_nhwc16<true, false>);
        } else {
            if (skip) go(k_upsample_add_nhwc16<false, true>);
            else go(k_upsample_add_nhwc16<false, false>);
        }
    } else {
        const long long work = (long long)g.total_blocks * c * g.bh * g.bw;
        const long long want = (work + kThreads - 1) / kThreads;
        const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
        hipLaunchKernelGGL(k_upsample_add_nchw32, dim3(grid), dim3(kThreads), 0, s,
                           (const float *)coarse, (const float *)skip, (float *)out, g, c, idx, count);
    }
    return hipGetLastError();
}

}  // namespace bc
