// Spatial pyramid pooling of the segmentation network's stride-32 feature, block-sparse
// (the context module of SwiftNet-style models; every layer of such single-stage
// networks runs block-sparsely, Section 4). Channels last, bf16 / fp16.
//
// A pyramid level averages the whole map over a grid of bins, so each level depends
// on every block of the input buffer. Following the method's definition (a layer's
// result equals the dense layer on its current input buffer, selected into the
// previous output at the executed blocks, Section 3.1), each call
//  1. computes every level densely from the whole input buffer (fresh where blocks
//     ran this frame, transferred elsewhere): per bin the mean of its pixels, a 1x1
//     convolution (weights [level][cl][c]) plus bias, ReLU, one round to the storage
//     format, written to the caller's level buffer [n][bins][cl] (k_spp_levels16,
//     one 1024-thread workgroup per bin; about 0.5 MB read at 2048x1024);
//  2. writes the executed output blocks of the concatenation [input, up(level 0),
//     ..., up(level L-1)]: the input's own bits, then each level resampled bilinearly
//     to the map (pixel centres aligned) and rounded (k_spp_concat16, one thread per
//     16 bytes of output; blocks that did not run are neither read nor written).
// Sums are taken in a fixed order (no atomics), so results do not depend on the
// schedule.
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

// Bin (i, j) of a rows x cols grid on an h x w map covers rows floor(i h / rows) ..
// ceil((i + 1) h / rows) - 1, and the same for columns.
__device__ __forceinline__ void bin_range(int i, int rows, int h, int &lo, int &hi)
{
    lo = (i * h) / rows;
    hi = ((i + 1) * h + rows - 1) / rows;
}

// One workgroup of kLvThreads threads per bin: (kLvThreads / vpp) pixel lanes x vpp
// channel vectors of 8 (vpp = c / 8 divides 256, so it divides kLvThreads; checked on
// the host). A thread keeps kSppBatch loads in flight (offsets past the bin read zero)
// and adds them in pixel order; the pixel lanes are then added pairwise in a fixed
// tree. The 1x1 convolution splits each output channel's dot product over
// kLvThreads / cl threads (channel ranges in order), their partial sums added in range
// order: every sum has a fixed order, so results do not depend on the schedule.
constexpr int kLvThreads = 1024;
constexpr int kSppBatch = 8;

template <bool BF16>
__global__ __launch_bounds__(kLvThreads) void k_spp_levels16(const uint16_t *__restrict__ in,
                                                              const uint16_t *__restrict__ w,
                                                              const float *__restrict__ bias,
                                                              uint16_t *__restrict__ levels,
                                                              SppGeom g)
{
    __shared__ float part[kLvThreads][8];
    __shared__ float mean[kMaxSppChannels];
    const int tid = threadIdx.x;
    const int tb = g.first[g.levels];
    const int img = blockIdx.x / tb, bin = blockIdx.x - img * tb;
    int l = 0;
    while (l + 1 < g.levels && bin >= g.first[l + 1]) ++l;
    const int local = bin - g.first[l];
    const int bi = local / g.cols[l], bj = local - bi * g.cols[l];
    int r0, r1, c0, c1;
    bin_range(bi, g.rows[l], g.h, r0, r1);
    bin_range(bj, g.cols[l], g.w, c0, c1);
    const int bw = c1 - c0, npix = (r1 - r0) * bw;
    const int lanes = kLvThreads / g.vpp;
    const int lane = tid / g.vpp, v = tid - lane * g.vpp;
    const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
        (void *)in, (short)0, g.in_bytes, kBufferFlags);
    // the convolution's first batch of weights is requested with the pixels (it does not
    // depend on them)
    const int Q = kLvThreads / g.cl;
    const int co = tid % g.cl, q = tid / g.cl;
    const int v0 = q < Q ? (q * g.vpp) / Q : 0, v1 = q < Q ? ((q + 1) * g.vpp) / Q : 0;
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void *)w, (short)0, g.w_bytes, kBufferFlags);
    const int row = (l * g.cl + co) * g.c * 2;           // bytes of weight row (l, co)
    i32x4 wv[kSppBatch];
    auto load_w = [&](int cv0, i32x4 (&r)[kSppBatch]) {
#pragma unroll
        for (int u = 0; u < kSppBatch; ++u)
            r[u] = __builtin_amdgcn_raw_buffer_load_b128(
                rw, cv0 + u < v1 ? row + (cv0 + u) * 16 : kOutOfRange, 0, 0);
    };
    load_w(v0, wv);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int p0 = lane; p0 < npix; p0 += kSppBatch * lanes) {
        i32x4 d[kSppBatch];
#pragma unroll
        for (int u = 0; u < kSppBatch; ++u) {
            const int p = p0 + u * lanes;
            const int y = r0 + p / bw, x = c0 + (p - (p / bw) * bw);
            d[u] = __builtin_amdgcn_raw_buffer_load_b128(
                rin, p < npix ? ((((img * g.h + y) * g.w + x) * g.vpp) + v) * 16 : kOutOfRange, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < kSppBatch; ++u)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                acc[2 * t] += h16_to_f32<BF16>((uint32_t)d[u][t] & 0xFFFFu);
                acc[2 * t + 1] += h16_to_f32<BF16>((uint32_t)d[u][t] >> 16);
            }
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) part[tid][t] = acc[t];
    __syncthreads();
    // pixel lanes pairwise: lane i takes lane i + half, halves shrinking (lanes is a
    // power of two: kLvThreads and vpp are)
    for (int half = lanes / 2; half >= 1; half /= 2) {
        if (lane < half) {
#pragma unroll
            for (int t = 0; t < 8; ++t) part[tid][t] += part[tid + half * g.vpp][t];
        }
        __syncthreads();
    }
    if (tid < g.vpp) {
#pragma unroll
        for (int t = 0; t < 8; ++t) mean[tid * 8 + t] = part[tid][t] / (float)npix;
    }
    __syncthreads();
    // 1x1 convolution: thread t = q * cl + co takes channel vectors [q vpp / Q, (q+1) vpp / Q)
    // of output channel co (Q = kLvThreads / cl parts)
    float z = 0.f;
    if (q < Q) {
        for (int cv0 = v0; cv0 < v1; cv0 += kSppBatch) {
            if (cv0 > v0) load_w(cv0, wv);               // the first batch came in with the pixels
#pragma unroll
            for (int u = 0; u < kSppBatch; ++u) {
                if (cv0 + u >= v1) break;
                const int cb = (cv0 + u) * 8;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    z += h16_to_f32<BF16>((uint32_t)wv[u][t] & 0xFFFFu) * mean[cb + 2 * t];
                    z += h16_to_f32<BF16>((uint32_t)wv[u][t] >> 16) * mean[cb + 2 * t + 1];
                }
            }
        }
    }
    part[tid][1] = z;                                    // column 1: free since the tree
    __syncthreads();
    if (tid < g.cl) {
        float zz = bias ? bias[l * g.cl + tid] : 0.f;
        for (int qq = 0; qq < Q; ++qq) zz += part[qq * g.cl + tid][1];   // parts in order
        zz = (zz > 0.f || zz != zz) ? zz : 0.f;
        levels[((size_t)img * tb + bin) * g.cl + tid] = (uint16_t)f32_to_h16<BF16>(zz);
    }
}

// Source row of output row y when a map of n_in rows is resampled to n_out rows with
// pixel centres aligned: s = ((2y + 1) n_in - n_out) / (2 n_out), 0 if negative; the
// numerator is exact in integers, so s is one rounding of the exact value.
__device__ __forceinline__ void src_coord(int y, int n_in, int n_out, int &i0, int &i1, float &f)
{
    const int num = (2 * y + 1) * n_in - n_out;
    float s = num <= 0 ? 0.f : (float)num / (float)(2 * n_out);
    i0 = min((int)s, n_in - 1);
    i1 = min(i0 + 1, n_in - 1);
    f = s - (float)i0;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_spp_concat16(const uint16_t *__restrict__ in,
                                                            const uint16_t *__restrict__ levels,
                                                            uint16_t *__restrict__ out, SppGeom g,
                                                            int chunks, const int32_t *__restrict__ idx,
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
    const int ovp = g.cout / 8;                          // output vectors per pixel
    const int nv = g.bh * g.bw * ovp;
    const int vi = chunk * kThreads + threadIdx.x;
    const int vv = min(vi, nv - 1);                      // clamped: every load is in range
    const int pix = vv / ovp, ov = vv - pix * ovp;
    const int r = pix / g.bw, c = pix - r * g.bw;
    const int y = gy * g.bh + r, x = gx * g.bw + c;
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void *)out, (short)0, g.out_bytes, kBufferFlags);
    const int ooff = vi < nv ? (((img * g.h + y) * g.w + x) * ovp + ov) * 16 : kOutOfRange;
    i32x4 res;
    if (ov < g.vpp) {                                    // the input's own channels
        const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
            (void *)in, (short)0, g.in_bytes, kBufferFlags);
        res = __builtin_amdgcn_raw_buffer_load_b128(rin, (((img * g.h + y) * g.w + x) * g.vpp + ov) * 16, 0, 0);
    } else {
        const int lv = ov - g.vpp, lvp = g.cl / 8;
        const int l = lv / lvp, cv = lv - l * lvp;
        int y0, y1, x0, x1;
        float fy, fx;
        src_coord(y, g.rows[l], g.h, y0, y1, fy);
        src_coord(x, g.cols[l], g.w, x0, x1, fx);
        const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
            (void *)levels, (short)0, g.lv_bytes, kBufferFlags);
        const int base = img * g.first[g.levels] + g.first[l];
        auto loff = [&](int yy, int xx) { return ((base + yy * g.cols[l] + xx) * g.cl + cv * 8) * 2; };
        const i32x4 a00 = __builtin_amdgcn_raw_buffer_load_b128(rl, loff(y0, x0), 0, 0);
        const i32x4 a10 = __builtin_amdgcn_raw_buffer_load_b128(rl, loff(y1, x0), 0, 0);
        const i32x4 a01 = __builtin_amdgcn_raw_buffer_load_b128(rl, loff(y0, x1), 0, 0);
        const i32x4 a11 = __builtin_amdgcn_raw_buffer_load_b128(rl, loff(y1, x1), 0, 0);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            uint32_t o = 0;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int sh = 16 * hh;
                const float p00 = h16_to_f32<BF16>(((uint32_t)a00[t] >> sh) & 0xFFFFu);
                const float p10 = h16_to_f32<BF16>(((uint32_t)a10[t] >> sh) & 0xFFFFu);
                const float p01 = h16_to_f32<BF16>(((uint32_t)a01[t] >> sh) & 0xFFFFu);
                const float p11 = h16_to_f32<BF16>(((uint32_t)a11[t] >> sh) & 0xFFFFu);
                // rows first, then columns
                const float t0 = (1.f - fy) * p00 + fy * p10;
                const float t1 = (1.f - fy) * p01 + fy * p11;
                o |= f32_to_h16<BF16>((1.f - fx) * t0 + fx * t1) << sh;
            }
            res[t] = (int)o;
        }
    }
    __builtin_amdgcn_raw_buffer_store_b128(res, ro, ooff, 0, 0);
}

}  // namespace

hipError_t launch_spp(const uint16_t *in, const uint16_t *w, const float *bias, uint16_t *levels,
                      uint16_t *out, const SppGeom &g, bool bf16, const int32_t *idx,
                      const int32_t *count, hipStream_t s)
{
    const unsigned bins = (unsigned)g.n * g.first[g.levels];
    if (bf16)
        hipLaunchKernelGGL(k_spp_levels16<true>, dim3(bins), dim3(kLvThreads), 0, s, in, w, bias, levels, g);
    else
        hipLaunchKernelGGL(k_spp_levels16<false>, dim3(bins), dim3(kLvThreads), 0, s, in, w, bias, levels, g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int nv = g.bh * g.bw * (g.cout / 8);
    const int chunks = (nv + kThreads - 1) / kThreads;
    const dim3 grid((unsigned)g.total_blocks * chunks);
    if (bf16)
        hipLaunchKernelGGL(k_spp_concat16<true>, grid, dim3(kThreads), 0, s, in, levels, out, g, chunks, idx, count);
    else
        hipLaunchKernelGGL(k_spp_concat16<false>, grid, dim3(kThreads), 0, s, in, levels, out, g, chunks, idx, count);
    return hipGetLastError();
}

}  // namespace bc
