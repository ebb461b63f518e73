// Block-sparse max pooling (the stem pooling of a ResNet backbone, run on active
// blocks like every other layer, Section 4). Padding is -inf: padded positions
// never win. Channels-last 16-bit storage: one thread produces 8 channels of one
// output pixel with 16-byte loads and stores; the max of stored values is itself
// a stored value, so no rounding happens.
#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float h16_to_f32(uint16_t v, bool bf16)
{
    if (bf16) return __uint_as_float((uint32_t)v << 16);
    return (float)__builtin_bit_cast(_Float16, v);
}

__device__ __forceinline__ void block_of(const LayerGeom &g, int k, int &img, int &gy, int &gx)
{
    const int bid = g.idx ? g.idx[k] : k;
    img = bid / (g.gh * g.gw);
    const int rem = bid - img * g.gh * g.gw;
    gy = rem / g.gw;
    gx = rem - gy * g.gw;
}

// grid.x = total_blocks * parts; each workgroup covers kThreads (pixel, 8-channel) pairs.
// KS > 0: a KS x KS window known at compile time; every tap's load is issued before any
// is used (coordinates clamped into the image, so every address is valid, and taps
// outside the image replaced by -inf afterwards), one memory round trip per thread.
// KS = 0: any window, taps in a loop.
template <int KS>
__global__ __launch_bounds__(kThreads) void k_maxpool_nhwc16(const uint16_t *__restrict__ x,
                                                             uint16_t *__restrict__ y,
                                                             LayerGeom g, int parts, int bf16)
{
    const int k = blockIdx.x / parts;
    const int part = blockIdx.x - k * parts;
    // the block id is read with the active count, in one round trip (the index holds
    // total_blocks entries, so the read is valid whether or not block k is active)
    const int bid = g.idx ? g.idx[k] : k;
    const int cnt = g.count ? *g.count : g.total_blocks;
    if (k >= cnt) return;
    const int cv = g.cout / 8;
    const int e = part * kThreads + threadIdx.x;
    if (e >= g.bh * g.bw * cv) return;
    const int img = bid / (g.gh * g.gw);
    const int rem = bid - img * g.gh * g.gw;
    const int gy = rem / g.gw, gx = rem - gy * g.gw;
    const int p = e / cv, c8 = e - p * cv;
    const int py = p / g.bw, px = p - py * g.bw;
    const int oy = gy * g.bh + py, ox = gx * g.bw + px;
    float m[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) m[q] = -__builtin_huge_valf();
    auto take = [&](const uint4 v) {
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            m[2 * q] = fmaxf(m[2 * q], h16_to_f32((uint16_t)(w4[q] & 0xFFFFu), bf16));
            m[2 * q + 1] = fmaxf(m[2 * q + 1], h16_to_f32((uint16_t)(w4[q] >> 16), bf16));
        }
    };
    const uint16_t *xi = x + (size_t)img * g.hin * g.win * g.cin + c8 * 8;
    if constexpr (KS > 0) {
        uint4 v[KS * KS];
        bool in[KS * KS];
#pragma unroll
        for (int i = 0; i < KS; ++i)
#pragma unroll
            for (int j = 0; j < KS; ++j) {
                const int iy = oy * g.stride - g.pad + i, ix = ox * g.stride - g.pad + j;
                in[i * KS + j] = iy >= 0 && iy < g.hin && ix >= 0 && ix < g.win;
                const int cy = min(max(iy, 0), g.hin - 1), cx = min(max(ix, 0), g.win - 1);
                v[i * KS + j] = *(const uint4 *)(xi + ((size_t)cy * g.win + cx) * g.cin);
            }
#pragma unroll
        for (int t = 0; t < KS * KS; ++t)
            if (in[t]) take(v[t]);
    } else {
        for (int i = 0; i < g.kh; ++i) {
            const int iy = oy * g.stride - g.pad + i;
            if (iy < 0 || iy >= g.hin) continue;
            for (int j = 0; j < g.kw; ++j) {
                const int ix = ox * g.stride - g.pad + j;
                if (ix < 0 || ix >= g.win) continue;
                take(*(const uint4 *)(xi + ((size_t)iy * g.win + ix) * g.cin));
            }
        }
    }
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t lo, hi;
        if (bf16) {
            lo = __float_as_uint(m[2 * q]) >> 16;      // exact: m holds a bf16 value
            hi = __float_as_uint(m[2 * q + 1]) >> 16;
        } else {
            lo = __builtin_bit_cast(uint16_t, (_Float16)m[2 * q]);
            hi = __builtin_bit_cast(uint16_t, (_Float16)m[2 * q + 1]);
        }
        o[q] = lo | (hi << 16);
    }
    *(uint4 *)(y + (((size_t)img * g.hout + oy) * g.wout + ox) * g.cout + c8 * 8) =
        make_uint4(o[0], o[1], o[2], o[3]);
}

__global__ __launch_bounds__(kThreads) void k_maxpool_nchw32(const float *__restrict__ x,
                                                             float *__restrict__ y, LayerGeom g,
                                                             int parts)
{
    const int k = blockIdx.x / parts;
    const int part = blockIdx.x - k * parts;
    const int cnt = g.count ? *g.count : g.total_blocks;
    if (k >= cnt) return;
    const int e = part * kThreads + threadIdx.x;
    if (e >= g.bh * g.bw * g.cout) return;
    int img, gy, gx;
    block_of(g, k, img, gy, gx);
    const int c = e / (g.bh * g.bw);
    const int p = e - c * g.bh * g.bw;
    const int py = p / g.bw, px = p - py * g.bw;
    const int oy = gy * g.bh + py, ox = gx * g.bw + px;
    float m = -__builtin_huge_valf();
    const float *xc = x + ((size_t)img * g.cin + c) * g.hin * (size_t)g.win;
    for (int i = 0; i < g.kh; ++i) {
        const int iy = oy * g.stride - g.pad + i;
        if (iy < 0 || iy >= g.hin) continue;
        for (int j = 0; j < g.kw; ++j) {
            const int ix = ox * g.stride - g.pad + j;
            if (ix < 0 || ix >= g.win) continue;
            m = fmaxf(m, xc[(size_t)iy * g.win + ix]);
        }
    }
    y[(((size_t)img * g.cout + c) * g.hout + oy) * g.wout + ox] = m;
}

}  // namespace

hipError_t launch_maxpool_nhwc16(const uint16_t *x, uint16_t *y, Half16 fmt, const LayerGeom &g,
                                 hipStream_t s)
{
    const int work = g.bh * g.bw * (g.cout / 8);
    const int parts = (work + kThreads - 1) / kThreads;
    const dim3 grid((unsigned)g.total_blocks * parts);
    const int bf = fmt == Half16::BF16 ? 1 : 0;
    if (g.kh == 3 && g.kw == 3)
        hipLaunchKernelGGL(k_maxpool_nhwc16<3>, grid, dim3(kThreads), 0, s, x, y, g, parts, bf);
    else
        hipLaunchKernelGGL(k_maxpool_nhwc16<0>, grid, dim3(kThreads), 0, s, x, y, g, parts, bf);
    return hipGetLastError();
}

hipError_t launch_maxpool_nchw32(const float *x, float *y, const LayerGeom &g, hipStream_t s)
{
    const int work = g.bh * g.bw * g.cout;
    const int parts = (work + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(k_maxpool_nchw32, dim3((unsigned)g.total_blocks * parts), dim3(kThreads), 0,
                       s, x, y, g, parts);
    return hipGetLastError();
}

}  // namespace bc
