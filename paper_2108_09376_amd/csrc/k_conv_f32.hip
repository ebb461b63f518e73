// Block-sparse convolution, channels-first fp32 (the small-channel correctness path).
//
// One workgroup computes one active output block for a tile of output channels.
// For each chunk of input channels it stages the block's halo tile
// [ci][(bh-1)*s + kh][(bw-1)*s + kw] (zeros outside the image) and the matching
// weights in LDS, then every thread accumulates a few (pixel, output channel)
// sums with fp32 FMAs in the fixed order ci -> i -> j. The epilogue adds bias and
// residual in fp32, applies ReLU and writes straight to the block's position of
// the persistent output; elements outside active blocks are never touched.
#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxPerThread = 8;
constexpr int kLdsBudget = 48 * 1024;

struct F32Args {
    const float *x, *w, *bias, *res;
    float *y;
    LayerGeom g;
    int th, tw, co_t, ci_t, n_co_tiles;
    int relu;
};

__global__ __launch_bounds__(kThreads) void k_conv_nchw_f32(F32Args a)
{
    extern __shared__ float lds[];
    const LayerGeom &g = a.g;
    const int k = blockIdx.x / a.n_co_tiles;
    const int cot = blockIdx.x - k * a.n_co_tiles;
    const int cnt = g.count ? *g.count : g.total_blocks;
    if (k >= cnt) return;
    const int bid = g.idx ? g.idx[k] : k;
    const int img = bid / (g.gh * g.gw);
    const int rem = bid - img * g.gh * g.gw;
    const int gy = rem / g.gw, gx = rem - (rem / g.gw) * g.gw;
    const int npx = g.bh * g.bw;
    const int co0 = cot * a.co_t;
    const int co_n = min(a.co_t, g.cout - co0);
    const int taps = g.kh * g.kw;
    const int y0 = gy * g.bh * g.stride - g.pad, x0 = gx * g.bw * g.stride - g.pad;
    const int tile = a.th * a.tw;
    float *xs = lds;                          // [ci_t][th][tw]
    float *ws = lds + (size_t)a.ci_t * tile;  // [co_t][ci_t][taps]

    float acc[kMaxPerThread];
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) acc[u] = 0.f;

    for (int c0 = 0; c0 < g.cin; c0 += a.ci_t) {
        const int cn = min(a.ci_t, g.cin - c0);
        __syncthreads();
        for (int e = threadIdx.x; e < cn * tile; e += kThreads) {
            const int ci = e / tile;
            const int r = e - ci * tile;
            const int ty = r / a.tw, tx = r - (r / a.tw) * a.tw;
            const int iy = y0 + ty, ix = x0 + tx;
            float v = 0.f;
            if (iy >= 0 && iy < g.hin && ix >= 0 && ix < g.win)
                v = a.x[(((size_t)img * g.cin + c0 + ci) * g.hin + iy) * (size_t)g.win + ix];
            xs[e] = v;
        }
        for (int e = threadIdx.x; e < co_n * cn * taps; e += kThreads) {
            const int co = e / (cn * taps);
            const int r = e - co * cn * taps;
            const int ci = r / taps, t = r - (r / taps) * taps;
            ws[((size_t)co * a.ci_t + ci) * taps + t] =
                a.w[(((size_t)(co0 + co) * g.cin) + c0 + ci) * taps + t];
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kMaxPerThread; ++u) {
            const int pair = threadIdx.x + u * kThreads;
            if (pair >= npx * co_n) break;
            const int co = pair / npx, p = pair - (pair / npx) * npx;
            const int py = p / g.bw, px = p - (p / g.bw) * g.bw;
            float s = acc[u];
            for (int ci = 0; ci < cn; ++ci) {
                const float *xr = xs + (size_t)ci * tile + (py * g.stride) * a.tw + px * g.stride;
                const float *wr = ws + ((size_t)co * a.ci_t + ci) * taps;
                for (int i = 0; i < g.kh; ++i)
                    for (int j = 0; j < g.kw; ++j) s = fmaf(wr[i * g.kw + j], xr[i * a.tw + j], s);
            }
            acc[u] = s;
        }
    }
#pragma unroll
    for (int u = 0; u < kMaxPerThread; ++u) {
        const int pair = threadIdx.x + u * kThreads;
        if (pair >= npx * co_n) break;
        const int co = pair / npx, p = pair - (pair / npx) * npx;
        const int py = p / g.bw, px = p - (p / g.bw) * g.bw;
        const size_t o = (((size_t)img * g.cout + co0 + co) * g.hout + gy * g.bh + py) * g.wout +
                         gx * g.bw + px;
        float z = acc[u];
        if (a.bias) z += a.bias[co0 + co];
        if (a.res) z += a.res[o];
        if (a.relu) z = (z > 0.f || z != z) ? z : 0.f;
        a.y[o] = z;
    }
}

}  // namespace

hipError_t launch_conv_nchw_f32(const float *x, const float *w, const float *bias,
                                const float *res, float *y, int relu, const LayerGeom &g,
                                hipStream_t s, const char **why)
{
    F32Args a;
    a.x = x; a.w = w; a.bias = bias; a.res = res; a.y = y; a.g = g; a.relu = relu;
    a.th = (g.bh - 1) * g.stride + g.kh;
    a.tw = (g.bw - 1) * g.stride + g.kw;
    const int npx = g.bh * g.bw;
    a.co_t = g.cout < (kThreads * kMaxPerThread) / npx ? g.cout : (kThreads * kMaxPerThread) / npx;
    if (a.co_t < 1) {
        *why = "fp32 path: output block larger than 2048 pixels";
        return hipErrorInvalidValue;
    }
    const int per_ci = (a.th * a.tw + a.co_t * g.kh * g.kw) * (int)sizeof(float);
    a.ci_t = kLdsBudget / per_ci;
    if (a.ci_t < 1) {
        *why = "fp32 path: one channel of the halo tile does not fit in LDS";
        return hipErrorInvalidValue;
    }
    if (a.ci_t > g.cin) a.ci_t = g.cin;
    a.n_co_tiles = (g.cout + a.co_t - 1) / a.co_t;
    const size_t lds = (size_t)a.ci_t * per_ci;
    hipLaunchKernelGGL(k_conv_nchw_f32, dim3((unsigned)g.total_blocks * a.n_co_tiles),
                       dim3(kThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace bc
