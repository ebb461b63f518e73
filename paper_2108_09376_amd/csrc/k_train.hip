// The policy network's online update (Section 4 configuration: RMSprop every 4 frames
// on the REINFORCE loss of Section 3.5). Channels-last 16-bit activations and
// gradients, fp32 weight gradients and optimiser state.
//
//  * logit gradient: dL/dz_b = -R_b (a_b - p_b), written to channel 0 of the head's
//    [n][gh][gw][c] gradient map (other channels 0);
//  * gradient combine: out = (a + b) * [y > 0]: the ReLU's backward pass (b absent),
//    a residual's gradient added to another (y absent), or both;
//  * input gradient of a convolution (the transposed convolution) runs on the forward
//    matrix-core conv: weights flipped and transposed ([cout][kh][kw][cin] ->
//    [cin][kh][kw][cout], taps reversed), and for stride 2 the output gradient spread
//    onto the even pixels of a map of the input's size (zeros between), then a
//    stride-1 convolution with padding k/2 (these two kernels are here);
//  * weight gradient: dW[co][i][j][ci] += sum_p G[p][co] X[p*s - pad + (i, j)][ci], an
//    implicit GEMM whose reduction runs over pixels. A workgroup owns a 64 x 64
//    (co, ci) tile of one tap and a range of 1024 pixels; per 128-pixel chunk it loads
//    G and the tap-shifted X rows with 16-byte requests (eight channels of one pixel),
//    transposes them in registers and stores them in LDS as [channel][pixel], so that
//    matrix-core fragments (eight consecutive pixels of one channel per lane) are
//    contiguous 16-byte LDS reads; the next two chunks' loads are in flight during the
//    current chunk's 16 MFMAs per wave (registers plus an LDS double buffer); the tile
//    is added to dW with fp32 atomics at the end (the order of those additions varies
//    between runs);
//  * bias gradient: db[co] += sum_p G[p][co], summed from the same G registers by the
//    workgroups of tap 0 (and the first ci tile), reduced across lanes, one atomic per
//    channel and workgroup;
//  * RMSprop (PyTorch's definition, no momentum): g' = g + wd w; v = alpha v +
//    (1 - alpha) g'^2; w -= lr g' / (sqrt(v) + eps); the gradient is reset to 0 and the
//    16-bit copy of w rewritten (round to nearest even); for one tensor, or for up to
//    kMaxParams tensors in one launch (their pointers and sizes in the kernel arguments).
#include <mutex>
#include <type_traits>

#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 256;
constexpr int kBufferFlags = 0x00020000;     // raw buffer, dword format
constexpr int kOutOfRange = 0x7FFFFF00;      // loads return 0, stores are dropped

typedef short short8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

template <bool BF16>
__device__ __forceinline__ float h16_to_f32(uint32_t h)
{
    if constexpr (BF16) return __uint_as_float(h << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

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

template <bool BF16>
__device__ __forceinline__ f32x4 mfma(short8 a, short8 b, f32x4 c)
{
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------- elementwise

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_logit_grad16(const float *__restrict__ reward,
                                                           const uint8_t *__restrict__ mask,
                                                           const float *__restrict__ prob,
                                                           uint4 *__restrict__ grad, int blocks,
                                                           int vpb)
{
    const int t = blockIdx.x * kThreads + threadIdx.x;
    if (t >= blocks * vpb) return;
    const int b = t / vpb, v = t - b * vpb;
    uint4 o = make_uint4(0u, 0u, 0u, 0u);
    if (v == 0) {
        const float a = mask[b] ? 1.f : 0.f;
        o.x = f32_to_h16<BF16>(-reward[b] * (a - prob[b]));
    }
    grad[t] = o;
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_grad_combine16(const uint4 *__restrict__ a,
                                                             const uint4 *__restrict__ b,
                                                             const uint4 *__restrict__ y,
                                                             uint4 *__restrict__ out, long long nvec)
{
    const long long t = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (t >= nvec) return;
    const uint4 va = a[t];
    const uint4 vb = b ? b[t] : make_uint4(0u, 0u, 0u, 0u);
    const uint4 vy = y ? y[t] : make_uint4(0u, 0u, 0u, 0u);
    const uint32_t aa[4] = {va.x, va.y, va.z, va.w}, bb[4] = {vb.x, vb.y, vb.z, vb.w};
    const uint32_t yy[4] = {vy.x, vy.y, vy.z, vy.w};
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t r = 0;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int sh = 16 * hh;
            float z = h16_to_f32<BF16>((aa[q] >> sh) & 0xFFFFu);
            if (b) z += h16_to_f32<BF16>((bb[q] >> sh) & 0xFFFFu);
            if (y && !(h16_to_f32<BF16>((yy[q] >> sh) & 0xFFFFu) > 0.f)) z = 0.f;
            r |= f32_to_h16<BF16>(z) << sh;
        }
        o[q] = r;
    }
    out[t] = make_uint4(o[0], o[1], o[2], o[3]);
}

// W [co][kh][kw][ci] -> W' [ci][kh][kw][co], taps reversed
// W' [ci][i][j][co] = W[co][k-1-i][k-1-j][ci]: the weights of the transposed convolution
__device__ __forceinline__ void flip_transpose_at(const uint16_t *__restrict__ w,
                                                  uint16_t *__restrict__ wt, int cout, int k,
                                                  int cin, int t)
{
    if (t >= cout * k * k * cin) return;
    const int co = t % cout;
    int r = t / cout;
    const int j = r % k;
    r /= k;
    const int i = r % k;
    const int ci = r / k;
    wt[t] = w[((co * k + (k - 1 - i)) * k + (k - 1 - j)) * cin + ci];
}

// Z [n][2h][2w][C]: Z[2y][2x] = G[y][x], zero elsewhere (16-byte vectors, C % 8 == 0)
__device__ __forceinline__ void zero_insert_at(const uint4 *__restrict__ g, uint4 *__restrict__ z,
                                               int n, int h, int w, int vpp, long long t)
{
    if (t >= (long long)n * 4 * h * w * vpp) return;
    const int v = (int)(t % vpp);
    long long r = t / vpp;
    const int x = (int)(r % (2 * w));
    r /= 2 * w;
    const int y = (int)(r % (2 * h));
    const int img = (int)(r / (2 * h));
    uint4 o = make_uint4(0u, 0u, 0u, 0u);
    if (!(x & 1) && !(y & 1)) o = g[(((long long)img * h + (y >> 1)) * w + (x >> 1)) * vpp + v];
    z[t] = o;
}

// Both inputs of the transposed convolution in one launch: workgroups below wblocks
// flip the weights, the rest (none at stride 1) spread the output gradient.
__global__ __launch_bounds__(kThreads) void k_input_grad_prep16(
    const uint16_t *__restrict__ w, uint16_t *__restrict__ wt, int cout, int k, int cin,
    unsigned wblocks, const uint4 *__restrict__ g, uint4 *__restrict__ z, int n, int h, int wd,
    int vpp)
{
    if (blockIdx.x < wblocks)
        flip_transpose_at(w, wt, cout, k, cin, (int)(blockIdx.x * kThreads + threadIdx.x));
    else
        zero_insert_at(g, z, n, h, wd, vpp,
                       (long long)(blockIdx.x - wblocks) * kThreads + threadIdx.x);
}

// ---------------------------------------------------------------- weight gradient

constexpr int kPx = 128;                      // pixels per chunk (four MFMA k steps)
constexpr int kRow = kPx * 2 + 16;            // LDS bytes per channel row (+16 pad)
constexpr int kWgPx = 1024;                   // pixels per workgroup (8 chunks)

struct WgradGeom {
    int n, hin, win, cin, hout, wout, cout, k, stride, pad;
    int npix;                                 // n * hout * wout
    int splits;                               // pixel ranges per (tile, tap)
    int x_bytes, g_bytes;
};

// LDS per chunk: G and X transposed, [channel][pixel], 64 rows of kRow bytes each. A
// thread holds eight channels (vector cv) of four consecutive pixels (quad pq) of each
// tensor and writes each channel's four pixels as one 8-byte word. With pq the fast
// index over a wave's lanes and a row pitch of 68 dwords, those writes and the MFMA
// fragment reads (16 rows at one column) are both free of bank conflicts.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_wgrad16(const uint16_t *__restrict__ x,
                                                      const uint16_t *__restrict__ g,
                                                      float *__restrict__ dw, float *__restrict__ db,
                                                      WgradGeom G)
{
    __shared__ __align__(16) uint8_t lds[2][2][64 * kRow];   // [buffer][G, X][channel][pixel]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    // blockIdx.x = ((co tile * ci tiles + ci tile) * taps + tap) * splits + split
    const int ci_tiles = (G.cin + 63) / 64, taps = G.k * G.k;
    int r = blockIdx.x;
    const int split = r % G.splits;
    r /= G.splits;
    const int tap = r % taps;
    r /= taps;
    const int cit = r % ci_tiles, cot = r / ci_tiles;
    const int co0 = cot * 64, ci0 = cit * 64;
    const int ti = tap / G.k, tj = tap - ti * G.k;
    const int p_lo = split * kWgPx, p_hi = min(G.npix, p_lo + kWgPx);
    const int nch = (p_hi - p_lo + kPx - 1) / kPx;
    // the bias gradient comes from the first ci tile's tap-0 workgroups
    const bool bias = db != nullptr && cit == 0 && tap == 0;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        (void *)x, (short)0, G.x_bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rg = __builtin_amdgcn_make_buffer_rsrc(
        (void *)g, (short)0, G.g_bytes, kBufferFlags);
    const int pq = tid & 31, cv = tid >> 5;
    const int hw = G.hout * G.wout;
    const bool ci_ok = ci0 + cv * 8 < G.cin;
    auto load = [&](int c, i32x4 (&vg)[4], i32x4 (&vx)[4]) {
        const int p0 = p_lo + c * kPx + 4 * pq;
        int img = 0, oy = 0, ox = 0;
        if (p0 < p_hi) {
            img = p0 / hw;
            const int rem = p0 - img * hw;
            oy = rem / G.wout;
            ox = rem - oy * G.wout;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int p = p0 + j;
            int og = kOutOfRange, oi = kOutOfRange;
            if (p < p_hi) {
                og = (p * G.cout + co0 + cv * 8) * 2;
                const int iy = oy * G.stride - G.pad + ti, ix = ox * G.stride - G.pad + tj;
                if (iy >= 0 && iy < G.hin && ix >= 0 && ix < G.win && ci_ok)
                    oi = (((img * G.hin + iy) * G.win + ix) * G.cin + ci0 + cv * 8) * 2;
            }
            asm volatile("" : "+v"(og), "+v"(oi));
            vg[j] = __builtin_amdgcn_raw_buffer_load_b128(rg, og, 0, 0);
            vx[j] = __builtin_amdgcn_raw_buffer_load_b128(rx, oi, 0, 0);
            if (++ox == G.wout) {
                ox = 0;
                if (++oy == G.hout) {
                    oy = 0;
                    ++img;
                }
            }
        }
    };
    float bsum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    // channel e of the four pixels: halves e&1 of dword e>>1, pixels 0..3 -> one 8-byte word
    auto pack = [](const i32x4 (&v)[4], int e) {
        const int w = e >> 1;
        uint2 o;
        if (e & 1) {
            o.x = ((uint32_t)v[0][w] >> 16) | ((uint32_t)v[1][w] & 0xFFFF0000u);
            o.y = ((uint32_t)v[2][w] >> 16) | ((uint32_t)v[3][w] & 0xFFFF0000u);
        } else {
            o.x = ((uint32_t)v[0][w] & 0xFFFFu) | ((uint32_t)v[1][w] << 16);
            o.y = ((uint32_t)v[2][w] & 0xFFFFu) | ((uint32_t)v[3][w] << 16);
        }
        return o;
    };
    auto store = [&](int buf, const i32x4 (&vg)[4], const i32x4 (&vx)[4]) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int off = (cv * 8 + e) * kRow + pq * 8;
            *(uint2 *)(lds[buf][0] + off) = pack(vg, e);
            *(uint2 *)(lds[buf][1] + off) = pack(vx, e);
        }
        if (bias) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    bsum[e] += h16_to_f32<BF16>(((uint32_t)vg[j][e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
        }
    };
    f32x4 acc[2][2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int buf) {
#pragma unroll
        for (int ks = 0; ks < kPx / 32; ++ks) {
            const int foff = ks * 64 + (lane >> 4) * 16;   // this lane's 8 pixels
            short8 af[2], bf[2];
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
                af[mi] = *(const short8 *)(lds[buf][0] + (wm * 32 + mi * 16 + (lane & 15)) * kRow + foff);
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
                bf[ni] = *(const short8 *)(lds[buf][1] + (wn * 32 + ni * 16 + (lane & 15)) * kRow + foff);
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = mfma<BF16>(af[mi], bf[ni], acc[mi][ni]);
        }
    };
    // two chunks in flight: register slot d holds chunk c (d = c & 1) until its store,
    // then receives chunk c + 2; LDS buffer d is rewritten two chunks after it was
    // read, and every thread passes the barrier in between
    i32x4 vg[2][4], vx[2][4];
    load(0, vg[0], vx[0]);
    load(1, vg[1], vx[1]);
    auto step = [&](auto dc, int cc) {
        constexpr int d = decltype(dc)::value;
        store(d, vg[d], vx[d]);
        __syncthreads();
        load(cc + 2, vg[d], vx[d]);              // past the range: zeros, never used
        compute(d);
    };
    // whole pairs of chunks in the loop (no exit inside it), then the odd last chunk
    int c = 0;
    for (; c + 2 <= nch; c += 2) {
        step(std::integral_constant<int, 0>{}, c);
        step(std::integral_constant<int, 1>{}, c + 1);
    }
    if (c < nch) step(std::integral_constant<int, 0>{}, c);
    // acc[mi][ni][i]: co = wm*32 + mi*16 + (lane>>4)*4 + i, ci = wn*32 + ni*16 + (lane&15)
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
            const int ci = ci0 + wn * 32 + ni * 16 + (lane & 15);
            if (ci >= G.cin) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int co = co0 + wm * 32 + mi * 16 + (lane >> 4) * 4 + i;
                unsafeAtomicAdd(&dw[((size_t)co * taps + tap) * G.cin + ci], acc[mi][ni][i]);
            }
        }
    if (bias) {
        // the 32 lanes of one channel vector (one half of the wave) hold its pixel quads
#pragma unroll
        for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int m = 1; m < 32; m <<= 1) bsum[e] += __shfl_xor(bsum[e], m, 64);
        if (pq == 0)
#pragma unroll
            for (int e = 0; e < 8; ++e) unsafeAtomicAdd(&db[co0 + cv * 8 + e], bsum[e]);
    }
}

// ---------------------------------------------------------------- RMSprop

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_rmsprop(float *__restrict__ w, float *__restrict__ v,
                                                      float *__restrict__ grad, long long count,
                                                      float lr, float alpha, float eps, float wd,
                                                      uint16_t *__restrict__ w16)
{
    const long long t = (long long)blockIdx.x * kThreads + threadIdx.x;
    if (t >= count) return;
    const float wi = w[t];
    const float gi = grad[t] + wd * wi;
    const float vi = alpha * v[t] + (1.f - alpha) * gi * gi;
    const float wn = wi - lr * gi / (sqrtf(vi) + eps);
    v[t] = vi;
    w[t] = wn;
    grad[t] = 0.f;
    if (w16) w16[t] = (uint16_t)f32_to_h16<BF16>(wn);
}

// Several tensors in one launch: workgroup b belongs to the tensor t with
// first[t] <= b < first[t + 1] (a uniform scan over at most kMaxParams entries of the
// kernel arguments), element (b - first[t]) * kThreads + thread of that tensor.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_rmsprop_many(RmspropMany m, float lr, float alpha,
                                                           float eps, float wd)
{
    const int b = blockIdx.x;
    int t = 0;
    while (t + 1 < m.n && m.first[t + 1] <= b) ++t;
    const long long i = (long long)(b - m.first[t]) * kThreads + threadIdx.x;
    if (i >= m.count[t]) return;
    float *w = m.w[t], *v = m.v[t], *grad = m.grad[t];
    const float wi = w[i];
    const float gi = grad[i] + wd * wi;
    const float vi = alpha * v[i] + (1.f - alpha) * gi * gi;
    const float wn = wi - lr * gi / (sqrtf(vi) + eps);
    v[i] = vi;
    w[i] = wn;
    grad[i] = 0.f;
    if (m.w16[t]) m.w16[t][i] = (uint16_t)f32_to_h16<BF16>(wn);
}

// ---------------------------------------------------------------- workspace

// Library-owned workspace of the input gradients, one per device. It grows by allocating
// a larger buffer; the old one is kept (never freed), so a graph that captured a call
// keeps a valid pointer. hipMalloc is not allowed during capture: a capturing call that
// would grow it is refused.
std::mutex g_tw_mu;
void *g_tw_ptr[64];
size_t g_tw_bytes[64];

hipError_t train_workspace(size_t bytes, hipStream_t s, void **out, const char **why)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_tw_mu);
    if (g_tw_bytes[dev] < bytes) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        e = hipStreamIsCapturing(s, &cs);
        if (e != hipSuccess) return e;
        if (cs != hipStreamCaptureStatusNone) {
            *why = "the input-gradient workspace must grow and the stream is capturing (no "
                   "allocation during capture): make one uncaptured call at the largest size first";
            return hipErrorStreamCaptureUnsupported;
        }
        size_t want = 2 * g_tw_bytes[dev];
        if (want < bytes) want = bytes;
        if (want < ((size_t)16 << 20)) want = (size_t)16 << 20;
        void *p = nullptr;
        e = hipMalloc(&p, want);
        if (e != hipSuccess) return e;
        g_tw_ptr[dev] = p;          // the previous buffer stays allocated (see above)
        g_tw_bytes[dev] = want;
    }
    *out = g_tw_ptr[dev];
    return hipSuccess;
}

unsigned blocks_for(long long n) { return (unsigned)((n + kThreads - 1) / kThreads); }

}  // namespace

hipError_t launch_logit_grad(const float *reward, const uint8_t *mask, const float *prob,
                             void *grad, int blocks, int c, bool bf16, hipStream_t s)
{
    const int vpb = c / 8;
    if (bf16)
        hipLaunchKernelGGL(k_logit_grad16<true>, dim3(blocks_for((long long)blocks * vpb)), dim3(kThreads), 0, s,
                           reward, mask, prob, (uint4 *)grad, blocks, vpb);
    else
        hipLaunchKernelGGL(k_logit_grad16<false>, dim3(blocks_for((long long)blocks * vpb)), dim3(kThreads), 0, s,
                           reward, mask, prob, (uint4 *)grad, blocks, vpb);
    return hipGetLastError();
}

hipError_t launch_grad_combine(const void *a, const void *b, const void *y, void *out,
                               long long elems, bool bf16, hipStream_t s)
{
    const long long nvec = elems / 8;
    if (bf16)
        hipLaunchKernelGGL(k_grad_combine16<true>, dim3(blocks_for(nvec)), dim3(kThreads), 0, s,
                           (const uint4 *)a, (const uint4 *)b, (const uint4 *)y, (uint4 *)out, nvec);
    else
        hipLaunchKernelGGL(k_grad_combine16<false>, dim3(blocks_for(nvec)), dim3(kThreads), 0, s,
                           (const uint4 *)a, (const uint4 *)b, (const uint4 *)y, (uint4 *)out, nvec);
    return hipGetLastError();
}

hipError_t launch_conv_input_grad(const uint16_t *grad_out, const uint16_t *w, const uint16_t *accum,
                                  uint16_t *grad_in, const LayerGeom &fwd, Half16 fmt,
                                  hipStream_t s, const char **why)
{
    // workspace: flipped weights, then (stride 2) the spread output gradient
    const size_t wbytes = ((size_t)fwd.cout * fwd.kh * fwd.kw * fwd.cin * 2 + 255) & ~(size_t)255;
    const size_t zbytes = fwd.stride == 2 ? (size_t)fwd.n * fwd.hin * fwd.win * fwd.cout * 2 : 0;
    void *ws = nullptr;
    hipError_t e = train_workspace(wbytes + zbytes, s, &ws, why);
    if (e != hipSuccess) return e;
    uint16_t *wt = (uint16_t *)ws;
    const unsigned wblocks = blocks_for((long long)fwd.cout * fwd.kh * fwd.kw * fwd.cin);
    const uint16_t *src = grad_out;
    uint16_t *z = nullptr;
    unsigned zblocks = 0;
    if (fwd.stride == 2) {
        z = (uint16_t *)((uint8_t *)ws + wbytes);
        zblocks = blocks_for((long long)fwd.n * fwd.hin * fwd.win * (fwd.cout / 8));
        src = z;
    }
    hipLaunchKernelGGL(k_input_grad_prep16, dim3(wblocks + zblocks), dim3(kThreads), 0, s, w, wt,
                       fwd.cout, fwd.kh, fwd.cin, wblocks, (const uint4 *)grad_out, (uint4 *)z,
                       fwd.n, fwd.hout, fwd.wout, fwd.cout / 8);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // stride-1 convolution of the (spread) output gradient with the flipped weights,
    // every block of the input-sized map (blocks of at most 8 x 8 pixels)
    LayerGeom L;
    L.n = fwd.n;
    L.cin = fwd.cout; L.hin = fwd.hin; L.win = fwd.win;
    L.cout = fwd.cin; L.hout = fwd.hin; L.wout = fwd.win;
    L.kh = fwd.kh; L.kw = fwd.kw; L.stride = 1; L.pad = fwd.kh / 2;
    L.bh = fwd.hin < 8 ? fwd.hin : 8;
    L.bw = fwd.win < 8 ? fwd.win : 8;
    L.gh = fwd.hin / L.bh; L.gw = fwd.win / L.bw;
    L.total_blocks = L.n * L.gh * L.gw;
    L.idx = nullptr;
    L.count = nullptr;
    return launch_conv_nhwc_mfma(src, wt, nullptr, accum, grad_in, 0, fmt, L, s, why);
}

hipError_t launch_conv_weight_grad(const uint16_t *x, const uint16_t *g, float *dw, float *db,
                                   const LayerGeom &fwd, bool bf16, hipStream_t s)
{
    WgradGeom G;
    G.n = fwd.n; G.hin = fwd.hin; G.win = fwd.win; G.cin = fwd.cin;
    G.hout = fwd.hout; G.wout = fwd.wout; G.cout = fwd.cout;
    G.k = fwd.kh; G.stride = fwd.stride; G.pad = fwd.pad;
    G.npix = fwd.n * fwd.hout * fwd.wout;
    G.splits = (G.npix + kWgPx - 1) / kWgPx;
    G.x_bytes = (int)((size_t)fwd.n * fwd.hin * fwd.win * fwd.cin * 2);
    G.g_bytes = (int)((size_t)G.npix * fwd.cout * 2);
    const unsigned grid = (unsigned)((fwd.cout / 64) * ((fwd.cin + 63) / 64) * G.k * G.k * G.splits);
    if (bf16) hipLaunchKernelGGL(k_wgrad16<true>, dim3(grid), dim3(kThreads), 0, s, x, g, dw, db, G);
    else hipLaunchKernelGGL(k_wgrad16<false>, dim3(grid), dim3(kThreads), 0, s, x, g, dw, db, G);
    return hipGetLastError();
}

hipError_t launch_rmsprop_many(const RmspropMany &m, float lr, float alpha, float eps, float wd,
                               bool bf16, hipStream_t s)
{
    const dim3 grid((unsigned)m.first[m.n]), block(kThreads);
    if (bf16)
        hipLaunchKernelGGL(k_rmsprop_many<true>, grid, block, 0, s, m, lr, alpha, eps, wd);
    else
        hipLaunchKernelGGL(k_rmsprop_many<false>, grid, block, 0, s, m, lr, alpha, eps, wd);
    return hipGetLastError();
}

hipError_t launch_rmsprop(float *w, float *v, float *grad, long long count, float lr, float alpha,
                          float eps, float wd, void *w16, bool bf16, hipStream_t s)
{
    if (bf16)
        hipLaunchKernelGGL(k_rmsprop<true>, dim3(blocks_for(count)), dim3(kThreads), 0, s, w, v, grad,
                           count, lr, alpha, eps, wd, (uint16_t *)w16);
    else
        hipLaunchKernelGGL(k_rmsprop<false>, dim3(blocks_for(count)), dim3(kThreads), 0, s, w, v, grad,
                           count, lr, alpha, eps, wd, (uint16_t *)w16);
    return hipGetLastError();
}

}  // namespace bc
