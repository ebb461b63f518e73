// The policy network's input and output stages (Section 3.3, Eq. 2). The network maps
// S_t = {I_t, H_{t-1}, A_{t-1}, O_{t-1}} to one execution probability per block; its
// convolutions run on the library's dense path (every block). Here:
//  * input: S_t is assembled at a quarter of the frame resolution (where the
//    segmentation output O_{t-1} lives) as 32 channels: the frame I_t and the frame
//    state H_{t-1} averaged over each 4x4 pixel cell, the class probabilities of
//    O_{t-1} (softmax over its first `classes` score channels), A_{t-1} of the pixel's
//    block, zeros. One thread per output pixel: 24 bytes per cell row of each RGB map
//    (three 8-byte loads), the class scores as 16-byte loads, one byte of the grid; all
//    issued before any use; fp32 arithmetic, one round to the storage format; four
//    16-byte stores.
//  * output: p_b = sigmoid(logit_b), the logit being channel 0 of the head's map, which
//    has one pixel per block.
#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 256;
constexpr int kBufferFlags = 0x00020000;     // raw buffer, dword format
constexpr int kOutOfRange = 0x7FFFFF00;      // loads return 0, stores are dropped
constexpr int kMaxClasses = 24;              // class scores read per pixel (three vectors)

typedef int i32x2 __attribute__((ext_vector_type(2)));
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

__device__ __forceinline__ uint32_t half_of(const i32x2 (&v)[3], int e)
{
    return ((uint32_t)v[e >> 2][(e >> 1) & 1] >> (16 * (e & 1))) & 0xFFFFu;
}

struct PolicyGeom {
    int n, h, w;                 // frame size (h, w multiples of 4)
    int c;                       // channels of the score map, classes of them used
    int classes;
    int gh, gw;                  // block grid of the frame
    int frame_bytes, score_bytes, out_bytes;
};

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_policy_input16(
    const uint16_t *__restrict__ frame, const uint16_t *__restrict__ state,
    const uint16_t *__restrict__ scores, const uint8_t *__restrict__ mask,
    uint16_t *__restrict__ out, PolicyGeom g)
{
    const int h4 = g.h >> 2, w4 = g.w >> 2;
    const int total = g.n * h4 * w4;
    const int t = blockIdx.x * kThreads + threadIdx.x;
    const int pix = min(t, total - 1);                  // clamped: every load is in range
    const int img = pix / (h4 * w4);
    const int rem = pix - img * h4 * w4;
    const int y = rem / w4, x = rem - y * w4;
    const __amdgpu_buffer_rsrc_t rf = __builtin_amdgcn_make_buffer_rsrc(
        (void *)frame, (short)0, g.frame_bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)state, (short)0, g.frame_bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)scores, (short)0, g.score_bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void *)out, (short)0, g.out_bytes, kBufferFlags);
    // a cell row is 4 pixels x 3 channels = 24 bytes, 8-byte aligned (w % 4 == 0)
    i32x2 fv[4][3], sv[4][3];
#pragma unroll
    for (int dy = 0; dy < 4; ++dy) {
        const int row = ((img * g.h + 4 * y + dy) * g.w + 4 * x) * 6;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            fv[dy][k] = __builtin_amdgcn_raw_buffer_load_b64(rf, row + 8 * k, 0, 0);
            sv[dy][k] = __builtin_amdgcn_raw_buffer_load_b64(rs, row + 8 * k, 0, 0);
        }
    }
    const int sbase = ((img * h4 + y) * w4 + x) * g.c * 2;
    i32x4 cv[3];
#pragma unroll
    for (int j = 0; j < 3; ++j)
        cv[j] = __builtin_amdgcn_raw_buffer_load_b128(rc, 16 * j < g.c * 2 ? sbase + 16 * j : kOutOfRange, 0, 0);
    const int bid = (img * g.gh + y / (h4 / g.gh)) * g.gw + x / (w4 / g.gw);
    const float a_prev = mask ? (float)(mask[bid] != 0) : 0.f;

    float z[32];
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        float sf = 0.f, ss = 0.f;
#pragma unroll
        for (int dy = 0; dy < 4; ++dy)
#pragma unroll
            for (int px = 0; px < 4; ++px) {
                sf += h16_to_f32<BF16>(half_of(fv[dy], px * 3 + ch));
                ss += h16_to_f32<BF16>(half_of(sv[dy], px * 3 + ch));
            }
        z[ch] = sf * 0.0625f;
        z[3 + ch] = ss * 0.0625f;
    }
    float sc[kMaxClasses];
    float mx = -__builtin_inff();
#pragma unroll
    for (int k = 0; k < kMaxClasses; ++k) {
        sc[k] = h16_to_f32<BF16>(((uint32_t)cv[k >> 3][(k >> 1) & 3] >> (16 * (k & 1))) & 0xFFFFu);
        if (k < g.classes) mx = fmaxf(mx, sc[k]);
    }
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxClasses; ++k) {
        sc[k] = k < g.classes ? __expf(sc[k] - mx) : 0.f;
        sum += sc[k];
    }
    const float inv = 1.f / sum;
#pragma unroll
    for (int k = 6; k < 32; ++k) z[k] = 0.f;
#pragma unroll
    for (int k = 0; k < kMaxClasses; ++k)
        if (k < g.classes) z[6 + k] = sc[k] * inv;
#pragma unroll
    for (int k = 0; k < 32 - 6; ++k)
        if (k == g.classes) z[6 + k] = a_prev;
    const int obase = t < total ? pix * 64 : kOutOfRange;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        i32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            o[q] = (int)(f32_to_h16<BF16>(z[8 * v + 2 * q]) | (f32_to_h16<BF16>(z[8 * v + 2 * q + 1]) << 16));
        __builtin_amdgcn_raw_buffer_store_b128(o, ro, obase + 16 * v, 0, 0);
    }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_policy_prob16(const uint16_t *__restrict__ logits,
                                                            int blocks, int c,
                                                            float *__restrict__ prob)
{
    const int b = blockIdx.x * kThreads + threadIdx.x;
    if (b >= blocks) return;
    const float l = h16_to_f32<BF16>(logits[(size_t)b * c]);
    prob[b] = 1.f / (1.f + __expf(-l));
}

}  // namespace

hipError_t launch_policy_input(const void *frame, const void *state, const void *scores,
                               const uint8_t *mask, void *out, int n, int h, int w, int c,
                               int classes, int gh, int gw, bool bf16, hipStream_t s)
{
    PolicyGeom g;
    g.n = n; g.h = h; g.w = w; g.c = c; g.classes = classes; g.gh = gh; g.gw = gw;
    g.frame_bytes = (int)((size_t)n * h * w * 3 * 2);
    g.score_bytes = (int)((size_t)n * (h / 4) * (w / 4) * c * 2);
    g.out_bytes = (int)((size_t)n * (h / 4) * (w / 4) * 32 * 2);
    const int total = n * (h / 4) * (w / 4);
    const dim3 grid((unsigned)((total + kThreads - 1) / kThreads)), block(kThreads);
    if (bf16)
        hipLaunchKernelGGL(k_policy_input16<true>, grid, block, 0, s, (const uint16_t *)frame,
                           (const uint16_t *)state, (const uint16_t *)scores, mask, (uint16_t *)out, g);
    else
        hipLaunchKernelGGL(k_policy_input16<false>, grid, block, 0, s, (const uint16_t *)frame,
                           (const uint16_t *)state, (const uint16_t *)scores, mask, (uint16_t *)out, g);
    return hipGetLastError();
}

hipError_t launch_policy_probabilities(const void *logits, int blocks, int c, bool bf16,
                                       float *prob, hipStream_t s)
{
    const dim3 grid((unsigned)((blocks + kThreads - 1) / kThreads)), block(kThreads);
    if (bf16)
        hipLaunchKernelGGL(k_policy_prob16<true>, grid, block, 0, s, (const uint16_t *)logits, blocks, c, prob);
    else
        hipLaunchKernelGGL(k_policy_prob16<false>, grid, block, 0, s, (const uint16_t *)logits, blocks, c, prob);
    return hipGetLastError();
}

}  // namespace bc
