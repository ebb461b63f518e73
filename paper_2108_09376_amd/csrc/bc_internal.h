// Internal declarations shared by the C-ABI layer (bc_api.cpp) and the HIP kernel
// translation units. Not part of the public ABI (that is include/bc.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

// Geometry of one block-sparse layer call, resolved and validated on the host.
// Output blocks are bh x bw pixels on a gh x gw grid per image; ids index them as
// (img * gh + gy) * gw + gx. idx == nullptr means "every block" (full frame).
struct LayerGeom {
    int n, cin, hin, win;      // input
    int cout, hout, wout;      // output
    int kh, kw, stride, pad;
    int gh, gw, bh, bw;
    int total_blocks;          // n * gh * gw
    const int32_t *idx;        // device, ascending active ids, or nullptr
    const int32_t *count;      // device, number of active ids, or nullptr
};

// Storage formats of the half-width paths.
enum class Half16 { BF16, F16 };

hipError_t launch_block_index(const uint8_t *mask, int total, int32_t *idx, int32_t *count,
                              hipStream_t s);

// Gather/scatter of halo tiles, any element size (2 or 4 bytes), NHWC or NCHW source.
hipError_t launch_gather_halo(const void *src, int esize, bool nhwc, const LayerGeom &g,
                              uint32_t pad_bits, void *packed, hipStream_t s);
hipError_t launch_scatter_blocks(const void *packed, int esize, bool nhwc, const LayerGeom &g,
                                 void *dst, hipStream_t s);

// Max pooling, NHWC bf16/f16 or NCHW f32.
hipError_t launch_maxpool_nhwc16(const uint16_t *x, uint16_t *y, Half16 fmt, const LayerGeom &g,
                                 hipStream_t s);
hipError_t launch_maxpool_nchw32(const float *x, float *y, const LayerGeom &g, hipStream_t s);

// Convolutions. Return hipErrorInvalidValue (with *why set) for shapes they cannot take.
hipError_t launch_conv_nchw_f32(const float *x, const float *w, const float *bias,
                                const float *res, float *y, int relu, const LayerGeom &g,
                                hipStream_t s, const char **why);
hipError_t launch_conv_nhwc_mfma(const uint16_t *x, const uint16_t *w, const float *bias,
                                 const uint16_t *res, uint16_t *y, int relu, Half16 fmt,
                                 const LayerGeom &g, hipStream_t s, const char **why);
// The same layer with split-K partials in the library's fixed `scratch` array instead of
// the allocated workspace: no allocation at any call. conv_nhwc_split_bytes gives the
// partials' size of a layer's plan (0 if it does not split K), conv_nhwc_scratch_bytes
// the array's size.
hipError_t launch_conv_nhwc_mfma_noalloc(const uint16_t *x, const uint16_t *w, const float *bias,
                                         const uint16_t *res, uint16_t *y, int relu, Half16 fmt,
                                         const LayerGeom &g, hipStream_t s, const char **why);
size_t conv_nhwc_split_bytes(const LayerGeom &g);
size_t conv_nhwc_scratch_bytes();
// Two independent channels-last layers: one launch when both are 1x1 layers whose plans
// pair (the second at stride 1, neither splitting K, BF16), else one launch each.
struct ConvCall {
    const uint16_t *x, *w, *res;
    const float *bias;
    uint16_t *y;
    int relu;
    LayerGeom g;
};
hipError_t launch_conv_pair_nhwc_mfma(const ConvCall &c1, const ConvCall &c2, Half16 fmt,
                                      hipStream_t s, const char **why);
// Host-side check used by the ABI validation before anything is enqueued.
bool conv_nhwc_mfma_supported(const LayerGeom &g, const char **why);

// Execution decisions from block probabilities (Philox4x32-10) fused with the index.
hipError_t launch_sample_index(const float *prob, int total, uint64_t seed, uint64_t frame,
                               uint8_t *mask, int32_t *idx, int32_t *count, hipStream_t s);
// Frame state: copy the active blocks of `frame` into `state` (same shape, any dtype).
hipError_t launch_frame_state(const void *frame, void *state, int n, int c, int h, int w,
                              int esize, bool nhwc, int gh, int gw, const int32_t *idx,
                              const int32_t *count, hipStream_t s);
// Per-block maximum of the per-pixel KL divergence of two score maps: the first
// `classes` of c channels, [n][c][h][w] fp32 or [n][h][w][c] bf16/fp16 (c % 8 == 0).
hipError_t launch_seg_information_gain(const void *lt, const void *lp, int n, int c, int classes,
                                       int h, int w, int esize, bool nhwc, bool bf16, int gh,
                                       int gw, const uint8_t *mask, float *ig, hipStream_t s);
// Rewards, cost, moving average and REINFORCE loss per image.
hipError_t launch_block_rewards(const float *ig, const uint8_t *mask, const float *prob, int n,
                                int blocks, float tau, float gamma, float mu, float *mavg,
                                float *reward, float *cost, float *loss, hipStream_t s);

// Decoder merge: out = up2(coarse) (+ skip) (ReLU) on the active output blocks; coarse
// [n][hc][wc][c] (bf16/fp16, c % 8 == 0) or [n][c][hc][wc] fp32, out/skip 2hc x 2wc.
hipError_t launch_upsample_add(const void *coarse, const void *skip, void *out, int n, int c,
                               int hc, int wc, int esize, bool nhwc, bool bf16, int gh, int gw,
                               const int32_t *idx, const int32_t *count, int relu, hipStream_t s);

// Pyramid pooling (k_spp.hip): levels computed densely from the whole input map, then
// the executed blocks of the concatenation [input, upsampled levels]. Channels last,
// bf16/fp16; c % 8 == 0 with c / 8 dividing 256 (c <= kMaxSppChannels), cl % 8 == 0.
constexpr int kMaxSppLevels = 8;
constexpr int kMaxSppChannels = 2048;
struct SppGeom {
    int n, h, w, c, vpp;                       // input [n][h][w][c], vpp = c / 8
    int levels, cl, cout;                      // cout = c + levels * cl
    int rows[kMaxSppLevels], cols[kMaxSppLevels];
    int first[kMaxSppLevels + 1];              // first bin of each level; first[levels] = bins
    int gh, gw, bh, bw, total_blocks;          // output blocks
    int in_bytes, w_bytes, lv_bytes, out_bytes;
};
hipError_t launch_spp(const uint16_t *in, const uint16_t *w, const float *bias, uint16_t *levels,
                      uint16_t *out, const SppGeom &g, bool bf16, const int32_t *idx,
                      const int32_t *count, hipStream_t s);

// Policy network input S_t at a quarter of the frame resolution (32 channels) and the
// block probabilities from the head's logits (channel 0 of c).
hipError_t launch_policy_input(const void *frame, const void *state, const void *scores,
                               const uint8_t *mask, void *out, int n, int h, int w, int c,
                               int classes, int gh, int gw, bool bf16, hipStream_t s);
hipError_t launch_policy_probabilities(const void *logits, int blocks, int c, bool bf16,
                                       float *prob, hipStream_t s);

// Policy training: logit gradient, gradient combine, conv input / weight gradients,
// RMSprop (k_train.hip).
hipError_t launch_logit_grad(const float *reward, const uint8_t *mask, const float *prob,
                             void *grad, int blocks, int c, bool bf16, hipStream_t s);
hipError_t launch_grad_combine(const void *a, const void *b, const void *y, void *out,
                               long long elems, bool bf16, hipStream_t s);
hipError_t launch_conv_input_grad(const uint16_t *grad_out, const uint16_t *w, const uint16_t *accum,
                                  uint16_t *grad_in, const LayerGeom &fwd, Half16 fmt,
                                  hipStream_t s, const char **why);
hipError_t launch_conv_weight_grad(const uint16_t *x, const uint16_t *g, float *dw, float *db,
                                   const LayerGeom &fwd, bool bf16, hipStream_t s);
// Multi-tensor RMSprop: up to kMaxParams tensors; first[t] is the first workgroup of
// tensor t (first[n] = the grid), each workgroup covering 256 elements.
constexpr int kMaxParams = 64;
struct RmspropMany {
    float *w[kMaxParams], *v[kMaxParams], *grad[kMaxParams];
    uint16_t *w16[kMaxParams];
    long long count[kMaxParams];
    int first[kMaxParams + 1];
    int n;
};
hipError_t launch_rmsprop_many(const RmspropMany &m, float lr, float alpha, float eps, float wd,
                               bool bf16, hipStream_t s);
hipError_t launch_rmsprop(float *w, float *v, float *grad, long long count, float lr, float alpha,
                          float eps, float wd, void *w16, bool bf16, hipStream_t s);

}  // namespace bc
