/*
 * bc.h -- C ABI of the MI355X (gfx950) block-sparse convolution library with
 * temporal feature copying (BlockCopy, Verelst & Tuytelaars, ICCV 2021).
 *
 * What the library computes (Section 3.1 and the caption of Fig. 3): a CNN layer
 * is executed only on the image blocks that the frame's execution grid selects
 * (a_b = 1, Section 3.5); every other block keeps the layer's representation from
 * the previous execution ("feature transfer", a_b = 0). A selected block is
 * computed with its halo read from its neighbours in the layer's current input,
 * so that there are no discontinuities between blocks (the BlockPadding idea the
 * paper builds on, Section 3.1). For one layer this equals
 *
 *     out = select(mask, layer(in), out_previous)
 *
 * where layer() is the ordinary dense layer and select() keeps out_previous bit
 * for bit outside the selected blocks. Non-selected blocks of `out` are never
 * read or written.
 *
 * Conventions for every entry point:
 *  - Pointers named d_* are DEVICE memory owned by the caller. The library never
 *    allocates, frees or retains caller memory, and never throws or aborts
 *    across the ABI.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream). Work is
 *    enqueued asynchronously; no call synchronises except bc_build_block_index
 *    with a non-NULL h_count.
 *  - All tensors are dense and contiguous in the stated layout.
 *  - Every argument check runs before anything is enqueued; on a non-OK status
 *    nothing was enqueued and no memory was touched. bc_last_error() then holds
 *    a thread-local description. A fault of earlier asynchronous work surfaces
 *    as BC_ERR_HIP on a later call.
 *  - Blocks: the execution grid has grid_h x grid_w blocks per image, the same
 *    grid for every layer of a network (Section 3.5: one decision per block). A
 *    layer whose output is H x W has output blocks of edge bh = H / grid_h,
 *    bw = W / grid_w; H and W must be divisible (else BC_ERR_NOT_DIVISIBLE).
 *    The grid indexes OUTPUT blocks; the input tile of output block (gy, gx) of
 *    a layer with kernel kh x kw, stride s and padding p spans input rows
 *    gy*bh*s - p .. gy*bh*s - p + (bh-1)*s + kh - 1 (same for columns).
 *  - Active-block index: int32 ids id = (img * grid_h + gy) * grid_w + gx of the
 *    selected blocks, strictly ascending, with their number in *d_count (device).
 *    Kernels read the count on the device, so no host round trip is needed.
 *    Passing d_idx = d_count = NULL to a layer call means "every block" (a full
 *    frame, as for the first frame of a clip, Section 4).
 */
#ifndef BC_H
#define BC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BC_ABI_VERSION 10

typedef enum {
    BC_OK = 0,
    BC_ERR_NULL = 1,          /* a required pointer is NULL                      */
    BC_ERR_SHAPE = 2,         /* tensor sizes inconsistent with each other/geometry */
    BC_ERR_DTYPE = 3,         /* dtype mismatch between tensors or unknown dtype  */
    BC_ERR_LAYOUT = 4,        /* layout mismatch or unknown layout               */
    BC_ERR_NOT_DIVISIBLE = 5, /* output size not divisible by the block grid     */
    BC_ERR_CAPACITY = 6,      /* index / packed capacity < n * grid_h * grid_w   */
    BC_ERR_ALIAS = 7,         /* output overlaps an input                        */
    BC_ERR_UNINITIALIZED = 8, /* sparse write into a registered, invalid buffer  */
    BC_ERR_UNSUPPORTED = 9,   /* valid request outside what the kernels implement */
    BC_ERR_HIP = 10,          /* HIP runtime error (launch or earlier async fault) */
    BC_ERR_CAPTURE = 11       /* a library allocation was needed while the stream is
                                 capturing a graph; nothing was enqueued            */
} bc_status;

typedef enum { BC_F32 = 0, BC_BF16 = 1, BC_F16 = 2 } bc_dtype;
typedef enum { BC_NCHW = 0, BC_NHWC = 1 } bc_layout;

/* Shape and format of a 4-D feature map. dtype is a bc_dtype, layout a bc_layout. */
typedef struct { int32_t n, c, h, w; int32_t dtype; int32_t layout; } bc_tensor;

/* Block grid per image. */
typedef struct { int32_t grid_h, grid_w; } bc_grid;

/* Convolution / pooling geometry: kernel kh x kw, stride, zero padding (pooling:
 * -inf padding), fused ReLU flag (conv only). Dilation and groups are 1. */
typedef struct { int32_t kh, kw, stride, pad, relu; } bc_conv;

/* ABI version (BC_ABI_VERSION) of the loaded library. */
int32_t bc_abi_version(void);

/* Static text for a status code. */
const char *bc_status_str(int32_t status);

/* Thread-local detail of the last non-OK status returned on this thread ("" if none). */
const char *bc_last_error(void);

/*
 * Mask -> active-block index (Section 3.5: the execution grid A_t, a_b = 1
 * executes block b).
 *   d_mask   uint8 [n][grid_h][grid_w], device; nonzero byte = execute.
 *   d_idx    int32 [capacity], device, written with the ascending ids of the
 *            nonzero entries; entries at and beyond the count are left untouched.
 *   d_count  int32 [1], device, written with the number of nonzero entries.
 *   h_count  optional host int32; if non-NULL the count is also copied to it and
 *            the call waits for the stream (the only synchronising call).
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE (n, grid <= 0 or n*grid_h*grid_w > 2^20),
 * BC_ERR_CAPACITY (capacity < n*grid_h*grid_w), BC_ERR_HIP.
 */
bc_status bc_build_block_index(const uint8_t *d_mask, int32_t n, bc_grid g,
                               int32_t *d_idx, int32_t capacity, int32_t *d_count,
                               int32_t *h_count, void *stream);

/*
 * Standalone halo gather (the BlockPadding step, Section 3.1): for the k-th active
 * output block of a layer with geometry *geom whose input is `src`, copy its input
 * tile to d_packed[k] = [th][tw][C] (channels last, src dtype), th = (bh-1)*s + kh,
 * tw = (bw-1)*s + kw, where bh x bw is the output block edge implied by src, geom
 * and the grid. Positions outside the image get pad_value (rounded to the dtype).
 *   d_src     src.layout (NCHW or NHWC), any dtype.
 *   d_packed  [capacity][th][tw][C]; only the first *d_count tiles are written.
 * d_idx/d_count may both be NULL (every block). Errors: BC_ERR_NULL, BC_ERR_SHAPE,
 * BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_NOT_DIVISIBLE, BC_ERR_CAPACITY, BC_ERR_ALIAS,
 * BC_ERR_UNSUPPORTED (stride outside {1,2}, kernel edge outside 1..7), BC_ERR_HIP.
 */
bc_status bc_gather_halo(const void *d_src, bc_tensor src, bc_grid g, const bc_conv *geom,
                         float pad_value, const int32_t *d_idx, const int32_t *d_count,
                         int32_t capacity, void *d_packed, void *stream);

/*
 * Standalone scatter into a persistent buffer (Section 3.1, stored representations):
 * d_packed[k] = [bh][bw][C] (channels last, dst dtype) is written to the position of
 * the k-th active block of `dst`, bh = dst.h / grid_h, bw = dst.w / grid_w. Every
 * other element of dst is neither read nor written.
 * Errors: as bc_gather_halo.
 */
bc_status bc_scatter_blocks(const void *d_packed, const int32_t *d_idx, const int32_t *d_count,
                            int32_t capacity, bc_grid g, void *d_dst, bc_tensor dst,
                            void *stream);

/*
 * Block-sparse convolution with fused epilogue (Section 3.1; every conv layer of a
 * single-stage network, Section 4):
 *   out[block] = act(conv(in)[block] + bias (+ residual[block]))  for active blocks,
 *   out[other] untouched (feature transfer).
 * conv is a cross-correlation with zero padding; act is ReLU when conv->relu.
 * Arithmetic: products of the stored operands accumulated in fp32, bias and
 * residual added in fp32, ReLU, then one round-to-nearest-even to out.dtype.
 *   in, out    same dtype and layout. NHWC: BF16 or F16 (matrix-core path).
 *              NCHW: F32 (fp32 FMA path).
 *   d_w        NHWC: [Cout][kh][kw][Cin] in in.dtype. NCHW: [Cout][Cin][kh][kw] F32.
 *   d_bias     [Cout] fp32 (batch norm folded in, see bc_fold_bn), or NULL.
 *   d_residual shaped and typed like out, or NULL; read only at active blocks.
 *   d_out      must not overlap d_in, d_w or d_residual (BC_ERR_ALIAS).
 * Sizes: out.n = in.n, out.h = (in.h + 2*pad - kh)/stride + 1 (same for w).
 * Supported (else BC_ERR_UNSUPPORTED with the reason in bc_last_error()): stride 1
 * or 2; kh = kw in {1, 3, 5, 7}. NHWC (matrix cores): Cout % 64 == 0; Cin % 8 == 0,
 * or Cin <= 4 with kw <= 7, or Cin < 8 with kw <= 3 (the stem form); input, output
 * and weights each below 2 GiB; the block width must divide 64 or 128 and the block's
 * halo must fit in LDS. NCHW (fp32): output blocks of at most 2048 pixels whose halo
 * tile (one channel) fits in LDS.
 * If d_out is a registered buffer (bc_buffer_register) that is not valid, a sparse
 * call (d_idx non-NULL) returns BC_ERR_UNINITIALIZED; a full call (d_idx = d_count
 * = NULL) makes it valid.
 * Library state used by NHWC calls whose layer splits K over several workgroups (the
 * tile plan depends on the layer's shape and grid only; it splits for few full-frame
 * tiles with a long K, e.g. the stride-32 layers of a ResNet at 2048x1024):
 *  - a split-K workspace of 64 MiB per device (fp32 partial tiles), owned by the
 *    library, allocated by the first such call on the device and never freed or
 *    moved (a captured graph keeps a valid pointer whatever runs later). That first
 *    allocation is refused with BC_ERR_CAPTURE if the stream is capturing a graph:
 *    make one uncaptured call of such a layer first, or use bc_sparse_conv2d_noalloc;
 *  - per-tile arrival counters in a static device array; the last K slice of a tile
 *    resets its counter, so no clearing is needed between calls or graph replays.
 * Both are shared by every call on a device: calls on one device must not overlap
 * in time (use one stream, or order the streams with events). Calls that do not
 * split K use neither. Results never depend on the plan's split: slices are added in
 * a fixed order, so an active block's output bits do not depend on the other blocks.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT,
 * BC_ERR_NOT_DIVISIBLE, BC_ERR_CAPACITY, BC_ERR_ALIAS, BC_ERR_UNINITIALIZED,
 * BC_ERR_UNSUPPORTED, BC_ERR_CAPTURE, BC_ERR_HIP.
 */
bc_status bc_sparse_conv2d(const bc_conv *conv,
                           const void *d_in, bc_tensor in,
                           const void *d_w, const float *d_bias, const void *d_residual,
                           void *d_out, bc_tensor out, bc_grid g,
                           const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                           void *stream);

/*
 * bc_sparse_conv2d for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc. Same
 * arguments, checks, kernels and results (bit for bit) as bc_sparse_conv2d; the only
 * difference is where a layer that splits K keeps its fp32 partial tiles: in a fixed
 * 16 MiB device array of the library (one per device, allocated when the library's
 * code object is loaded on that device and held until the process ends), never in a
 * workspace the call allocates. No call allocates or frees memory.
 * The array holds the partials of any layer whose plan needs at most 16 MiB: every
 * layer of ResNet-18/50 and SwiftNet at 2048x1024 with 128-pixel blocks. Layers whose
 * partials need more (3x3 layers with 512 or more input channels and 513..2048 full-
 * frame tiles of 64x64, e.g. 3x3 512->1024 on a 64x128 map with 8x8 blocks) are
 * refused with BC_ERR_CAPACITY before anything is enqueued.
 * The array and the split counters are shared by every call on a device and keep the
 * last call's contents: calls on one device that overlap in time race (use one
 * stream, or order streams with events). Nothing needs clearing between calls.
 * Errors: those of bc_sparse_conv2d except BC_ERR_CAPTURE; BC_ERR_CAPACITY as above.
 */
bc_status bc_sparse_conv2d_noalloc(const bc_conv *conv,
                                   const void *d_in, bc_tensor in,
                                   const void *d_w, const float *d_bias, const void *d_residual,
                                   void *d_out, bc_tensor out, bc_grid g,
                                   const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                   void *stream);

/* The arguments of one bc_sparse_conv2d call (grid and index aside). */
typedef struct bc_conv_call {
    bc_conv conv;
    const void *d_in;
    bc_tensor in;
    const void *d_w;
    const float *d_bias;
    const void *d_residual;
    void *d_out;
    bc_tensor out;
} bc_conv_call;

/*
 * Two independent convolutions of one frame on the same execution grid and index:
 * the same results, bit for bit, as bc_sparse_conv2d for *a followed by
 * bc_sparse_conv2d for *b (every layer runs on the executed blocks only, Section 3.1).
 * Meant for independent layers of one frame, such as a residual block's shortcut
 * projection and the first convolution of its branch (one input), or a decoder's
 * lateral projection and an encoder layer: when both are NHWC BF16 1x1 layers, b at
 * stride 1, and neither tile plan splits K, both run in one launch, one dependent
 * launch fewer on the frame's chain; any other pair runs as two launches in order.
 *   a, b   each call's arguments, checked as bc_sparse_conv2d checks them; neither
 *          output may overlap any tensor of the other call (BC_ERR_ALIAS).
 * Every check of both calls runs before anything is enqueued.
 * Errors: those of bc_sparse_conv2d; BC_ERR_NULL if a or b is NULL.
 */
bc_status bc_sparse_conv2d_pair(const bc_conv_call *a, const bc_conv_call *b, bc_grid g,
                                const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                void *stream);

/* Pyramid pooling geometry: `levels` levels (1..8); level l averages the input over a
 * rows[l] x cols[l] grid of bins (1 <= rows[l] <= h, 1 <= cols[l] <= w) and projects to
 * cl channels (cl % 8 == 0, 8 <= cl <= 256). */
typedef struct { int32_t levels, cl; int32_t rows[8], cols[8]; } bc_spp_geom;

/*
 * Block-sparse spatial pyramid pooling: the context module of SwiftNet-style
 * segmentation networks on the encoder's last feature, run like every other layer of
 * a single-stage network (Section 4), with the layer result defined as the dense
 * layer on the current input buffer selected into the previous output (Section 3.1):
 *   level l (every pixel, every call): bin (i, j) of the rows[l] x cols[l] grid covers
 *     input rows floor(i h / rows) .. ceil((i+1) h / rows) - 1 (same for columns);
 *     L_l[i][j] = round(ReLU(bias[l] + W[l] . mean of the bin)), W[l] a 1x1 conv
 *     [cl][c], written to d_levels [n][bins][cl] (bins = sum of rows[l] * cols[l],
 *     level by level, raster order);
 *   out[block] = [in, up(L_0), ..., up(L_{levels-1})] on the active blocks, where up()
 *     resamples to h x w bilinearly with pixel centres aligned (output row y samples
 *     level row ((2y + 1) rows - h) / (2h), 0 if negative, neighbours clamped) and
 *     rounds once; out[other] untouched (feature transfer).
 * Because the levels pool the whole map, they read every block of d_in (fresh where
 * blocks ran this frame, transferred elsewhere); the concatenation is written at the
 * active blocks only. Arithmetic in fp32 (sums in a fixed order), RNE to the dtype.
 *   in        NHWC BF16/F16 [n][h][w][c], c % 8 == 0 and c / 8 dividing 256 (c <= 2048).
 *   d_w       [levels][cl][c] in in.dtype (batch norm folded, bc_fold_bn).
 *   d_bias    [levels][cl] fp32, or NULL.
 *   d_levels  caller-owned scratch [n][bins][cl] in in.dtype, rewritten by every call.
 *   out       [n][h][w][c + levels * cl], same dtype and layout; grid blocks of out.
 * Registered-buffer rule as bc_sparse_conv2d. Errors: BC_ERR_NULL, BC_ERR_SHAPE,
 * BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_NOT_DIVISIBLE, BC_ERR_CAPACITY, BC_ERR_ALIAS,
 * BC_ERR_UNINITIALIZED, BC_ERR_UNSUPPORTED, BC_ERR_HIP.
 */
bc_status bc_sparse_spp(const void *d_in, bc_tensor in, const bc_spp_geom *spp,
                        const void *d_w, const float *d_bias, void *d_levels,
                        void *d_out, bc_tensor out, bc_grid g,
                        const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                        void *stream);

/*
 * Block-sparse max pooling (the ResNet stem pooling run block-sparsely), kernel
 * kh x kw, stride, padding with -inf (padded positions never win). Same selection
 * contract, layouts, dtypes and registered-buffer rule as bc_sparse_conv2d; the
 * relu field is ignored. NaN inputs give unspecified results.
 */
bc_status bc_sparse_maxpool2d(const bc_conv *geom, const void *d_in, bc_tensor in,
                              void *d_out, bc_tensor out, bc_grid g,
                              const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                              void *stream);

/*
 * Block-sparse decoder merge (Section 4: the semantic segmentation network is a
 * SwiftNet-style encoder-decoder, whose decoder upsamples a coarse feature map and adds
 * the lateral features of the finer level):
 *   out[block] = act(up2(coarse)[block] (+ skip[block]))  for the active blocks,
 *   out[other] untouched (feature transfer).
 * up2 is bilinear upsampling by two with pixel centres aligned and edges replicated:
 * output row 2i takes 3/4 of coarse row i and 1/4 of row i-1, row 2i+1 takes 3/4 of
 * row i and 1/4 of row i+1 (a row outside the image is replaced by the nearest edge
 * row); columns alike. An output block reads a one-pixel coarse halo from d_coarse as
 * it stands. act is ReLU when relu = 1. Arithmetic fp32, one round-to-nearest-even
 * to out.dtype.
 *   coarse, out  same dtype and layout; out = [n][c][2 coarse.h][2 coarse.w]. NHWC:
 *                BF16 or F16 with c % 8 == 0, out below 2 GiB. NCHW: F32.
 *   d_skip       shaped and typed like out, or NULL; read only at active blocks.
 *   d_out        must not overlap d_coarse, d_skip or the index (BC_ERR_ALIAS).
 * Index, capacity and registered-buffer rules as bc_sparse_conv2d.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_NOT_DIVISIBLE,
 * BC_ERR_CAPACITY, BC_ERR_ALIAS, BC_ERR_UNINITIALIZED, BC_ERR_UNSUPPORTED, BC_ERR_HIP.
 */
bc_status bc_sparse_upsample_add(const void *d_coarse, bc_tensor coarse, const void *d_skip,
                                 void *d_out, bc_tensor out, bc_grid g, int32_t relu,
                                 const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                 void *stream);

/*
 * Host only. Fold inference-mode batch normalisation into the preceding conv:
 * w_out = w * gamma / sqrt(var + eps), b_out = beta + (conv_bias - mean) * gamma /
 * sqrt(var + eps), computed in double and rounded to float. w is [cout][per_out]
 * (per_out = everything after the output channel), conv_bias may be NULL (zero).
 * w_out may equal w (in place). Errors: BC_ERR_NULL, BC_ERR_SHAPE.
 */
bc_status bc_fold_bn(const float *w, int32_t cout, int32_t per_out, const float *conv_bias,
                     const float *gamma, const float *beta, const float *mean,
                     const float *var, float eps, float *w_out, float *b_out);

/*
 * Host only. Repack fp32 OIHW weights [cout][cin][kh][kw] into the NHWC weight layout
 * [cout][kh][kw][cin] of `dtype` (BC_BF16 / BC_F16: round to nearest even;
 * BC_F32: copy). h_out receives cout*kh*kw*cin elements. Errors: BC_ERR_NULL,
 * BC_ERR_SHAPE, BC_ERR_DTYPE.
 */
bc_status bc_repack_weights(const float *w_oihw, int32_t cout, int32_t cin, int32_t kh,
                            int32_t kw, int32_t dtype, void *h_out);

/*
 * Persistent per-layer buffers (Section 3.1: representations throughout the network
 * are stored and reused). A registration wraps caller memory (it does not copy or
 * own it) and tracks whether the buffer holds a complete representation: it
 * starts invalid, becomes valid after a full-frame write, and a sparse write into
 * an invalid buffer is refused (the first frame of a clip is executed
 * completely, Section 4).
 */
typedef struct bc_buffer_s *bc_buffer;

/* Register d_mem with descriptor desc. Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE,
 * BC_ERR_LAYOUT, BC_ERR_ALIAS (overlaps a registered buffer). */
bc_status bc_buffer_register(void *d_mem, bc_tensor desc, bc_buffer *out);
/* Forget a registration (the memory is the caller's). Errors: BC_ERR_NULL. */
bc_status bc_buffer_release(bc_buffer b);
/* Start of a new clip: the next write must be a full one. Errors: BC_ERR_NULL. */
bc_status bc_buffer_invalidate(bc_buffer b);
/* Record a write done by other means: full_mask != 0 makes the buffer valid;
 * full_mask == 0 on an invalid buffer returns BC_ERR_UNINITIALIZED. */
bc_status bc_buffer_mark_written(bc_buffer b, int32_t full_mask);
/* 1 if valid, 0 if not, -1 for a NULL or unknown handle. */
int32_t bc_buffer_is_valid(bc_buffer b);

/* ------------------------------------------------------------------------------
 * Steps around the block-sparse network: execution decisions, frame state,
 * information gain and rewards (Sections 3.3 to 3.5).
 * ------------------------------------------------------------------------------ */

/*
 * Execution decisions sampled from the policy's block probabilities, fused with the
 * index build (Section 3.5: P_t holds p_b in [0, 1] per block; A_t = [a_b] is drawn
 * from it stochastically rather than by a threshold). The paper names no generator;
 * this library uses Philox4x32-10 (Salmon et al., SC 2011): block b (raster id, as in
 * the index) draws the first output word x of counter (b, frame mod 2^32,
 * frame div 2^32, 0) under key (seed mod 2^32, seed div 2^32), u_b = (x >> 8) * 2^-24,
 * and a_b = 1 exactly when u_b < p_b (fp32 compare; a NaN probability gives 0). The
 * same (seed, frame, probabilities) always give the same grid.
 *   d_prob   float32 [n][grid_h][grid_w], device.
 *   d_mask   uint8 [n][grid_h][grid_w], device, written with a_b (0 or 1).
 *   d_idx, d_count, h_count: as bc_build_block_index (ascending ids of a_b = 1).
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE (n, grid <= 0 or more than 2^20 blocks),
 * BC_ERR_CAPACITY, BC_ERR_ALIAS (outputs overlapping each other or d_prob), BC_ERR_HIP.
 */
bc_status bc_sample_execution_grid(const float *d_prob, int32_t n, bc_grid g, uint64_t seed,
                                   uint64_t frame, uint8_t *d_mask, int32_t *d_idx,
                                   int32_t capacity, int32_t *d_count, int32_t *h_count,
                                   void *stream);

/*
 * Frame-state update (Section 3.3: the previous frame state H_{t-1} is an RGB frame
 * whose every block holds the image content of the last executed block there):
 *   d_state[block] = d_frame[block] for the active blocks (a bit copy),
 *   every other element of d_state untouched.
 *   desc     shape/format of both tensors (any dtype, NCHW or NHWC); blocks are
 *            desc.h / grid_h x desc.w / grid_w.
 * d_idx/d_count may both be NULL (every block: the first frame of a clip).
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_NOT_DIVISIBLE,
 * BC_ERR_CAPACITY, BC_ERR_ALIAS (frame and state overlap), BC_ERR_HIP.
 */
bc_status bc_update_frame_state(const void *d_frame, void *d_state, bc_tensor desc, bc_grid g,
                                const int32_t *d_idx, const int32_t *d_count, int32_t capacity,
                                void *stream);

/*
 * Information gain for semantic segmentation (Section 3.4): per output pixel the KL
 * divergence KL(O_t || O_{t-1}) between the class distributions of frame t and frame
 * t-1, O = softmax over classes of the network's per-class scores; per block the
 * maximum over its pixels (Eq. 1):
 *   d_ig[n][gy][gx] = max over pixels p of block (gy, gx) of
 *                     sum_c O_t[c,p] (log O_t[c,p] - log O_{t-1}[c,p]).
 * The class scores are the first `classes` channels of the score maps (the rest, e.g.
 * channels a head pads to a tile multiple, is never read). The maps can be the
 * network's output at any resolution (the blocks are desc.h / grid_h x desc.w / grid_w
 * pixels of it). Arithmetic: fp32 (log-sum-exp with the per-pixel maximum subtracted);
 * a per-pixel value below zero (rounding, the exact KL is >= 0) counts as 0. A block
 * whose scores were copied from frame t-1 (not executed) gets exactly 0.
 *   d_logits, d_prev_logits  frame t and frame t-1, same desc: F32 NCHW
 *            [n][c][h][w], or BF16/F16 NHWC [n][h][w][c] with c % 8 == 0.
 *   classes  1 .. min(c, 32).
 *   d_mask   the frame's execution grid, uint8 [n][grid_h][grid_w] (nonzero = the block
 *            ran), or NULL (every block). A block that did not run gets 0 without its
 *            scores being read (they are frame t-1's own, so the gain is exactly 0): the
 *            caller only needs frame t-1's scores of the executed blocks in
 *            d_prev_logits (e.g. bc_update_frame_state with the index before the frame).
 *   d_ig     float32 [n][grid_h][grid_w], device (written completely).
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE (classes), BC_ERR_DTYPE (NCHW not F32, NHWC F32),
 * BC_ERR_LAYOUT, BC_ERR_NOT_DIVISIBLE, BC_ERR_ALIAS (d_ig overlapping an input),
 * BC_ERR_UNSUPPORTED (classes > 32, NHWC c % 8 != 0, an image's scores >= 2 GiB),
 * BC_ERR_HIP.
 */
bc_status bc_seg_information_gain(const void *d_logits, const void *d_prev_logits,
                                  bc_tensor desc, int32_t classes, bc_grid g,
                                  const uint8_t *d_mask, float *d_ig, void *stream);

/*
 * Input of the policy network (Section 3.3, Eq. 2: S_t = {I_t, H_{t-1}, A_{t-1},
 * O_{t-1}}), assembled at a quarter of the frame resolution, where the segmentation
 * output lives, as 32 channels per pixel:
 *   0-2   I_t averaged over the pixel's 4x4 cell of the frame,
 *   3-5   H_{t-1} (the frame state) averaged the same way,
 *   6 .. 5+classes   softmax over the first `classes` channels of O_{t-1}'s scores,
 *   6+classes        a_b of A_{t-1} for the block the pixel lies in (0 if NULL),
 *   the rest 0.
 * Arithmetic fp32, one round-to-nearest-even to the storage dtype.
 *   d_frame, d_state  [n][h][w][3] NHWC, BF16 or F16, h and w multiples of 4, < 2 GiB.
 *   d_scores          [n][h/4][w/4][c] NHWC, same dtype, c % 8 == 0, 1 <= classes <= min(c, 24).
 *   d_prev_mask       uint8 [n][grid_h][grid_w] or NULL; the grid divides h/4 x w/4.
 *   d_out             [n][h/4][w/4][32] NHWC, same dtype, written completely.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_NOT_DIVISIBLE,
 * BC_ERR_ALIAS (d_out overlapping an input), BC_ERR_UNSUPPORTED, BC_ERR_HIP.
 */
bc_status bc_policy_input(const void *d_frame, const void *d_state, bc_tensor frame,
                          const void *d_scores, bc_tensor scores, int32_t classes,
                          const uint8_t *d_prev_mask, bc_grid g, void *d_out, bc_tensor out,
                          void *stream);

/*
 * Block probabilities P_t of the policy network (Section 3.5: p_b in [0, 1] per block):
 * p_b = 1 / (1 + exp(-logit_b)), logit_b = channel 0 of the head's output map, which
 * has one pixel per block.
 *   d_logits  [n][grid_h][grid_w][c] NHWC, BF16 or F16 (desc.h, desc.w = the grid).
 *   d_prob    float32 [n][grid_h][grid_w], device, written.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_ALIAS, BC_ERR_HIP.
 */
bc_status bc_policy_probabilities(const void *d_logits, bc_tensor logits, float *d_prob,
                                  void *stream);

/* ------------------------------------------------------------------------------
 * Online training of the policy network (Section 4 configuration: RMSprop on the
 * REINFORCE loss of Section 3.5, every 4 frames). Gradient maps are channels-last
 * BF16/F16 like the activations; weight gradients and optimiser state are fp32.
 * ------------------------------------------------------------------------------ */

/*
 * Gradient of the loss L = -sum_b R_b log pi(a_b) (pi(1) = p_b = sigmoid(z_b)) with
 * respect to the head's logits: dL/dz_b = -R_b (a_b - p_b), written to channel 0 of
 * d_grad [n][grid_h][grid_w][c] (desc: the head's output map); other channels 0.
 *   d_reward, d_prob  float32 [n][grid_h][grid_w]; d_mask uint8 (nonzero = executed).
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_ALIAS,
 * BC_ERR_UNSUPPORTED (c % 8 != 0), BC_ERR_HIP.
 */
bc_status bc_policy_logit_grad(const float *d_reward, const uint8_t *d_mask, const float *d_prob,
                               void *d_grad, bc_tensor grad, void *stream);

/*
 * d_out = (d_a + d_b) * [d_y > 0], elementwise in fp32, one round to the dtype; d_b
 * and d_y may be NULL (then omitted). With d_y: the backward pass of a ReLU whose
 * output is d_y; with d_b: two gradients of one tensor added. d_out may equal d_a or
 * d_b. desc: NHWC BF16/F16 with c % 8 == 0 (all four tensors alike).
 * Errors: BC_ERR_NULL, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_ALIAS, BC_ERR_UNSUPPORTED,
 * BC_ERR_HIP.
 */
bc_status bc_grad_combine(const void *d_a, const void *d_b, const void *d_y, bc_tensor desc,
                          void *d_out, void *stream);

/*
 * Input gradient of a convolution (its transposed convolution) over every pixel:
 *   d_grad_in = convT(d_grad_out, d_w) (+ d_accum if not NULL),
 * for a layer with kernel k x k (k = 1 or 3), stride 1 or 2, pad k/2, weights d_w
 * [cout][k][k][cin] in the map dtype. grad_in is the layer's input shape
 * [n][h][w][cin] (cin % 64 == 0, h and w multiples of the stride, and of 8 when
 * above 8), grad_out its output shape [n][h/s][w/s][cout] (cout % 64 == 0). Runs on
 * the matrix-core convolution with flipped, transposed weights (and for stride 2 the
 * output gradient spread onto even pixels) in a library-owned workspace, one per
 * device, used in stream order (calls on different streams of one device race). The
 * workspace grows when a call needs more than it holds, by allocating a larger
 * buffer; earlier buffers are kept until the process ends, so a captured graph never
 * holds a freed pointer. Growth is refused with BC_ERR_CAPTURE while the stream is
 * capturing: a caller that captures makes one eager call at the largest size first.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_ALIAS
 * (d_grad_in overlapping an input), BC_ERR_UNSUPPORTED, BC_ERR_CAPTURE, BC_ERR_HIP.
 */
bc_status bc_conv2d_input_grad(const bc_conv *geom, const void *d_grad_out, bc_tensor grad_out,
                               const void *d_w, const void *d_accum, void *d_grad_in,
                               bc_tensor grad_in, void *stream);

/*
 * Weight and bias gradients of a convolution, ADDED to d_dw and d_db:
 *   d_dw[co][i][j][ci] += sum_p grad_out[p][co] * in[p*s - pad + (i, j)][ci],
 *   d_db[co] += sum_p grad_out[p][co]    (d_db may be NULL).
 * Geometry and shapes as bc_conv2d_input_grad (in: [n][h][w][cin], cin % 8 == 0).
 * fp32 accumulation; partial sums are added with fp32 atomics, so the low bits of a
 * result may differ between runs.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_LAYOUT, BC_ERR_ALIAS,
 * BC_ERR_UNSUPPORTED, BC_ERR_HIP.
 */
bc_status bc_conv2d_weight_grad(const bc_conv *geom, const void *d_in, bc_tensor in,
                                const void *d_grad_out, bc_tensor grad_out, float *d_dw,
                                float *d_db, void *stream);

/*
 * One RMSprop step over `count` fp32 parameters (PyTorch's definition, no momentum):
 *   g = d_grad + weight_decay * w;  v = alpha v + (1 - alpha) g^2;
 *   w = w - lr * g / (sqrt(v) + eps);  d_grad = 0;
 * and, if d_w16 is not NULL, its 16-bit copy (dtype BC_BF16 or BC_F16, round to
 * nearest even) rewritten, e.g. the weights the convolutions read.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE, BC_ERR_DTYPE, BC_ERR_ALIAS, BC_ERR_HIP.
 */
bc_status bc_rmsprop_step(float *d_w, float *d_v, float *d_grad, int64_t count, float lr,
                          float alpha, float eps, float weight_decay, void *d_w16, int32_t dtype,
                          void *stream);

/* One parameter tensor of a multi-tensor RMSprop step: fp32 weights, squared-gradient
 * average and gradient of `count` elements, and an optional 16-bit copy of the weights. */
typedef struct { float *w, *v, *grad; void *w16; int64_t count; } bc_param;

/*
 * bc_rmsprop_step on n tensors (1 <= n <= 64) in one launch, same arithmetic and the
 * same hyper-parameters for all; `params` is a host array read during the call (its
 * pointers and sizes travel in the launch's arguments, nothing is allocated). Every
 * w16 copy has the dtype `dtype`. No two buffers of any tensors may overlap.
 * Errors: BC_ERR_NULL, BC_ERR_SHAPE (n or a count out of range), BC_ERR_DTYPE,
 * BC_ERR_ALIAS, BC_ERR_HIP.
 */
bc_status bc_rmsprop_step_many(const bc_param *params, int32_t n, float lr, float alpha, float eps,
                               float weight_decay, int32_t dtype, void *stream);

/*
 * Block rewards and the policy loss (Section 3.5), per image n of the batch:
 *   C_t = (number of executed blocks) / (grid_h * grid_w);
 *   M_t = (1 - mu) * C_t + mu * M_{t-1}        (moving average of the cost);
 *   R_b = (a_b ? IG_b : -IG_b) + gamma * (a_b ? tau - M_t : -(tau - M_t));
 *   L   = -sum_b R_b * log(a_b ? p_b : 1 - p_b)   (REINFORCE).
 *   d_ig      float32 [n][grid_h][grid_w] (bc_seg_information_gain's output).
 *   d_mask    uint8 [n][grid_h][grid_w], nonzero = executed.
 *   d_prob    float32 [n][grid_h][grid_w] or NULL (then no loss is computed).
 *   d_mavg    float32 [n], device, in: M_{t-1}, out: M_t (the caller's state).
 *   d_reward  float32 [n][grid_h][grid_w], device, written.
 *   d_cost    float32 [n] or NULL: C_t.   d_loss  float32 [n] or NULL: L (needs d_prob).
 * Arithmetic fp32; sums in a fixed order (the result does not depend on scheduling).
 * Errors: BC_ERR_NULL (d_ig, d_mask, d_mavg, d_reward; d_loss without d_prob),
 * BC_ERR_SHAPE, BC_ERR_ALIAS (outputs overlapping each other or an input), BC_ERR_HIP.
 */
bc_status bc_block_rewards(const float *d_ig, const uint8_t *d_mask, const float *d_prob,
                           int32_t n, bc_grid g, float tau, float gamma, float mu, float *d_mavg,
                           float *d_reward, float *d_cost, float *d_loss, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* BC_H */
