// Block-sparse convolution on the CDNA4 matrix cores (channels-last bf16 / fp16).
//
// The layer is an implicit GEMM over the active output pixels:
//   M = active blocks * bh * bw output pixels, N = Cout, K = kh * kw * Cin,
//   Y[m, co] = sum_{i, j, ci} W[co, i, j, ci] * X[pixel(m) * s - pad + (i, j), ci]
// which is the dense layer of Section 3.1 evaluated only on the blocks the
// execution grid selects (Section 3.5). Every row m belongs to one active block,
// so a workgroup tile of BM rows is either a band of R rows of one block (large
// blocks) or P whole blocks (small blocks); in both cases the tile's input is a
// union of P halo patches of HR x HC pixels.
//
// Per K step (one chunk of 32 input channels):
//  * the halo patches of the tile are staged once in LDS, one 64-byte slot per
//    input pixel (zeros outside the image: the layer's own zero padding, which
//    makes halos come from neighbouring blocks of the current input buffer);
//  * for each of the kh*kw taps the 32 x BN weight slice is staged in LDS
//    (double-buffered, the next tap's slice is fetched to registers while the
//    current one is multiplied) and every wave issues 16x16x32 MFMAs whose A
//    fragments are the slots shifted by the tap offset (i * HC + j);
// so each input pixel is fetched from memory once per chunk instead of kh*kw times.
//
// Workgroups are numbered XCD-first: consecutive tiles of one block (which share
// halo rows) and all N tiles of one M tile land on the same XCD and its L2. The grid
// is sized for a full frame; workgroups beyond the device-side active count exit at
// once, so no host round trip is needed and cost follows the active fraction.
//
// Epilogue (fused): fp32 accumulators are transposed through LDS so each lane owns
// 8 consecutive channels of one pixel; bias and residual are added in fp32, ReLU
// applied, the result rounded to the storage format (round to nearest even) and
// written with 16-byte stores straight to the block's position of the persistent
// output buffer. Nothing outside active blocks is read or written.
//
// The stem form handles layers with few input channels (kw * Cin <= 32, e.g. the
// 7x7 RGB stem): K is ordered (kernel row i, then the kw*Cin values of that row,
// which are contiguous in a channels-last row), one MFMA k step per kernel row.
#include <mutex>
#include <type_traits>

#include "bc_internal.h"

namespace bc {
namespace {

typedef short short8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x3 __attribute__((ext_vector_type(3)));

// Raw buffer resource: no swizzle, 32-bit dword data format; loads at offsets beyond
// num_records return zeros instead of faulting.
constexpr int kBufferFlags = 0x00020000;
constexpr int kOutOfRange = 0x7FFFFF00;     // byte offset past every buffer (< 2^31 - 256 bytes)

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, int byte_off)
{
    const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
    return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}

constexpr int kThreads = 256;
constexpr int BK = 32;               // input channels per K step (one MFMA k)
constexpr int PITCH = BK * 2 + 16;   // bytes per LDS slot / weight row (64 data + 16 pad)
constexpr int kMaxAV = 12;           // halo slots per thread quarter: nslot <= 64 * kMaxAV
constexpr int EPITCH = 36;           // floats per epilogue scratch row (32 + 4 pad)
constexpr size_t kMaxLds = 64 * 1024;

// Division by a per-launch constant d: q = umulhi(n, ceil(2^32 / d)), exact whenever
// n * d < 2^32 (all uses here have n, d < 2^14); d = 1 is stored as m = 0.
struct FastDiv {
    uint32_t m;
};

__device__ __forceinline__ int fdiv(int n, FastDiv f)
{
    return f.m ? (int)__umulhi((uint32_t)n, f.m) : n;
}

FastDiv make_fastdiv(int d)
{
    return FastDiv{d == 1 ? 0u : (uint32_t)((((uint64_t)1 << 32) + (uint64_t)d - 1) / (uint64_t)d)};
}

struct MfmaArgs {
    const uint16_t *x, *w, *res;
    const float *bias;
    uint16_t *y;
    const int32_t *idx, *count;
    int hin, win, cin, hout, wout, cout, pad, relu;
    int gh, gw, bh, bw, total_blocks;
    int R, P, HR, HC, nslot, tpb, ntn;  // tiling: patch rows, patches/tile, patch rows/cols,
                                        // LDS slots, M tiles per block, N tiles
    int rowpitch;                       // stem form: elements per LDS halo row
    float *ws;                          // split-K partial sums (pipelined form)
    int x_bytes, w_bytes, y_bytes;      // buffer extents
    FastDiv f_hrhc, f_hc, f_rbw, f_bw;  // divisions by HR*HC, HC, R*bw, bw
    int ksplit, cps;                    // K slices per tile, 32-channel chunks per slice
    int tiles_full;                     // tiles (incl. K slices) of a full frame
    int slots;                          // stem form: workgroups resident on the device
    int xu, gx;                         // XCD grouping of the tile order (xcd_tile), 0 = off
    int grp_lds;                        // pipelined form: LDS bytes of one wave group
};

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

template <bool BF16>
__device__ __forceinline__ float to_f32(uint32_t h)
{
    if constexpr (BF16) return __uint_as_float(h << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values -> two storage values packed in 32 bits (low = first), round to
// nearest even; NaN stays NaN. bf16 uses the gfx950 packed conversion instruction.
template <bool BF16>
__device__ __forceinline__ uint32_t pack_h16(float z0, float z1)
{
    if constexpr (BF16) {
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{z0, z1}, bf16x2));
    } else {
        return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)z0) |
               ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)z1) << 16);
    }
}

// fp32 -> storage format, round to nearest even; NaN stays NaN.
template <bool BF16>
__device__ __forceinline__ uint32_t to_h16(float z)
{
    if constexpr (BF16) {
        const uint32_t u = __float_as_uint(z);
        if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
        return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    } else {
        return __builtin_bit_cast(uint16_t, (_Float16)z);
    }
}

// Blocks of one M tile, loaded once into LDS: patch p of the tile has output origin
// (img, oy0, ox0); img < 0 marks a patch beyond the active count. Thread p < P loads
// the active count and the block id in one round trip (ids are read unconditionally:
// the index holds at least n*gh*gw entries). Returns false if the whole tile is
// inactive (uniform across the workgroup).
struct TileBlocks {
    int img[16], oy0[16], ox0[16];
    int live;
};

__device__ __forceinline__ bool load_tile_blocks(const MfmaArgs &a, int mt, TileBlocks &tb)
{
    const int tid = threadIdx.x;
    if (tid < a.P) {
        const int cnt = a.count ? *a.count : a.total_blocks;
        int k, r0;
        if (a.P == 1) {
            k = mt / a.tpb;
            r0 = (mt - k * a.tpb) * a.R;
        } else {
            k = mt * a.P + tid;
            r0 = 0;
        }
        int img = -1, oy0 = 0, ox0 = 0;
        if (k < a.total_blocks) {
            const int bid = a.idx ? a.idx[k] : k;
            if (k < cnt) {
                img = bid / (a.gh * a.gw);
                const int rem = bid - img * a.gh * a.gw;
                const int gy = rem / a.gw;
                oy0 = gy * a.bh + r0;
                ox0 = (rem - gy * a.gw) * a.bw;
            }
        }
        tb.img[tid] = img;
        tb.oy0[tid] = oy0;
        tb.ox0[tid] = ox0;
        if (tid == 0) tb.live = img >= 0;
    }
    __syncthreads();
    return tb.live != 0;
}

// Fused epilogue: bias + residual + ReLU + rounding, 16-byte stores to block positions.
// prefetch() runs before the main loop: it requests the bias and the residual of every
// output this lane will write, so those round trips overlap the K loop. finish() transposes the fp32 accumulators through LDS (each lane then owns 8
// consecutive channels of one pixel), adds bias and residual, applies ReLU, rounds to
// the storage format and writes with 16-byte buffer stores; rows of inactive patches
// use an out-of-range offset, which the hardware drops. `tid` is the thread's index in
// its group of four waves; a group that is not `live` only takes the barriers.
template <bool BF16, int BM, int BN>
struct Epilogue {
    static constexpr int WM = BM / 2, WN = BN / 2, MI = WM / 16;
    static constexpr int NP = WN / 32, NU = WM / 16;
    int rowoff[NU];            // byte offset of the output pixel of item u (kOutOfRange: none)
    uint4 res[NP][NU];
    uint4 bias[NP][2];         // bias of this lane's 8 output channels per pass (fp32 bits)

    __device__ __forceinline__ void prefetch(const MfmaArgs &a, const TileBlocks &tb, int n0,
                                             int tid = threadIdx.x)
    {
        const int lane = tid & 63, wave = tid >> 6;
        const int wm = wave >> 1, wn = wave & 1;
        // no bias: an empty buffer, every load returns zeros
        const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
            (void *)a.bias, (short)0, a.bias ? a.cout * 4 : 0, kBufferFlags);
#pragma unroll
        for (int np = 0; np < NP; ++np) {
            const int co = n0 + wn * WN + np * 32 + (lane & 3) * 8;
            bias[np][0] = bload(br, co * 4);
            bias[np][1] = bload(br, co * 4 + 16);
        }
        const int rbw = a.R * a.bw;
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int m = wm * WM + (lane >> 2) + 16 * u;
            const int p = fdiv(m, a.f_rbw);
            const int local = m - p * rbw;
            const int pr = fdiv(local, a.f_bw), pc = local - pr * a.bw;
            const int img = tb.img[p];
            rowoff[u] = img >= 0 ? (((img * a.hout + tb.oy0[p] + pr) * a.wout + tb.ox0[p] + pc) *
                                    a.cout) * 2
                                 : kOutOfRange;
        }
        if (a.res) {
            const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
                (void *)a.res, (short)0, a.y_bytes, kBufferFlags);
#pragma unroll
            for (int np = 0; np < NP; ++np) {
                const int co = n0 + wn * WN + np * 32 + (lane & 3) * 8;
#pragma unroll
                for (int u = 0; u < NU; ++u)
                    res[np][u] = bload(rr, rowoff[u] != kOutOfRange ? rowoff[u] + co * 2 : kOutOfRange);
            }
        }
    }

    __device__ __forceinline__ void finish(const MfmaArgs &a, f32x4 (&acc)[BM / 32][BN / 32],
                                           uint8_t *smem, int n0, int tid = threadIdx.x,
                                           bool live = true)
    {
        const int lane = tid & 63, wave = tid >> 6;
        const int wn = wave & 1;
        float *scr = (float *)smem + wave * (WM * EPITCH);
        const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
            (void *)a.y, (short)0, a.y_bytes, kBufferFlags);
#pragma unroll
        for (int np = 0; np < NP; ++np) {
            __syncthreads();
            if (live) {
#pragma unroll
                for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                    for (int nn = 0; nn < 2; ++nn)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            scr[(mi * 16 + 4 * (lane >> 4) + i) * EPITCH + nn * 16 + (lane & 15)] =
                                acc[mi][np * 2 + nn][i];
            }
            __syncthreads();
            if (!live) continue;
            const int cl = wn * WN + np * 32 + (lane & 3) * 8;   // column within the tile
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int row = (lane >> 2) + 16 * u;
                const float4 s0 = *(const float4 *)(scr + row * EPITCH + (lane & 3) * 8);
                const float4 s1 = *(const float4 *)(scr + row * EPITCH + (lane & 3) * 8 + 4);
                const uint4 b0 = bias[np][0], b1 = bias[np][1];
                float z[8] = {s0.x + __uint_as_float(b0.x), s0.y + __uint_as_float(b0.y),
                              s0.z + __uint_as_float(b0.z), s0.w + __uint_as_float(b0.w),
                              s1.x + __uint_as_float(b1.x), s1.y + __uint_as_float(b1.y),
                              s1.z + __uint_as_float(b1.z), s1.w + __uint_as_float(b1.w)};
                if (a.res) {
                    const uint32_t rw[4] = {res[np][u].x, res[np][u].y, res[np][u].z, res[np][u].w};
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        z[2 * t] += to_f32<BF16>(rw[t] & 0xFFFFu);
                        z[2 * t + 1] += to_f32<BF16>(rw[t] >> 16);
                    }
                }
                i32x4 o;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    float z0 = z[2 * t], z1 = z[2 * t + 1];
                    if (a.relu) {
                        z0 = (z0 > 0.f || z0 != z0) ? z0 : 0.f;
                        z1 = (z1 > 0.f || z1 != z1) ? z1 : 0.f;
                    }
                    o[t] = (int)pack_h16<BF16>(z0, z1);
                }
                __builtin_amdgcn_raw_buffer_store_b128(
                    o, yr, rowoff[u] != kOutOfRange ? rowoff[u] + (n0 + cl) * 2 : kOutOfRange, 0, 0);
            }
        }
    }
};

// ------------------------------------------------------------------ general form

template <bool BF16, int BM, int BN, int KS, int S>
__global__ __launch_bounds__(kThreads) void k_conv_mfma(MfmaArgs a)
{
    constexpr int SS = (KS == 1) ? S : 1;  // input-pixel step between adjacent slots
    constexpr int ST = S / SS;             // slot step between adjacent output pixels
    constexpr int KT = KS * KS;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int MI = WM / 16, NI = WN / 16;
    constexpr int BV = BN / 64;            // weight vectors per thread per K step
    extern __shared__ __align__(16) uint8_t smem[];

    __shared__ TileBlocks tb;
    const int mt = blockIdx.x / a.ntn, nt = blockIdx.x - (blockIdx.x / a.ntn) * a.ntn;
    const int n0 = nt * BN;
    if (!load_tile_blocks(a, mt, tb)) return;
    Epilogue<BF16, BM, BN> epi;
    epi.prefetch(a, tb, n0);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int q = tid & 3;                 // 16-byte quarter of a 64-byte slot / weight row
    uint8_t *sA = smem;
    uint8_t *sB = smem + a.nslot * PITCH;

    // Input pixel of each halo slot this thread stages (-1: zero padding / no block).
    const int hrhc = a.HR * a.HC;
    int aoff[kMaxAV];
#pragma unroll
    for (int u = 0; u < kMaxAV; ++u) {
        const int slot = (tid >> 2) + 64 * u;
        aoff[u] = -1;
        if (slot < a.nslot) {
            const int p = slot / hrhc;
            const int r = slot - p * hrhc;
            const int ra = r / a.HC, rb = r - (r / a.HC) * a.HC;
            const int img = tb.img[p];
            if (img >= 0) {
                const int iy = tb.oy0[p] * S - a.pad + ra * SS, ix = tb.ox0[p] * S - a.pad + rb * SS;
                if (iy >= 0 && iy < a.hin && ix >= 0 && ix < a.win)
                    aoff[u] = ((img * a.hin + iy) * a.win + ix) * a.cin;
            }
        }
    }
    // Slot of each A-fragment row at tap (0, 0).
    int abase[MI];
    const int rbw = a.R * a.bw;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int m = wm * WM + mi * 16 + (lane & 15);
        const int p = m / rbw;
        const int local = m - p * rbw;
        const int pr = local / a.bw, pc = local - (local / a.bw) * a.bw;
        abase[mi] = p * hrhc + pr * ST * a.HC + pc * ST;
    }

    const int nchunk = (a.cin + BK - 1) / BK;
    const int ktot = nchunk * KT;
    const size_t wrow = (size_t)KT * a.cin;
    uint4 breg[BV];
    auto load_b = [&](int it) {
        const int c = it / KT, tap = it - (it / KT) * KT;
        const int ci = c * BK + q * 8;
#pragma unroll
        for (int v = 0; v < BV; ++v) {
            const int co = n0 + (tid >> 2) + 64 * v;
            breg[v] = ci < a.cin ? *(const uint4 *)(a.w + co * wrow + (size_t)tap * a.cin + ci)
                                 : make_uint4(0, 0, 0, 0);
        }
    };

    f32x4 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

    load_b(0);
    for (int c = 0; c < nchunk; ++c) {
        __syncthreads();  // every wave is done with the previous chunk's halo
        const int ci = c * BK + q * 8;
        uint4 av[kMaxAV];
#pragma unroll
        for (int u = 0; u < kMaxAV; ++u)
            av[u] = (aoff[u] >= 0 && ci < a.cin) ? *(const uint4 *)(a.x + aoff[u] + ci)
                                                 : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int u = 0; u < kMaxAV; ++u) {
            const int slot = (tid >> 2) + 64 * u;
            if (slot < a.nslot) *(uint4 *)(sA + slot * PITCH + q * 16) = av[u];
        }
        for (int tap = 0; tap < KT; ++tap) {
            const int it = c * KT + tap;
            uint8_t *sb = sB + (it & 1) * BN * PITCH;
#pragma unroll
            for (int v = 0; v < BV; ++v)
                *(uint4 *)(sb + ((tid >> 2) + 64 * v) * PITCH + q * 16) = breg[v];
            __syncthreads();
            if (it + 1 < ktot) load_b(it + 1);
            const int ti = tap / KS, tj = tap - (tap / KS) * KS;
            const int toff = ti * a.HC + tj;
            short8 af[MI], bf[NI];
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                af[mi] = *(const short8 *)(sA + (abase[mi] + toff) * PITCH + (lane >> 4) * 16);
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                bf[ni] = *(const short8 *)(sb + (wn * WN + ni * 16 + (lane & 15)) * PITCH +
                                           (lane >> 4) * 16);
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = mfma<BF16>(af[mi], bf[ni], acc[mi][ni]);
        }
    }
    epi.finish(a, acc, smem, n0);
}

// ------------------------------------------------------------------ pipelined form (1x1, 3x3)
//
// The layers of ResNet backbones (1x1 and 3x3, stride 1 or 2) run here. At the
// active fractions of sparse frames most layers have only a few workgroups per CU,
// so time is set by one workgroup's chain of dependent memory round trips and by the
// per-CU issue rate of its loads and LDS traffic, not by the matrix cores. This form
// therefore
//  * loads the active count and the tile's block ids in one round trip (ids are
//    read unconditionally; the index holds at least n*gh*gw entries);
//  * 1x1: every k step is a new 32-channel chunk; SG chunks (one, or two with 64x64
//    tiles) are staged under one barrier, and halo and weights ride register rings
//    four chunks deep (the data of stage j+D is requested right after stage j is
//    staged to LDS);
//  * 3x3, SG = 1: a chunk is nine k steps (one per tap); the weights of all taps are
//    requested a chunk ahead and staged one tap per barrier, the halo once per chunk;
//  * 3x3, SG = 9: the halo and all nine weight slices of a chunk are staged under one
//    barrier and whole chunks ride a 2-deep register ring (more LDS, fewer barriers:
//    chosen for layers with few tiles, where LDS residency does not matter);
//  * splits K over `ksplit` workgroups for layers with few output tiles: each slice
//    stores its fp32 partial tile, and the last slice to finish (a per-tile counter)
//    adds the partials in fixed slice order 0, 1, ... and runs the epilogue, so the
//    result does not depend on arrival order. The counter is reset by that last
//    workgroup, so no memset is needed between calls (safe under graph replay);
//  * splits K over two groups of four waves inside one workgroup for 1x1 layers with
//    a long K on few tiles (conv_pipe_tile's WGS): eight waves per CU read LDS faster
//    than four where the workgroups do not fill the CUs.
// The summation order over K (chunk by chunk, taps in order) is the same for every
// stage grouping, so the grouping never changes results; the K splits fix their own
// order (slices, then the halves of a wave-group split, added in order).

constexpr int kMaxSplitTiles = 1 << 16;
constexpr int kMaxSplit = 4;        // K slices per tile
__device__ uint32_t g_split_counter[kMaxSplitTiles];   // zero at load, reset after use

// Split-K hand-off: every K slice of a tile stores its fp32 partial (the four waves'
// MI x NI fragments), and the last slice to arrive (per-tile counter) adds all
// partials in slice order 0, 1, ... into `acc` and returns true; the others return
// false and exit. A fragment's four values per lane are one 16-byte access and a
// wave's 64 lanes one contiguous kilobyte. Partials are written through to the
// device-coherent level (the SC1 cache policy of agent-scope atomic stores), all of
// this workgroup's stores are waited for before the per-tile counter is incremented,
// and the last slice reads the others' partials with the same policy, so no cache-wide
// write-back or invalidate is needed. The last slice resets the counter, so no memset
// is needed between calls (safe under graph replay).
constexpr int kCoherentSC1 = 16;            // cache policy: SC1 (device-coherent access)

template <int MI, int NI>
__device__ __forceinline__ bool split_k_handoff(const MfmaArgs &a, f32x4 (&acc)[MI][NI], int tile,
                                                int ks, int *s_last)
{
    constexpr int SLICE = 4 * MI * NI * 64 * 4;     // floats of one slice's partial tile
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.ws + (size_t)tile * a.ksplit * SLICE), (short)0, a.ksplit * SLICE * 4,
        kBufferFlags);
    auto frag_off = [&](int sl, int mi, int ni) {
        return (sl * SLICE + (((wave * MI + mi) * NI + ni) * 64 + lane) * 4) * 4;
    };
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, acc[mi][ni]), pr,
                                                   frag_off(ks, mi, ni), 0, kCoherentSC1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0)
        *s_last = __hip_atomic_fetch_add(&g_split_counter[tile], 1u, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)(a.ksplit - 1);
    __syncthreads();
    if (!*s_last) return false;
    // request every other slice's partial first, then add in slice order 0, 1, ...
    f32x4 part[kMaxSplit][MI][NI];
#pragma unroll
    for (int sl = 0; sl < kMaxSplit; ++sl) {
        if (sl >= a.ksplit || sl == ks) continue;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                part[sl][mi][ni] = __builtin_bit_cast(
                    f32x4, __builtin_amdgcn_raw_buffer_load_b128(pr, frag_off(sl, mi, ni), 0,
                                                                 kCoherentSC1));
    }
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            f32x4 tot = (ks == 0) ? acc[mi][ni] : part[0][mi][ni];
#pragma unroll
            for (int sl = 1; sl < kMaxSplit; ++sl)
                if (sl < a.ksplit) tot += (sl == ks) ? acc[mi][ni] : part[sl][mi][ni];
            acc[mi][ni] = tot;
        }
    if (tid == 0)
        __hip_atomic_store(&g_split_counter[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

// Halo vectors (16 bytes) each thread stages per chunk: the halo of a 64-row tile has at
// most 192 slots at stride 1 and 384 at stride 2 (a 128-row tile: 704). Every vector
// costs a load instruction even when it falls outside the halo, so the bound is kept
// tight per stride.
template <int BM, int KT, int S>
struct PipeShape {
    static constexpr int AU = (KT == 1) ? BM / 64 : (BM == 64 ? (S == 1 ? 3 : 6) : 11);
};

// Ring of compile-time slots: calls f(integral_constant<I>, j + I) for I = 0 .. D-1 while
// j + I < n, so every ring slot is a constant index in the step body it runs.
template <int I, int D>
struct RingSteps {
    template <class F>
    __device__ __forceinline__ static void run(F &f, int j, int n)
    {
        if (j + I < n) {
            f(std::integral_constant<int, I>{}, j + I);
            RingSteps<I + 1, D>::run(f, j, n);
        }
    }
};
template <int D>
struct RingSteps<D, D> {
    template <class F>
    __device__ __forceinline__ static void run(F &, int, int) {}
};

// Runs a ring of D steps over n steps: a loop of whole rings (no exit inside, so the
// loop's back edge only carries the state after the last slot, and the compiler's wait
// counting sees every slot's requests at their true age), then the partial ring.
template <int I, int D>
struct RingAll {
    template <class F>
    __device__ __forceinline__ static void run(F &f, int j)
    {
        f(std::integral_constant<int, I>{}, j + I);
        RingAll<I + 1, D>::run(f, j);
    }
};
template <int D>
struct RingAll<D, D> {
    template <class F>
    __device__ __forceinline__ static void run(F &, int) {}
};

template <int D, class F>
__device__ __forceinline__ void ring_loop(F &f, int n)
{
    int j = 0;
    for (; j + D <= n; j += D) RingAll<0, D>::run(f, j);
    RingSteps<0, D>::run(f, j, n);
}

// SG (stage grouping) sets how much of K one barrier covers: one tap (SG = 1), all KT
// taps of a 32-channel chunk (SG = KT, 3x3 layers), or two chunks (SG = 2, 1x1 layers).
// One workgroup's tile L of the launch grid (the kernels below give it blockIdx.x).
// WGS groups of four waves split the tile's K slice in two contiguous halves (the
// first group takes the first half); each group runs the same number of steps (a
// shorter second half walks zeros at the end), and the second group's partial sums
// are added to the first's through LDS before the epilogue: eight waves per tile raise
// the LDS read rate of the few-tile layers whose workgroups do not fill the CUs.
template <bool BF16, int BM, int BN, int KS, int S, int SG, int WGS = 1>
__device__ __forceinline__ void conv_pipe_tile(const MfmaArgs &a, const int L)
{
    constexpr int SS = (KS == 1) ? S : 1;
    constexpr int ST = S / SS;
    constexpr int KT = KS * KS;
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int MI = WM / 16, NI = WN / 16;
    constexpr int BV = BN / 64;
    constexpr int AU = PipeShape<BM, KT, S>::AU;
    extern __shared__ __align__(16) uint8_t smem[];
    __shared__ TileBlocks tb;
    __shared__ int s_last;

    const int grp = (WGS == 1) ? 0 : (int)(threadIdx.x >> 8);
    const int tid = threadIdx.x & (kThreads - 1), lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1, q = tid & 3;
    // natural tile order L = (mt * ntn + nt) * ksplit + ks: N tile and K slice are known
    // without the active count
    const int ks = L % a.ksplit;
    const int mn = L / a.ksplit;
    const int nt = mn % a.ntn;
    const int mt = mn / a.ntn;
    const int n0 = nt * BN;
    const int nchunk = (a.cin + BK - 1) / BK;
    const int s_lo = ks * a.cps, s_hi = min(nchunk, s_lo + a.cps);
    const int half = (s_hi - s_lo + WGS - 1) / WGS;      // chunks per group (the trip count)
    const int c_lo = s_lo + grp * half;
    const int c_hi = min(s_hi, c_lo + half);
    const int nsteps = (c_hi > c_lo ? c_hi - c_lo : 0) * KT;   // this group's real steps
    const int nstrip = half * KT;                         // steps every group runs

    // Every request is issued unconditionally as a raw buffer load: lanes without data
    // (zero padding, inactive patches, channels past Cin, steps past the slice) use an
    // offset beyond the buffer, for which the hardware returns zeros. The loops below
    // are therefore straight-line code and the compiler can wait for exactly the request
    // a step needs instead of draining every outstanding one. Requests return in issue
    // order, so they are issued in the order they are needed: halo, weights, epilogue.
    if (!load_tile_blocks(a, mt, tb)) return;   // tile beyond the active count (uniform)
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.w, (short)0, a.w_bytes, kBufferFlags);
    const int wq = ((n0 + (tid >> 2)) * KT * a.cin + q * 8) * 2;   // byte offset, tap 0 chunk 0
    auto load_b = [&](int j, uint4 (&r)[BV]) {
        const int c = c_lo + j / KT, tap = j - (j / KT) * KT;
        const bool ok = j < nsteps && c * BK + q * 8 < a.cin;
#pragma unroll
        for (int v = 0; v < BV; ++v)
            r[v] = bload(wr, ok ? wq + (64 * v * KT * a.cin + tap * a.cin + c * BK) * 2 : kOutOfRange);
    };
    static_assert(SG == 1 || (KT > 1 && SG == KT) || (KT == 1 && SG == 2),
                  "stage grouping: one tap, every tap of a chunk, or two 1x1 chunks");
    constexpr int AG = (KT == 1) ? SG : 1;        // halo chunks per stage buffer
    const int hrhc = a.HR * a.HC;
    const int aslot = ((a.nslot + 15) & ~15) * PITCH;
    uint8_t *sA = smem + grp * a.grp_lds;
    uint8_t *sB = sA + 2 * AG * aslot;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.x, (short)0, a.x_bytes, kBufferFlags);

    // halo slot -> byte offset of its input pixel (kOutOfRange: zero padding / inactive patch)
    int aoff[AU];
#pragma unroll
    for (int u = 0; u < AU; ++u) {
        const int slot = (tid >> 2) + 64 * u;
        aoff[u] = kOutOfRange;
        if (slot < a.nslot) {
            const int p = fdiv(slot, a.f_hrhc);
            const int r = slot - p * hrhc;
            const int hy = fdiv(r, a.f_hc), hx = r - hy * a.HC;
            const int img = tb.img[p];
            if (img >= 0) {
                const int iy = tb.oy0[p] * S - a.pad + hy * SS;
                const int ix = tb.ox0[p] * S - a.pad + hx * SS;
                if (iy >= 0 && iy < a.hin && ix >= 0 && ix < a.win)
                    aoff[u] = (((img * a.hin + iy) * a.win + ix) * a.cin + q * 8) * 2;
            }
        }
    }
    auto load_a = [&](int c, uint4 (&r)[AU]) {
        const bool ok = c < c_hi && c * BK + q * 8 < a.cin;
#pragma unroll
        for (int u = 0; u < AU; ++u)
            r[u] = bload(xr, (ok && aoff[u] != kOutOfRange) ? aoff[u] + c * BK * 2 : kOutOfRange);
    };
    auto store_a = [&](uint8_t *sa, const uint4 (&r)[AU]) {
#pragma unroll
        for (int u = 0; u < AU; ++u) {
            const int slot = (tid >> 2) + 64 * u;
            if (slot < a.nslot) *(uint4 *)(sa + slot * PITCH + q * 16) = r[u];
        }
    };
    auto store_b = [&](uint8_t *sb, const uint4 (&r)[BV]) {
#pragma unroll
        for (int v = 0; v < BV; ++v) *(uint4 *)(sb + ((tid >> 2) + 64 * v) * PITCH + q * 16) = r[v];
    };
    int abase[MI];
    const int rbw = a.R * a.bw;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int m = wm * WM + mi * 16 + (lane & 15);
        const int p = fdiv(m, a.f_rbw);
        const int local = m - p * rbw;
        const int pr = fdiv(local, a.f_bw), pc = local - pr * a.bw;
        abase[mi] = (p * hrhc + pr * ST * a.HC + pc * ST) * PITCH + (lane >> 4) * 16;
    }
    const int boff = (wn * WN + (lane & 15)) * PITCH + (lane >> 4) * 16;

    f32x4 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](const uint8_t *sa, const uint8_t *sb, int toff) {
        short8 af[MI], bf[NI];
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) af[mi] = *(const short8 *)(sa + abase[mi] + toff);
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) bf[ni] = *(const short8 *)(sb + boff + ni * 16 * PITCH);
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = mfma<BF16>(af[mi], bf[ni], acc[mi][ni]);
    };

    Epilogue<BF16, BM, BN> epi;
    if constexpr (KT == 1) {
        // every k step is a new chunk; a stage is SG chunks under one barrier, and halo
        // and weights ride a ring of D stages (four chunks in flight)
        constexpr int D = 4 / SG;
        uint4 ra[D][SG][AU];
        uint4 rb[D][SG][BV];
        auto load_stage = [&](int st, uint4 (&xa)[SG][AU], uint4 (&xb)[SG][BV]) {
#pragma unroll
            for (int g = 0; g < SG; ++g) {
                load_a(c_lo + st * SG + g, xa[g]);
                load_b(st * SG + g, xb[g]);
            }
        };
#pragma unroll
        for (int d = 0; d < D; ++d) load_stage(d, ra[d], rb[d]);
        if (grp == 0) epi.prefetch(a, tb, n0, tid);
        auto step = [&](auto dc, int st) {
            constexpr int d = decltype(dc)::value;
            uint8_t *sa = sA + (st & 1) * SG * aslot;
            uint8_t *sb = sB + (st & 1) * SG * BN * PITCH;
#pragma unroll
            for (int g = 0; g < SG; ++g) {
                store_a(sa + g * aslot, ra[d][g]);
                store_b(sb + g * BN * PITCH, rb[d][g]);
            }
            __syncthreads();
            load_stage(st + D, ra[d], rb[d]);
#pragma unroll
            for (int g = 0; g < SG; ++g) compute(sa + g * aslot, sb + g * BN * PITCH, 0);
        };
        ring_loop<D>(step, (nstrip + SG - 1) / SG);
    } else if constexpr (SG == 1) {
        // one chunk = KT steps: the next chunk's weights (all taps) and halo are requested
        // while the current chunk is multiplied
        uint4 ra[AU];
        uint4 rb[KT][BV];
        load_a(c_lo, ra);
#pragma unroll
        for (int t = 0; t < KT; ++t) load_b(t, rb[t]);
        if (grp == 0) epi.prefetch(a, tb, n0, tid);
        const int nch = nstrip / KT;
        for (int cj = 0; cj < nch; ++cj) {
            uint8_t *sa = sA + (cj & 1) * aslot;
            store_a(sa, ra);
#pragma unroll
            for (int t = 0; t < KT; ++t) {
                const int j = cj * KT + t;
                uint8_t *sb = sB + (j & 1) * BN * PITCH;
                store_b(sb, rb[t]);
                __syncthreads();
                load_b(j + KT, rb[t]);
                if (t == 0) load_a(c_lo + cj + 1, ra);
                compute(sa, sb, ((t / KS) * a.HC + (t % KS)) * PITCH);
            }
        }
    } else {
        // a stage is one chunk with every tap: its halo and all KT weight slices are
        // staged under one barrier; chunks ride a 2-deep register ring and an LDS double
        // buffer (sB holds KT slices per buffer)
        constexpr int D = 2;
        const int nch = nstrip / KT;
        uint4 ra[D][AU];
        uint4 rb[D][KT][BV];
        auto load_stage = [&](int cj, uint4 (&xa)[AU], uint4 (&xb)[KT][BV]) {
            load_a(c_lo + cj, xa);
#pragma unroll
            for (int t = 0; t < KT; ++t) load_b(cj * KT + t, xb[t]);
        };
#pragma unroll
        for (int d = 0; d < D; ++d) load_stage(d, ra[d], rb[d]);
        if (grp == 0) epi.prefetch(a, tb, n0, tid);
        auto step = [&](auto dc, int cj) {
            constexpr int d = decltype(dc)::value;
            uint8_t *sa = sA + (cj & 1) * aslot;
            uint8_t *sb = sB + (cj & 1) * KT * BN * PITCH;
            store_a(sa, ra[d]);
#pragma unroll
            for (int t = 0; t < KT; ++t) store_b(sb + t * BN * PITCH, rb[d][t]);
            __syncthreads();
            load_stage(cj + D, ra[d], rb[d]);
#pragma unroll
            for (int t = 0; t < KT; ++t)
                compute(sa, sb + t * BN * PITCH, ((t / KS) * a.HC + (t % KS)) * PITCH);
        };
        ring_loop<D>(step, nch);
    }

    if constexpr (WGS == 2) {
        // the second group's partial sums join the first's (first + second, per element)
        __syncthreads();                  // both groups are done with their stage buffers
        f32x4 *red = (f32x4 *)smem + (wave * MI * NI) * 64 + lane;
        if (grp == 1) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) red[(mi * NI + ni) * 64] = acc[mi][ni];
        }
        __syncthreads();
        if (grp == 0) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = acc[mi][ni] + red[(mi * NI + ni) * 64];
        }
        __syncthreads();                  // the epilogue scratch reuses the same LDS
    }
    if constexpr (BM == 64 && BN == 64 && WGS == 1)
        if (a.ksplit > 1 && !split_k_handoff(a, acc, mt * a.ntn + nt, ks, &s_last)) return;
    epi.finish(a, acc, smem, n0, tid, grp == 0);
}

// Tile order grouped by XCD. Workgroups go to the 8 XCDs in turn (workgroup b to XCD
// b % 8), and each XCD has an L2 of its own. The R = ntn * ksplit workgroups of one M
// tile read the same input rows; in plain order they land on every XCD, and each XCD
// fetches those rows. Grouped, an M tile's workgroups form gx units of xu = R / gx
// consecutive tiles; unit U = mt * gx + part runs on XCD U % 8, so the input rows of an
// M tile are fetched by gx XCDs, and consecutive M tiles (the active ones come first)
// still spread over all XCDs. Returns the natural tile index, or a value past the grid
// for the padding workgroups (their tile is beyond the frame, and they exit).
__device__ __forceinline__ int xcd_tile(const MfmaArgs &a, int b)
{
    if (!a.xu) return b;
    const int j = b >> 3;
    const int U = (b & 7) + 8 * (j / a.xu);
    const int mt = U / a.gx, part = U - mt * a.gx;
    return (mt * a.gx + part) * a.xu + (j - (j / a.xu) * a.xu);
}

template <bool BF16, int BM, int BN, int KS, int S, int SG, int WGS = 1>
__global__ __launch_bounds__(kThreads * WGS) void k_conv_pipe(MfmaArgs a)
{
    conv_pipe_tile<BF16, BM, BN, KS, S, SG, WGS>(a, xcd_tile(a, blockIdx.x));
}

// Two independent 1x1 layers of one frame in one launch (a block's shortcut projection
// and the first convolution of its residual branch read the same input): workgroups
// below grid1 run tiles of the first layer, the rest tiles of the second (stride 1).
// Each tile runs exactly as in its own launch, so results are the same bits. Neither
// layer may split K: both would index the same per-tile counters and partials, which
// one launch of one layer owns.
template <bool BF16, int BN1, int S1, int SG1, int BN2, int SG2>
__global__ __launch_bounds__(kThreads) void k_conv_pipe_pair(MfmaArgs a1, MfmaArgs a2, int grid1)
{
    if ((int)blockIdx.x < grid1)
        conv_pipe_tile<BF16, 64, BN1, 1, S1, SG1>(a1, blockIdx.x);
    else
        conv_pipe_tile<BF16, 64, BN2, 1, 1, SG2>(a2, (int)blockIdx.x - grid1);
}

// ------------------------------------------------------------------ stem form
//
// Layers with few input channels (the RGB stem): Cin <= 4 with kw <= 8, or Cin <= 8 with
// kw <= 4. In LDS every input pixel carries CP = 4 (or 8) channels, zero-padded, so one
// kernel row of one output pixel is a run of kw*CP <= 32 values and one MFMA k step
// covers it: k = j*CP + c for tap column j and channel c (k with j >= kw or c >= Cin
// meets zero weights). A lane's 8 consecutive k are then 16 contiguous bytes of LDS.
// Weights arrive as one contiguous [BN][kh*kw*Cin] run (16-byte buffer loads) and are
// rearranged in LDS into the padded [kh][BN][32] k order.

template <bool BF16, int BM, int BN, int KS, int S, int CP>
__global__ __launch_bounds__(kThreads) void k_conv_mfma_stem(MfmaArgs a)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int MI = WM / 16, NI = WN / 16;
    constexpr int BKP = 40;                  // elements per LDS weight row (32 + 8 pad)
    constexpr int PPK = 8 / CP;              // pixels per 8 consecutive k
    static_assert(BN == 64, "stem form: one 64-channel N tile per workgroup");
    extern __shared__ __align__(16) uint8_t smem[];

    __shared__ TileBlocks tb;
    const int grp = blockIdx.x / a.ntn, nt = blockIdx.x - (blockIdx.x / a.ntn) * a.ntn;
    const int n0 = nt * BN;
    // A workgroup stages the N tile's weights once and computes `per` consecutive M
    // tiles with them, `per` chosen so the active tiles fill at most the resident
    // workgroups. A tile's result does not depend on which workgroup computes it.
    const int cnt = a.count ? *a.count : a.total_blocks;
    const int act = (a.P == 1) ? cnt * a.tpb : (cnt + a.P - 1) / a.P;   // active M tiles
    const int slots = max(1, a.slots);
    const int per = max(1, (act * a.ntn + slots - 1) / slots);
    const int mt0 = grp * per;
    if (mt0 >= act) return;                  // uniform
    load_tile_blocks(a, mt0, tb);            // active: mt0 < act
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int hcp = a.rowpitch;              // pixels per LDS halo row (>= (bw-1)*S + 32/CP)
    const int kwc = KS * a.cin;              // weight values per kernel row
    const int wvals = BN * KS * kwc;         // weights of this N tile
    // LDS: rearranged weights, then the halo and the raw weights (the epilogue's scratch
    // reuses the halo and raw-weight space)
    uint16_t *sB = (uint16_t *)smem;                                 // [KS][BN][BKP]
    uint8_t *sA = smem + KS * BN * BKP * 2;                          // [P][HR][hcp][CP]
    const int a_bytes = ((a.P * a.HR * hcp * CP * 2) + 15) & ~15;
    uint16_t *sW = (uint16_t *)(sA + a_bytes);                       // raw [BN][KS*kwc]

    // raw weights of the N tile: one contiguous run, 16-byte requests
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.w, (short)0, a.w_bytes, kBufferFlags);
    const int wbase = n0 * KS * kwc * 2;
    const int nvec = (wvals * 2 + 15) / 16;
    // every thread's requests (halo values, then raw weights) are issued before any of
    // them is used, so the staging costs one memory round trip instead of one per item
    constexpr int WPT = 6;                   // 16-byte weight vectors per thread per batch
    constexpr int SPT = 6;                   // halo pixels per thread per batch
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.x, (short)0, a.x_bytes, kBufferFlags);
    const int npix = a.P * a.HR * hcp;
    auto halo_batch = [&](int e0, uint16_t (&v)[SPT][CP]) {
#pragma unroll
        for (int u = 0; u < SPT; ++u) {
            const int e = e0 + u * kThreads + tid;
            const int row = fdiv(e, a.f_hc);                  // f_hc holds 1 / hcp here
            const int col = e - row * hcp;
            const int p = min(fdiv(row, a.f_hrhc), a.P - 1);  // f_hrhc holds 1 / HR here
            const int hy = row - p * a.HR;
            const int img = tb.img[p];
            const int iy = tb.oy0[p] * S - a.pad + hy, ix = tb.ox0[p] * S - a.pad + col;
            int off = (e < npix && img >= 0 && col < a.HC && iy >= 0 && iy < a.hin && ix >= 0 &&
                       ix < a.win)
                          ? (((img * a.hin + iy) * a.win + ix) * a.cin) * 2
                          : kOutOfRange;
            asm volatile("" : "+v"(off));
#pragma unroll
            for (int c = 0; c < CP; ++c)
                v[u][c] = c < a.cin ? __builtin_amdgcn_raw_buffer_load_b16(xr, off + 2 * c, 0, 0)
                                    : (uint16_t)0;
        }
    };
    auto halo_store = [&](int e0, const uint16_t (&v)[SPT][CP]) {
#pragma unroll
        for (int u = 0; u < SPT; ++u) {
            const int e = e0 + u * kThreads + tid;
            if (e >= npix) continue;
            if constexpr (CP == 4) {
                *(uint2 *)(sA + (size_t)e * 8) = make_uint2(v[u][0] | ((uint32_t)v[u][1] << 16),
                                                            v[u][2] | ((uint32_t)v[u][3] << 16));
            } else {
                *(uint4 *)(sA + (size_t)e * 16) = make_uint4(
                    v[u][0] | ((uint32_t)v[u][1] << 16), v[u][2] | ((uint32_t)v[u][3] << 16),
                    v[u][4] | ((uint32_t)v[u][5] << 16), v[u][6] | ((uint32_t)v[u][7] << 16));
            }
        }
    };
    // Three channels of 16 bits and an even row width: the two pixels at image x = 2q and
    // 2q + 1 are 12 contiguous bytes at a 4-byte aligned offset, one 12-byte request
    // instead of one 2-byte request per pixel and channel. Pairs cover halo columns
    // -1 .. hcp; columns at or past HC get zeros (as in the per-channel path).
    const bool pairs = CP == 4 && a.cin == 3 && (a.win & 1) == 0;
    const int npr = (hcp + 3) >> 1;          // pairs per halo row
    const int nprs = a.P * a.HR * npr;
    constexpr int PPT = 3;                   // pairs per thread per batch
    auto pair_geom = [&](int e, int &row, int &x, int &c0, int &off) {
        row = e / npr;
        const int k = e - row * npr;
        const int p = min(row / a.HR, a.P - 1);
        const int hy = row - p * a.HR;
        const int img = tb.img[p];
        const int ix0 = tb.ox0[p] * S - a.pad;          // image x of halo column 0
        x = 2 * ((ix0 >> 1) + k);                       // even image x of the pair
        c0 = x - ix0;                                   // its halo column: 2k or 2k - 1
        const int iy = tb.oy0[p] * S - a.pad + hy;
        off = (e < nprs && img >= 0 && iy >= 0 && iy < a.hin && x >= 0 && x < a.win)
                  ? ((img * a.hin + iy) * a.win + x) * 6
                  : kOutOfRange;
    };
    auto pair_batch = [&](int e0, i32x3 (&v)[PPT]) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            int row, x, c0, off;
            pair_geom(e0 + u * kThreads + tid, row, x, c0, off);
            asm volatile("" : "+v"(off));
            v[u] = __builtin_amdgcn_raw_buffer_load_b96(xr, off, 0, 0);
        }
    };
    auto pair_store = [&](int e0, const i32x3 (&v)[PPT]) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = e0 + u * kThreads + tid;
            if (e >= nprs) continue;
            int row, x, c0, off;
            pair_geom(e, row, x, c0, off);
            const uint32_t w0 = (uint32_t)v[u][0], w1 = (uint32_t)v[u][1], w2 = (uint32_t)v[u][2];
            uint8_t *rp = sA + (size_t)row * hcp * 8;
            if (c0 >= 0 && c0 < hcp)
                *(uint2 *)(rp + c0 * 8) = c0 < a.HC ? make_uint2(w0, w1 & 0xFFFFu) : make_uint2(0u, 0u);
            if (c0 + 1 < hcp)
                *(uint2 *)(rp + (c0 + 1) * 8) =
                    c0 + 1 < a.HC ? make_uint2((w1 >> 16) | (w2 << 16), w2 >> 16) : make_uint2(0u, 0u);
        }
    };
    uint16_t hv[SPT][CP];
    i32x3 pv[PPT];
    if (pairs)
        pair_batch(0, pv);
    else
        halo_batch(0, hv);
    for (int v0 = 0; v0 < nvec; v0 += WPT * kThreads) {
        uint4 wv[WPT];
#pragma unroll
        for (int u = 0; u < WPT; ++u) {
            const int v = v0 + u * kThreads + tid;
            wv[u] = bload(wr, v < nvec ? wbase + v * 16 : kOutOfRange);
        }
#pragma unroll
        for (int u = 0; u < WPT; ++u) {
            const int v = v0 + u * kThreads + tid;
            if (v < nvec) *(uint4 *)((uint8_t *)sW + v * 16) = wv[u];
        }
    }
    __syncthreads();
    // rearrange weights: B[i][n][kk] = W[n][i][j][c] with kk = j*CP + c, zero elsewhere
    // (sB is complete after the barrier that follows the first tile's halo)
    {
        const int n = tid >> 2, kq = tid & 3;
        const uint16_t *src = sW + n * KS * kwc;
#pragma unroll
        for (int i = 0; i < KS; ++i) {
            uint32_t w2[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                uint32_t pr = 0;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int kk = kq * 8 + t * 2 + h;
                    const int j = kk / CP, c = kk % CP;
                    const uint32_t val = (j < KS && c < a.cin) ? src[i * kwc + j * a.cin + c] : 0u;
                    pr |= val << (16 * h);
                }
                w2[t] = pr;
            }
            *(uint4 *)(sB + (i * BN + n) * BKP + kq * 8) = make_uint4(w2[0], w2[1], w2[2], w2[3]);
        }
    }

    const int rbw = a.R * a.bw;
    int aoffs[MI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int m = wm * WM + mi * 16 + (lane & 15);
        const int p = fdiv(m, a.f_rbw);
        const int local = m - p * rbw;
        const int pr = fdiv(local, a.f_bw), pc = local - pr * a.bw;
        aoffs[mi] = ((p * a.HR + pr * S) * hcp + pc * S + (lane >> 4) * PPK) * CP * 2;
    }
    for (int t = 0;;) {
        Epilogue<BF16, BM, BN> epi;
        epi.prefetch(a, tb, n0);
        // halo pixels with CP channels each (zeros outside the image, past Cin, in the tail)
        if (pairs) {
            pair_store(0, pv);
            for (int e0 = PPT * kThreads; e0 < nprs; e0 += PPT * kThreads) {
                pair_batch(e0, pv);
                pair_store(e0, pv);
            }
        } else {
            halo_store(0, hv);
            for (int e0 = SPT * kThreads; e0 < npix; e0 += SPT * kThreads) {
                halo_batch(e0, hv);
                halo_store(e0, hv);
            }
        }
        __syncthreads();
        f32x4 acc[MI][NI];
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
        for (int i = 0; i < KS; ++i) {
            short8 af[MI], bf[NI];
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) {
                const uint8_t *src = sA + aoffs[mi] + i * hcp * CP * 2;
                if constexpr (CP == 8 || S % 2 == 0) {
                    af[mi] = *(const short8 *)src;                  // 16-byte aligned
                } else {
                    const uint2 lo = *(const uint2 *)src, hi = *(const uint2 *)(src + 8);
                    af[mi] = __builtin_bit_cast(short8, make_uint4(lo.x, lo.y, hi.x, hi.y));
                }
            }
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
                bf[ni] = *(const short8 *)(sB + (i * BN + wn * WN + ni * 16 + (lane & 15)) * BKP +
                                           (lane >> 4) * 8);
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
#pragma unroll
                for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = mfma<BF16>(af[mi], bf[ni], acc[mi][ni]);
        }
        epi.finish(a, acc, sA, n0);
        if (++t == per || mt0 + t >= act) break;
        // the next tile: its blocks (the barrier inside also keeps the halo stores below
        // behind every wave's epilogue reads of the scratch), then its first halo batch
        load_tile_blocks(a, mt0 + t, tb);
        if (pairs)
            pair_batch(0, pv);
        else
            halo_batch(0, hv);
    }
}

// ------------------------------------------------------------------ planning

enum class Form { General, Stem, Pipe };

struct Plan {
    int BM, BN;
    Form form;
    MfmaArgs a;
    int sg = 1;                // pipelined form: stage grouping (k_conv_pipe's SG)
    int wgs = 1;               // pipelined form: groups of four waves per tile (K halves)
    unsigned tiles;            // output tiles of a full frame (before any K split)
    size_t lds;
    size_t ws_bytes;
    unsigned grid;
};

constexpr size_t kMaxLdsPipe = 159 * 1024;   // 160 KB less room for static shared memory

size_t epi_lds(int BM) { return (size_t)4 * (BM / 2) * EPITCH * sizeof(float); }

// Compute units of the current device (cached per device; 256 if the query fails).
int device_cus()
{
    static int cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cus[dev] <= 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cus[dev] = n;
    }
    return cus[dev];
}
size_t round16(size_t v) { return (v + 15) & ~(size_t)15; }

// LDS of the pipelined form: double buffers of the halo and of the weight slices (SG per
// buffer; 1x1 layers stage SG halo chunks too), or the epilogue scratch if larger.
size_t pipe_lds(int nslot, int BM, int BN, int SG, int KT)
{
    const size_t ag = KT == 1 ? (size_t)SG : 1;
    const size_t main = 2 * ag * round16(nslot) * PITCH + (size_t)2 * SG * BN * PITCH;
    return main > epi_lds(BM) ? main : epi_lds(BM);
}

// Tiling of the output blocks into M tiles of BM rows; false if BM cannot take them.
bool tile_rows(const LayerGeom &g, int BM, MfmaArgs &a)
{
    if (g.bw > BM || BM % g.bw) return false;
    int R = BM / g.bw;
    if (R > g.bh) R = g.bh;
    if (R < g.bh && g.bh % R) return false;
    if (BM % (R * g.bw)) return false;
    const int P = BM / (R * g.bw);
    if (P > 1 && R != g.bh) return false;
    if (P > 16) return false;
    a.R = R;
    a.P = P;
    a.tpb = (P == 1) ? g.bh / R : 1;
    return true;
}

int pipe_au(int BM, int KT, int S) { return KT == 1 ? BM / 64 : (BM == 64 ? (S == 1 ? 3 : 6) : 11); }

bool make_plan(const LayerGeom &g, int BM, int BN, Plan &pl)
{
    MfmaArgs &a = pl.a;
    a.xu = a.gx = 0;
    a.grp_lds = 0;
    pl.wgs = 1;
    if (g.cout % BN) return false;
    if (!tile_rows(g, BM, a)) return false;
    const int KS = g.kh, S = g.stride;
    a.ksplit = 1;
    a.cps = (g.cin + BK - 1) / BK;
    pl.ws_bytes = 0;
    if (g.cin % 8) {
        pl.form = Form::Stem;
        const int CP = g.cin <= 4 ? 4 : 8;
        if (g.cin > 8 || KS * CP > 32 || BN != 64) return false;
        a.HR = (a.R - 1) * S + KS;
        a.HC = (g.bw - 1) * S + KS;
        a.rowpitch = (((g.bw - 1) * S + 32 / CP) + 1) & ~1;   // pixels per LDS halo row, even
        a.nslot = 0;
        const size_t abytes = ((size_t)a.P * a.HR * a.rowpitch * CP * 2 + 15) & ~(size_t)15;
        const size_t staged = abytes + (((size_t)BN * KS * KS * g.cin * 2 + 15) & ~(size_t)15);
        pl.lds = (size_t)KS * BN * 40 * 2 + (staged > epi_lds(BM) ? staged : epi_lds(BM));
        if (pl.lds > kMaxLdsPipe) return false;
        const int per_cu = (int)((160 * 1024) / pl.lds);
        a.slots = device_cus() * (per_cu < 1 ? 1 : per_cu > 4 ? 4 : per_cu);
    } else {
        if (KS == 1) {
            a.HR = a.R;
            a.HC = g.bw;
        } else {
            a.HR = (a.R - 1) * S + KS;
            a.HC = (g.bw - 1) * S + KS;
        }
        a.nslot = a.P * a.HR * a.HC;
        a.rowpitch = 0;
        if (KS == 1 || KS == 3) {
            pl.form = Form::Pipe;
            if (a.nslot > 64 * pipe_au(BM, KS * KS, S)) return false;
            pl.sg = 1;
            pl.lds = pipe_lds(a.nslot, BM, BN, 1, KS * KS);
            if (pl.lds > kMaxLdsPipe) return false;
        } else {
            pl.form = Form::General;
            if (a.nslot > 64 * kMaxAV) return false;
            const size_t main = (size_t)a.nslot * PITCH + (size_t)2 * BN * PITCH;
            pl.lds = main > epi_lds(BM) ? main : epi_lds(BM);
            if (pl.lds > kMaxLds) return false;
        }
    }
    pl.BM = BM;
    pl.BN = BN;
    a.ntn = g.cout / BN;
    const int mt_full = (a.P == 1) ? g.total_blocks * a.tpb : (g.total_blocks + a.P - 1) / a.P;
    pl.tiles = (unsigned)mt_full * a.ntn;
    pl.grid = pl.tiles;
    return true;
}

// Tile choice for the pipelined form (1x1 and 3x3 layers), from a sweep of tile shape
// and K split over every ResNet-50 layer of a 2048x1024 frame with 30 % of the blocks
// active: 64-row tiles are fastest everywhere (at these sizes the kernel is bound by
// latency and occupancy, and 64x64 tiles keep the most workgroups resident); 128-wide N
// tiles pay off for 1x1 layers with Cout a multiple of 128 and blocks of 1024 or more
// pixels (the stride-4 maps), or blocks of 256 pixels (stride 8) with Cout >= 512 (with
// fewer output channels the halved tile count costs more: a same-process A/B of whole
// ResNet-50 frames, 0.6446 -> 0.6330 ms at 30 % active, 0.4699 -> 0.4602 at 10 %);
// splitting K in two pays off when a full frame has at most 256 tiles (the stride-32
// layers) and for 3x3 layers with 512 or more input channels and 513 to 2048 tiles
// (where nine-tap stages do not apply); 1x1 layers with at most 256 tiles split K in
// three from 32 chunks on (ResNet-50's stride-32 2048->512: 0.6410 -> 0.6384 ms at 30 %,
// no cost at 50 or 100 %) and not below (SwiftNet's decoder laterals with 8 and 16
// chunks: 7.3 -> 5.3 and 7.2 -> 6.6 us unsplit); three slices of the nine-tap 3x3
// layers gain at 10-30 % but lose 2 % at 50-100 %, where their workgroups outnumber
// the CUs. 1x1 layers with >= 16 chunks on at most 512 tiles that keep K whole take
// two wave groups per tile (the stride-16 1024 -> 256 layers: 8.6 -> 7.7 us with one
// active block, 9.1 -> 8.4 us with 38; frames -0.7 % at 30 %, +1.5 % with every block).
// Other forms take the largest tile with >= 2048 workgroups on a full frame. The choice
// depends on the layer's shape only, never on the active count, so an active block's
// result does not depend on which other blocks are active.
bool choose_plan(const LayerGeom &g, Plan &best)
{
    if ((g.kh == 1 || g.kh == 3) && g.cin % 8 == 0) {
        const int bpx = g.bh * g.bw;
        const int bn = (g.kh == 1 && g.cout % 128 == 0 && (bpx >= 1024 || (bpx >= 256 && g.cout >= 512)))
                           ? 128 : 64;
        if (make_plan(g, 64, bn, best) || make_plan(g, 64, 64, best)) {
            MfmaArgs &a = best.a;
            const int nchunk = (g.cin + BK - 1) / BK;
            const unsigned tiles = best.grid;
            // split K for few tiles with a long K (3x3: two slices from 8 chunks, four
            // with at most 64 tiles; 1x1: three slices from 32 chunks, shorter 1x1 slices
            // do not pay for the hand-off),
            // and in two for 3x3 layers with at least 512 input channels (sixteen chunks of
            // nine taps per tile otherwise) whose tiles are too many for nine-tap stages
            const bool split = (tiles <= 256 && nchunk >= (g.kh == 1 ? 32 : 8)) ||
                               (g.kh == 3 && nchunk >= 16 && tiles > 512 && tiles <= 2048);
            if (best.BM == 64 && best.BN == 64 && split && tiles <= (unsigned)kMaxSplitTiles) {
                const int ns = g.kh == 1 ? 3 : (tiles <= 64 && nchunk >= 8 ? 4 : 2);
                a.cps = (nchunk + ns - 1) / ns;
                a.ksplit = (nchunk + a.cps - 1) / a.cps;
                best.ws_bytes = (size_t)tiles * a.ksplit * best.BM * best.BN * sizeof(float);
                best.grid = tiles * a.ksplit;
            }
            // Stage grouping (3x3): with at most 512 tiles on a full frame (the stride-16
            // and stride-32 layers: few workgroups, long K) staging all nine taps of a
            // chunk under one barrier is faster; with more tiles the smaller LDS footprint
            // of one tap per barrier keeps more workgroups resident, which wins. A call
            // without an index runs every tile: there nine-tap stages (one workgroup per
            // CU) need the tiles to fit one round, at most 256. SG does not change the
            // summation order, so this choice never changes a result.
            const unsigned sg9_tiles = g.count ? 512u : 256u;
            if (g.kh == 3 && best.BM == 64 && best.BN == 64 && best.tiles <= sg9_tiles && a.cps >= 2) {
                const size_t lds = pipe_lds(a.nslot, best.BM, best.BN, 9, 9);
                if (lds <= kMaxLdsPipe) {
                    best.sg = 9;
                    best.lds = lds;
                }
            }
            // 1x1 layers with 64x64 tiles stage two chunks per barrier (a same-process A/B
            // of full ResNet-50 frames: 0.6642 -> 0.6583 ms; with 64x128 tiles, or four
            // chunks per barrier, the larger footprint costs more than the saved barriers)
            if (g.kh == 1 && best.BM == 64 && best.BN == 64) {
                const size_t lds = pipe_lds(a.nslot, 64, 64, 2, 1);
                if (lds <= kMaxLdsPipe) {
                    best.sg = 2;
                    best.lds = lds;
                }
            }
            // 1x1 layers with a long K on few tiles (stride-16 1024 -> 256): two groups of
            // four waves per tile, each taking half of K; the workgroups do not fill the
            // CUs there, and eight waves per CU read LDS faster than four
            if (g.kh == 1 && best.BM == 64 && best.BN == 64 && best.sg == 2 && a.ksplit == 1 &&
                nchunk >= 16 && tiles <= 512) {
                const size_t main = pipe_lds(a.nslot, 64, 64, 2, 1);
                a.grp_lds = (int)main;
                best.wgs = 2;
                best.lds = 2 * main;
            }
            // 1x1 layers whose M tiles have several workgroups: grouped by XCD (xcd_tile),
            // units of at most 16 workgroups. The tile a workgroup computes, and so the
            // result, does not change; only which XCD computes it.
            best.a.xu = best.a.gx = 0;
            const int R = a.ntn * a.ksplit;
            if (g.kh == 1 && R >= 2) {
                a.gx = (R + 15) / 16;
                while (R % a.gx) ++a.gx;
                a.xu = R / a.gx;
                const unsigned mt_full = best.grid / (unsigned)R;
                const unsigned units = mt_full * (unsigned)a.gx;
                best.grid = ((units + 7) / 8) * 8 * (unsigned)a.xu;
            }
            best.a.tiles_full = (int)best.grid;
            return true;
        }
    }
    static const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
    bool have = false;
    for (const auto &c : cand) {
        Plan p;
        if (!make_plan(g, c[0], c[1], p)) continue;
        if (!have || p.grid > best.grid) best = p;
        have = true;
        if (p.grid >= 2048) {
            best = p;
            break;
        }
    }
    if (have) best.a.tiles_full = (int)best.grid;
    return have;
}

// Split-K partials. A plan splits K only for layers with at most 2048 full-frame tiles
// (two slices) or at most 256 (up to four), so one call needs at most
// 2048 * 2 * 64 * 64 * 4 bytes = 64 MiB (choose_plan; checked again in launch_plan).
constexpr size_t kWorkspaceBytes = (size_t)64 << 20;

// bc_sparse_conv2d: a library-owned workspace of kWorkspaceBytes per device, allocated by
// the first call that splits K and never freed or moved, so a graph that captured a
// split call keeps a valid pointer whatever runs later. hipMalloc is not allowed while
// the stream is capturing: a capturing call that would allocate is refused (a prior
// uncaptured split call on the device, or bc_sparse_conv2d_noalloc, avoids that).
std::mutex g_ws_mu;
void *g_ws_ptr[64];

hipError_t workspace(hipStream_t s, float **out, const char **why)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_ws_mu);
    if (!g_ws_ptr[dev]) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        e = hipStreamIsCapturing(s, &cs);
        if (e != hipSuccess) return e;
        if (cs != hipStreamCaptureStatusNone) {
            *why = "the split-K workspace of this device is not allocated yet and the stream is "
                   "capturing (no allocation during capture): make one uncaptured call that "
                   "splits K first, or use bc_sparse_conv2d_noalloc";
            return hipErrorStreamCaptureUnsupported;
        }
        void *p = nullptr;
        e = hipMalloc(&p, kWorkspaceBytes);
        if (e != hipSuccess) return e;
        g_ws_ptr[dev] = p;
    }
    *out = (float *)g_ws_ptr[dev];
    return hipSuccess;
}

// bc_sparse_conv2d_noalloc: the partials live in a fixed device array instead. In host
// code `scratch` only names the symbol; its device address (one copy per device) comes
// from hipGetSymbolAddress, taken once per device on the first call with that device
// current, and only that address is passed to kernels.
constexpr size_t kScratchBytes = (size_t)16 << 20;
__device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];
std::mutex g_scr_mu;
float *g_scr_ptr[64];

hipError_t scratch_ptr(float **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scr_mu);
    if (!g_scr_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scr_ptr[dev] = (float *)p;
    }
    *out = g_scr_ptr[dev];
    return hipSuccess;
}

// Dynamic LDS each kernel has opted in to: a fixed table (a launch allocates no host
// memory either); the library has a few dozen kernel instantiations.
struct LdsOptIn {
    const void *fn;
    size_t lds;
};
constexpr int kMaxOptIn = 256;
std::mutex g_attr_mu;
LdsOptIn g_attr_lds[kMaxOptIn];
int g_attr_n = 0;

template <typename K>
hipError_t launch_kernel(K kernel, const Plan &p, hipStream_t s)
{
    if (p.lds >= 60 * 1024) {
        // opt in to 60 KB or more of dynamic LDS (gfx950: 160 KB per workgroup, static
        // shared memory included), raised per kernel to the largest size launched so far
        std::lock_guard<std::mutex> lk(g_attr_mu);
        int i = 0;
        while (i < g_attr_n && g_attr_lds[i].fn != (const void *)kernel) ++i;
        if (i == g_attr_n) {
            if (g_attr_n == kMaxOptIn) return hipErrorOutOfMemory;
            g_attr_lds[g_attr_n++] = LdsOptIn{(const void *)kernel, 0};
        }
        if (g_attr_lds[i].lds < p.lds) {
            const hipError_t e = hipFuncSetAttribute(
                (const void *)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds);
            if (e != hipSuccess) return e;
            g_attr_lds[i].lds = p.lds;
        }
    }
    hipLaunchKernelGGL(kernel, dim3(p.grid), dim3(kThreads * p.wgs), p.lds, s, p.a);
    return hipSuccess;
}

template <bool BF16, int BM, int BN, int KS, int S>
hipError_t launch_one(const Plan &p, hipStream_t s)
{
    if (p.form == Form::Stem) {
        if constexpr (BN == 64) {
            if (p.a.cin <= 4) return launch_kernel(k_conv_mfma_stem<BF16, BM, BN, KS, S, 4>, p, s);
            else if constexpr (KS <= 4) return launch_kernel(k_conv_mfma_stem<BF16, BM, BN, KS, S, 8>, p, s);
        }
    } else if (p.form == Form::Pipe) {
        if constexpr (KS == 1 || KS == 3) {
            // all-tap stages exist for the 64x64 tiles the planner gives them to
                if constexpr (BM == 64 && BN == 64 && KS == 3)
                if (p.sg == 9) return launch_kernel(k_conv_pipe<BF16, BM, BN, KS, S, 9>, p, s);
            if constexpr (BM == 64 && BN == 64 && KS == 1) {
                if (p.sg == 2 && p.wgs == 2) return launch_kernel(k_conv_pipe<BF16, BM, BN, KS, S, 2, 2>, p, s);
                if (p.sg == 2) return launch_kernel(k_conv_pipe<BF16, BM, BN, KS, S, 2>, p, s);
            }
            if (p.sg == 1) return launch_kernel(k_conv_pipe<BF16, BM, BN, KS, S, 1>, p, s);
        }
    } else {
        return launch_kernel(k_conv_mfma<BF16, BM, BN, KS, S>, p, s);
    }
    return hipErrorInvalidValue;   // no kernel for this plan
}

template <bool BF16, int KS, int S>
hipError_t launch_tiles(const Plan &p, hipStream_t s)
{
    if (p.BM == 128 && p.BN == 128) return launch_one<BF16, 128, 128, KS, S>(p, s);
    if (p.BM == 128) return launch_one<BF16, 128, 64, KS, S>(p, s);
    if (p.BN == 128) return launch_one<BF16, 64, 128, KS, S>(p, s);
    return launch_one<BF16, 64, 64, KS, S>(p, s);
}

template <bool BF16>
hipError_t launch_geom(const Plan &p, int ks, int stride, hipStream_t s)
{
    if (ks == 1) return stride == 1 ? launch_tiles<BF16, 1, 1>(p, s) : launch_tiles<BF16, 1, 2>(p, s);
    if (ks == 3) return stride == 1 ? launch_tiles<BF16, 3, 1>(p, s) : launch_tiles<BF16, 3, 2>(p, s);
    if (ks == 5) return stride == 1 ? launch_tiles<BF16, 5, 1>(p, s) : launch_tiles<BF16, 5, 2>(p, s);
    return stride == 1 ? launch_tiles<BF16, 7, 1>(p, s) : launch_tiles<BF16, 7, 2>(p, s);
}

}  // namespace

bool conv_nhwc_mfma_supported(const LayerGeom &g, const char **why)
{
    if (g.kh != g.kw || (g.kh != 1 && g.kh != 3 && g.kh != 5 && g.kh != 7)) {
        *why = "matrix-core path: kernel must be square with edge 1, 3, 5 or 7";
        return false;
    }
    if (g.stride != 1 && g.stride != 2) {
        *why = "matrix-core path: stride must be 1 or 2";
        return false;
    }
    if (g.cout % 64) {
        *why = "matrix-core path: Cout must be a multiple of 64";
        return false;
    }
    if (g.cin % 8 && !(g.cin <= 4 && g.kw <= 7) && !(g.cin < 8 && g.kw <= 3)) {
        *why = "matrix-core path: Cin must be a multiple of 8, or Cin <= 4 with a kernel edge "
               "<= 7, or Cin < 8 with a kernel edge <= 3 (stem form)";
        return false;
    }
    if (2.0 * g.n * g.hin * g.win * g.cin >= 2147483392.0 ||
        2.0 * g.n * g.hout * g.wout * g.cout >= 2147483392.0 ||
        2.0 * g.cout * g.kh * g.kw * g.cin >= 2147483392.0) {
        *why = "matrix-core path: input, output or weight tensor of 2 GiB or more";
        return false;
    }
    Plan p;
    if (!choose_plan(g, p)) {
        *why = "matrix-core path: no tile shape fits this block size (block width must divide "
               "64 or 128 and the halo must fit in LDS)";
        return false;
    }
    return true;
}

namespace {

// The plan of one channels-last layer with its arguments filled in (no launch).
void fill_plan(const uint16_t *x, const uint16_t *w, const float *bias, const uint16_t *res,
               uint16_t *y, int relu, const LayerGeom &g, Plan &p)
{
    choose_plan(g, p);
    MfmaArgs &a = p.a;
    a.x = x; a.w = w; a.bias = bias; a.res = res; a.y = y;
    a.idx = g.idx; a.count = g.count;
    a.hin = g.hin; a.win = g.win; a.cin = g.cin;
    a.hout = g.hout; a.wout = g.wout; a.cout = g.cout;
    a.pad = g.pad; a.relu = relu;
    a.gh = g.gh; a.gw = g.gw; a.bh = g.bh; a.bw = g.bw; a.total_blocks = g.total_blocks;
    a.ws = nullptr;
    a.x_bytes = (int)((size_t)g.n * g.hin * g.win * g.cin * 2);
    a.w_bytes = (int)((size_t)g.cout * g.kh * g.kw * g.cin * 2);
    a.y_bytes = (int)((size_t)g.n * g.hout * g.wout * g.cout * 2);
    if (p.form == Form::Stem) {            // stem form: divisions by the halo row pitch and HR
        a.f_hc = make_fastdiv(a.rowpitch);
        a.f_hrhc = make_fastdiv(a.HR);
    } else {
        a.f_hrhc = make_fastdiv(a.HR * a.HC > 0 ? a.HR * a.HC : 1);
        a.f_hc = make_fastdiv(a.HC > 0 ? a.HC : 1);
    }
    a.f_rbw = make_fastdiv(a.R * g.bw);
    a.f_bw = make_fastdiv(g.bw);
}

// Where a split plan keeps its partials: the library-owned workspace, or the fixed
// `scratch` array (bc_sparse_conv2d_noalloc).
enum class Partials { Workspace, Scratch };

hipError_t launch_plan(Plan &p, Half16 fmt, const LayerGeom &g, hipStream_t s, const char **why,
                       Partials where = Partials::Workspace)
{
    if (p.grid == 0) return hipSuccess;
    if (p.ws_bytes) {
        const size_t cap = where == Partials::Scratch ? kScratchBytes : kWorkspaceBytes;
        if (p.ws_bytes > cap) {
            *why = "split-K partials larger than the buffer that holds them";
            return hipErrorInvalidValue;
        }
        const hipError_t e = where == Partials::Scratch ? scratch_ptr(&p.a.ws)
                                                        : workspace(s, &p.a.ws, why);
        if (e != hipSuccess) return e;
    }
    const hipError_t e = fmt == Half16::BF16 ? launch_geom<true>(p, g.kh, g.stride, s)
                                             : launch_geom<false>(p, g.kh, g.stride, s);
    if (e != hipSuccess) return e;
    return hipGetLastError();
}

// The (tile width, stage grouping) variants of 64-row 1x1 pipelined plans: 0 = 64 wide,
// two chunks per barrier; 1 = 128 wide, one chunk; -1 = another form.
int pair_variant(const Plan &p)
{
    if (p.form != Form::Pipe || p.BM != 64 || p.a.ksplit != 1 || p.wgs != 1) return -1;
    if (p.BN == 64 && p.sg == 2) return 0;
    if (p.BN == 128 && p.sg == 1) return 1;
    return -1;
}

template <int BN1, int S1, int SG1>
hipError_t launch_pair_second(const Plan &p1, const Plan &p2, int v2, hipStream_t s)
{
    const size_t lds = p1.lds > p2.lds ? p1.lds : p2.lds;
    const unsigned grid = p1.grid + p2.grid;
    if (v2 == 0)
        hipLaunchKernelGGL((k_conv_pipe_pair<true, BN1, S1, SG1, 64, 2>), dim3(grid),
                           dim3(kThreads), lds, s, p1.a, p2.a, (int)p1.grid);
    else
        hipLaunchKernelGGL((k_conv_pipe_pair<true, BN1, S1, SG1, 128, 1>), dim3(grid),
                           dim3(kThreads), lds, s, p1.a, p2.a, (int)p1.grid);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_nhwc_mfma(const uint16_t *x, const uint16_t *w, const float *bias,
                                 const uint16_t *res, uint16_t *y, int relu, Half16 fmt,
                                 const LayerGeom &g, hipStream_t s, const char **why)
{
    if (!conv_nhwc_mfma_supported(g, why)) return hipErrorInvalidValue;
    Plan p;
    fill_plan(x, w, bias, res, y, relu, g, p);
    return launch_plan(p, fmt, g, s, why);
}

size_t conv_nhwc_split_bytes(const LayerGeom &g)
{
    Plan p;
    return choose_plan(g, p) ? p.ws_bytes : 0;
}

size_t conv_nhwc_scratch_bytes() { return kScratchBytes; }

hipError_t launch_conv_nhwc_mfma_noalloc(const uint16_t *x, const uint16_t *w, const float *bias,
                                         const uint16_t *res, uint16_t *y, int relu, Half16 fmt,
                                         const LayerGeom &g, hipStream_t s, const char **why)
{
    if (!conv_nhwc_mfma_supported(g, why)) return hipErrorInvalidValue;
    Plan p;
    fill_plan(x, w, bias, res, y, relu, g, p);
    return launch_plan(p, fmt, g, s, why, Partials::Scratch);
}

hipError_t launch_conv_pair_nhwc_mfma(const ConvCall &c1, const ConvCall &c2, Half16 fmt,
                                      hipStream_t s, const char **why)
{
    if (!conv_nhwc_mfma_supported(c1.g, why) || !conv_nhwc_mfma_supported(c2.g, why))
        return hipErrorInvalidValue;
    Plan p1, p2;
    fill_plan(c1.x, c1.w, c1.bias, c1.res, c1.y, c1.relu, c1.g, p1);
    fill_plan(c2.x, c2.w, c2.bias, c2.res, c2.y, c2.relu, c2.g, p2);
    const int v1 = pair_variant(p1), v2 = pair_variant(p2);
    for (Plan *p : {&p1, &p2})                  // the paired launch keeps the plain tile order
        if (p->a.xu) {
            p->a.xu = p->a.gx = 0;
            p->grid = p->tiles * (unsigned)p->a.ksplit;
        }
    if (fmt == Half16::BF16 && c1.g.kh == 1 && c2.g.kh == 1 && c2.g.stride == 1 && v1 >= 0 &&
        v2 >= 0 && p1.grid > 0 && p2.grid > 0 && (size_t)p1.grid + p2.grid < (1u << 31) &&
        p1.lds < 60 * 1024 && p2.lds < 60 * 1024) {   // no dynamic-LDS opt-in needed
        if (c1.g.stride == 1)
            return v1 == 0 ? launch_pair_second<64, 1, 2>(p1, p2, v2, s)
                           : launch_pair_second<128, 1, 1>(p1, p2, v2, s);
        return v1 == 0 ? launch_pair_second<64, 2, 2>(p1, p2, v2, s)
                       : launch_pair_second<128, 2, 1>(p1, p2, v2, s);
    }
    // any other pair: one launch per layer, in order
    hipError_t e = launch_plan(p1, fmt, c1.g, s, why);
    if (e != hipSuccess) return e;
    return launch_plan(p2, fmt, c2.g, s, why);
}

}  // namespace bc
