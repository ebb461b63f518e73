// Steps around the block-sparse network (Sections 3.3 to 3.5): execution decisions
// sampled from the policy's block probabilities and compacted into the active-block
// index in one pass, the frame-state update, the information gain of semantic
// segmentation (per-pixel KL divergence, max-pooled per block, Eq. 1) and the block
// rewards with the REINFORCE loss.
//
// All of these are small or streaming kernels: the sampling and the rewards touch one
// value per block, the frame state copies the executed blocks of the RGB frame, and
// the information gain streams the class scores of two score maps once (HBM bound).
#include "bc_internal.h"
#include "compact.h"

namespace bc {
namespace {

// ---------------------------------------------------------------- Philox4x32-10
//
// Counter-based generator of Salmon, Moraes, Dror and Shaw (SC 2011): ten rounds of
// two 32x32 -> 64-bit multiplications (constants 0xD2511F53, 0xCD9E8D57) that mix the
// four counter words, with the two key words added in and bumped by the Weyl
// constants (0x9E3779B9, 0xBB67AE85) between rounds. Only the first output word is
// used here.
__device__ __forceinline__ uint32_t philox_word0(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
        const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c0;
}

// ---------------------------------------------------------------- sampling + index

// One workgroup walks the grid in rounds of 1024 blocks: each thread draws its block's
// decision and writes it to the mask, and the stable ballot compaction of compact.h
// writes the executed ids in ascending order (no sort).
__global__ __launch_bounds__(kCompactThreads) void k_sample_index(
    const float *__restrict__ prob, int total, uint32_t f0, uint32_t f1, uint32_t s0,
    uint32_t s1, uint8_t *__restrict__ mask, int32_t *__restrict__ idx,
    int32_t *__restrict__ count)
{
    __shared__ int wave_total[kCompactWaves];
    int running = 0;
    for (int base = 0; base < total; base += kCompactThreads) {
        const int i = base + (int)threadIdx.x;
        bool act = false;
        if (i < total) {
            const uint32_t x = philox_word0((uint32_t)i, f0, f1, 0u, s0, s1);
            const float u = (float)(x >> 8) * 0x1p-24f;   // exact: 24-bit integer * 2^-24
            act = u < prob[i];                            // false for a NaN probability
            mask[i] = act ? 1 : 0;
        }
        running += compact_round(act, i, idx, running, wave_total);
    }
    if (threadIdx.x == 0) *count = running;
}

// ---------------------------------------------------------------- frame state

constexpr int kCopyThreads = 256;
constexpr int kCopyVecPerThread = 4;
constexpr int kCopyVecPerWG = kCopyThreads * kCopyVecPerThread;
constexpr int kBufferFlags = 0x00020000;     // raw buffer, dword format
constexpr int kOutOfRange = 0x7FFFFF00;      // loads return 0, stores are dropped
typedef int i32x4 __attribute__((ext_vector_type(4)));

struct CopyGeom {
    int gh, gw, bh, bw, total_blocks;
    int rows;          // rows of 16-byte vectors per block: bh (NHWC) or c * bh (NCHW)
    int rowv;          // vectors per row
    int pitch;         // vectors between image rows
    int plane;         // vectors between channel planes (NCHW), 0 for NHWC
    long long img;     // vectors per image
    int colv;          // vectors from one block column to the next (bw * c or bw elements)
    int span_bytes;    // byte extent of one block's footprint from its first vector
};

// A block of the frame is `rows` runs of `rowv` 16-byte vectors at the same positions
// in frame and state. A workgroup copies one chunk of kCopyVecPerWG vectors of one
// block; loads and stores are raw buffer accesses whose offsets past the block's
// footprint read zero and are dropped, so the ragged end of a chunk needs no branch
// and every load is in flight before the first store.
__global__ __launch_bounds__(kCopyThreads) void k_frame_state16(
    const uint4 *__restrict__ frame, uint4 *__restrict__ state, CopyGeom g, int chunks,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ count)
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
    const long long origin = img * g.img + (long long)gy * g.bh * g.pitch + (long long)gx * g.colv;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(frame + origin), (short)0, g.span_bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(state + origin), (short)0, g.span_bytes, kBufferFlags);
    const int nv = g.rows * g.rowv;
    int off[kCopyVecPerThread];
    __attribute__((ext_vector_type(4))) int val[kCopyVecPerThread];
#pragma unroll
    for (int u = 0; u < kCopyVecPerThread; ++u) {
        const int v = chunk * kCopyVecPerWG + u * kCopyThreads + threadIdx.x;
        const int r = v / g.rowv;
        const int t = v - r * g.rowv;
        int ro;
        if (g.plane) {
            const int c = r / g.bh;
            ro = c * g.plane + (r - c * g.bh) * g.pitch;
        } else {
            ro = r * g.pitch;
        }
        off[u] = v < nv ? (ro + t) * 16 : kOutOfRange;
        val[u] = __builtin_amdgcn_raw_buffer_load_b128(rs, off[u], 0, 0);
    }
#pragma unroll
    for (int u = 0; u < kCopyVecPerThread; ++u)
        __builtin_amdgcn_raw_buffer_store_b128(val[u], rd, off[u], 0, 0);
}

// Element-wise fallback (rows not a multiple of 16 bytes): one thread per element.
template <typename E>
__global__ __launch_bounds__(kCopyThreads) void k_frame_state_elem(
    const E *__restrict__ frame, E *__restrict__ state, int n, int c, int h, int w, int gh,
    int gw, int nhwc, const int32_t *__restrict__ idx, const int32_t *__restrict__ count,
    int per_block)
{
    const int total = n * gh * gw;
    const int cnt = count ? *count : total;
    const int bh = h / gh, bw = w / gw;
    for (long long e = blockIdx.x * (long long)kCopyThreads + threadIdx.x;
         e < (long long)cnt * per_block; e += (long long)gridDim.x * kCopyThreads) {
        const int k = (int)(e / per_block);
        int rem = (int)(e - (long long)k * per_block);
        const int bid = idx ? idx[k] : k;
        const int img = bid / (gh * gw);
        const int r2 = bid - img * gh * gw;
        const int gy = r2 / gw, gx = r2 - gy * gw;
        int ch, y, x;
        if (nhwc) {            // element order within the block: row, column, channel
            ch = rem % c;
            rem /= c;
            x = rem % bw;
            y = rem / bw;
        } else {               // channel, row, column
            x = rem % bw;
            rem /= bw;
            y = rem % bh;
            ch = rem / bh;
        }
        const long long yy = (long long)gy * bh + y, xx = (long long)gx * bw + x;
        const long long o = nhwc ? (((long long)img * h + yy) * w + xx) * c + ch
                                 : (((long long)img * c + ch) * h + yy) * w + xx;
        state[o] = frame[o];
    }
}

// ---------------------------------------------------------------- information gain

constexpr int kIgThreads = 256;
constexpr int kIgPixPerWG = 1024;

__global__ void k_fill_zero(float *__restrict__ p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

template <bool BF16>
__device__ __forceinline__ float h16_to_f32(uint32_t h)
{
    if constexpr (BF16) return __uint_as_float(h << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// KL(p || q) of one pixel from its first C class scores a (frame t) and b (frame t-1),
// p = softmax(a), q = softmax(b):
//   sum_c e^(a_c - Ma) (a_c - b_c) / Sa - (Ma + log Sa) + (Mb + log Sb),
// Ma, Mb = maxima, Sa, Sb = sums of e^(x - max). Entries past C are ignored.
template <int CMAX>
__device__ __forceinline__ float pixel_kl(const float (&a)[CMAX], const float (&b)[CMAX], int C)
{
    float ml = -__builtin_inff(), mm = -__builtin_inff();
#pragma unroll
    for (int c = 0; c < CMAX; ++c) {
        if (c < C) {
            ml = fmaxf(ml, a[c]);
            mm = fmaxf(mm, b[c]);
        }
    }
    float sl = 0.f, sm = 0.f, t = 0.f;
#pragma unroll
    for (int c = 0; c < CMAX; ++c) {
        if (c < C) {
            const float ea = __expf(a[c] - ml);
            sl += ea;
            t += ea * (a[c] - b[c]);
            sm += __expf(b[c] - mm);
        }
    }
    return t / sl - (ml + __logf(sl)) + (mm + __logf(sm));
}

struct IgGeom {
    int classes;       // class scores per pixel (the first `classes` channels)
    int c;             // channels of the score tensor (>= classes)
    int h, w, gh, gw;
    int rows, strips;  // image rows per workgroup, workgroups per block
    int bytes;         // one image's scores in bytes (< 2 GiB)
    const uint8_t *mask;   // execution grid [n][gh][gw] or null (every block)
};

// Which block and which rows of it a workgroup covers.
struct IgPart {
    int blk, img, gx, y0, npix, bw;
};

__device__ __forceinline__ IgPart ig_part(const IgGeom &g)
{
    IgPart q;
    q.blk = blockIdx.x / g.strips;
    const int strip = blockIdx.x - q.blk * g.strips;
    q.img = q.blk / (g.gh * g.gw);
    const int rem = q.blk - q.img * g.gh * g.gw;
    const int gy = rem / g.gw;
    q.gx = rem - gy * g.gw;
    const int bh = g.h / g.gh;
    q.bw = g.w / g.gw;
    q.y0 = gy * bh + strip * g.rows;
    q.npix = min(g.rows, gy * bh + bh - q.y0) * q.bw;
    return q;
}

// Workgroup maximum (butterfly within each wave, then across the waves) into the
// block's slot by an integer atomic max: the values are >= 0, whose IEEE bit patterns
// order like the numbers, and the slot starts at +0.
__device__ __forceinline__ void block_max_out(float best, float *wave_max, float *slot, bool whole)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) best = fmaxf(best, __shfl_xor(best, o));
    if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = best;
    __syncthreads();
    if (threadIdx.x == 0) {
        float m = wave_max[0];
#pragma unroll
        for (int i = 1; i < kIgThreads / 64; ++i) m = fmaxf(m, wave_max[i]);
        // one workgroup per block: the value itself; else the maximum over the block's
        // workgroups (non-negative floats order like their bit patterns)
        if (whole)
            *slot = m;
        else
            atomicMax((unsigned int *)slot, __float_as_uint(m));
    }
}

// Channels first, fp32: one workgroup covers `rows` image rows of one block (about
// kIgPixPerWG pixels, or a quarter of that); per pixel all 2*classes scores are
// requested at once (raw buffer loads, classes past the count return zero and are left
// out of every sum).
template <int CMAX>
__global__ __launch_bounds__(kIgThreads) void k_seg_kl_blockmax(
    const float *__restrict__ lt, const float *__restrict__ lp, IgGeom g, float *__restrict__ ig)
{
    __shared__ float wave_max[kIgThreads / 64];
    const IgPart q = ig_part(g);
    if (g.mask && !g.mask[q.blk]) {   // not executed: its scores were copied, the gain is 0
        if (g.strips == 1 && threadIdx.x == 0) ig[q.blk] = 0.f;
        return;
    }
    const size_t plane = (size_t)g.h * g.w;
    const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(lt + (size_t)q.img * g.c * plane), (short)0, g.bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(lp + (size_t)q.img * g.c * plane), (short)0, g.bytes, kBufferFlags);
    float best = 0.f;
    for (int p = threadIdx.x; p < q.npix; p += kIgThreads) {
        const int y = q.y0 + p / q.bw, x = q.gx * q.bw + p % q.bw;
        const int pix = (y * g.w + x) * 4;
        float a[CMAX], b[CMAX];
#pragma unroll
        for (int c = 0; c < CMAX; ++c) {
            const int o = c < g.classes ? pix + c * (int)plane * 4 : kOutOfRange;
            a[c] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rt, o, 0, 0));
            b[c] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rp, o, 0, 0));
        }
        const float kl = pixel_kl<CMAX>(a, b, g.classes);
        best = kl > best ? kl : best;
    }
    block_max_out(best, wave_max, &ig[q.blk], g.strips == 1);
}

// Channels last, bf16/fp16 (c % 8 == 0): per pixel the CV 16-byte vectors that hold the
// class scores (8 channels each, CV = ceil(classes / 8)) of both maps; a thread requests
// those of kIgUnroll pixels before using any (pixels past the range read zeros and are
// left out); arithmetic in fp32 as above.
constexpr int kIgUnroll = 4;
template <bool BF16, int CV>
__global__ __launch_bounds__(kIgThreads) void k_seg_kl_blockmax_nhwc16(
    const uint4 *__restrict__ lt, const uint4 *__restrict__ lp, IgGeom g, float *__restrict__ ig)
{
    __shared__ float wave_max[kIgThreads / 64];
    const IgPart q = ig_part(g);
    if (g.mask && !g.mask[q.blk]) {   // not executed: its scores were copied, the gain is 0
        if (g.strips == 1 && threadIdx.x == 0) ig[q.blk] = 0.f;
        return;
    }
    const int vpp = g.c / 8;
    const size_t img_vec = (size_t)g.h * g.w * vpp;
    const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(lt + q.img * img_vec), (short)0, g.bytes, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(lp + q.img * img_vec), (short)0, g.bytes, kBufferFlags);
    float best = 0.f;
    for (int p0 = threadIdx.x; p0 < q.npix; p0 += kIgThreads * kIgUnroll) {
        i32x4 va[kIgUnroll][CV], vb[kIgUnroll][CV];
#pragma unroll
        for (int u = 0; u < kIgUnroll; ++u) {
            const int p = p0 + u * kIgThreads;
            const int y = q.y0 + p / q.bw, x = q.gx * q.bw + p % q.bw;
            int base = p < q.npix ? (y * g.w + x) * vpp * 16 : kOutOfRange;
            asm volatile("" : "+v"(base));
#pragma unroll
            for (int j = 0; j < CV; ++j) {
                va[u][j] = __builtin_amdgcn_raw_buffer_load_b128(rt, base + 16 * j, 0, 0);
                vb[u][j] = __builtin_amdgcn_raw_buffer_load_b128(rp, base + 16 * j, 0, 0);
            }
        }
#pragma unroll
        for (int u = 0; u < kIgUnroll; ++u) {
            if (p0 + u * kIgThreads >= q.npix) break;
            float a[8 * CV], b[8 * CV];
#pragma unroll
            for (int j = 0; j < CV; ++j) {
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const int sh = 16 * (t & 1);
                    a[8 * j + t] = h16_to_f32<BF16>(((uint32_t)va[u][j][t >> 1] >> sh) & 0xFFFFu);
                    b[8 * j + t] = h16_to_f32<BF16>(((uint32_t)vb[u][j][t >> 1] >> sh) & 0xFFFFu);
                }
            }
            const float kl = pixel_kl<8 * CV>(a, b, g.classes);
            best = kl > best ? kl : best;
        }
    }
    block_max_out(best, wave_max, &ig[q.blk], g.strips == 1);
}

// ---------------------------------------------------------------- rewards

constexpr int kRwThreads = 256;

// Sum over the workgroup in a fixed order (thread partials, then a fixed tree).
__device__ float block_sum(float v, float *scratch)
{
    scratch[threadIdx.x] = v;
    __syncthreads();
#pragma unroll
    for (int s = kRwThreads / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) scratch[threadIdx.x] += scratch[threadIdx.x + s];
        __syncthreads();
    }
    const float r = scratch[0];
    __syncthreads();
    return r;
}

// One workgroup per image: C_t, M_t, the rewards of every block and the loss.
__global__ __launch_bounds__(kRwThreads) void k_block_rewards(
    const float *__restrict__ ig, const uint8_t *__restrict__ mask, const float *__restrict__ prob,
    int blocks, float tau, float gamma, float mu, float *__restrict__ mavg,
    float *__restrict__ reward, float *__restrict__ cost, float *__restrict__ loss)
{
    __shared__ float scratch[kRwThreads];
    const int img = blockIdx.x;
    const size_t base = (size_t)img * blocks;
    int executed = 0;
    for (int b = threadIdx.x; b < blocks; b += kRwThreads) executed += mask[base + b] != 0;
    const float m_prev = mavg[img];
    const float ne = block_sum((float)executed, scratch);     // exact: integer < 2^24
    const float c_t = ne / (float)blocks;
    const float m_t = (1.f - mu) * c_t + mu * m_prev;
    const float slack = tau - m_t;
    float part = 0.f;
    for (int b = threadIdx.x; b < blocks; b += kRwThreads) {
        const bool a = mask[base + b] != 0;
        const float g = ig[base + b];
        const float r = (a ? g : -g) + gamma * (a ? slack : -slack);
        reward[base + b] = r;
        if (loss) {
            const float p = prob[base + b];
            part += r * logf(a ? p : 1.f - p);
        }
    }
    if (loss) {
        const float tot = block_sum(part, scratch);
        if (threadIdx.x == 0) loss[img] = -tot;
    }
    if (threadIdx.x == 0) {
        mavg[img] = m_t;       // every thread read m_prev before the sums' barriers
        if (cost) cost[img] = c_t;
    }
}

}  // namespace

hipError_t launch_sample_index(const float *prob, int total, uint64_t seed, uint64_t frame,
                               uint8_t *mask, int32_t *idx, int32_t *count, hipStream_t s)
{
    hipLaunchKernelGGL(k_sample_index, dim3(1), dim3(kCompactThreads), 0, s, prob, total,
                       (uint32_t)frame, (uint32_t)(frame >> 32), (uint32_t)seed,
                       (uint32_t)(seed >> 32), mask, idx, count);
    return hipGetLastError();
}

hipError_t launch_frame_state(const void *frame, void *state, int n, int c, int h, int w,
                              int esize, bool nhwc, int gh, int gw, const int32_t *idx,
                              const int32_t *count, hipStream_t s)
{
    const int bh = h / gh, bw = w / gw;
    const int total = n * gh * gw;
    const long long row_bytes = nhwc ? (long long)bw * c * esize : (long long)bw * esize;
    const long long pitch_bytes = nhwc ? (long long)w * c * esize : (long long)w * esize;
    const long long plane_bytes = nhwc ? 0 : (long long)h * w * esize;
    const long long span = nhwc ? (bh - 1) * pitch_bytes + row_bytes
                                : (c - 1) * plane_bytes + (bh - 1) * pitch_bytes + row_bytes;
    const bool vec = row_bytes % 16 == 0 && pitch_bytes % 16 == 0 && plane_bytes % 16 == 0 &&
                     ((uintptr_t)frame % 16) == 0 && ((uintptr_t)state % 16) == 0 &&
                     span < kOutOfRange;
    if (vec) {
        CopyGeom g;
        g.gh = gh; g.gw = gw; g.bh = bh; g.bw = bw; g.total_blocks = total;
        g.rows = nhwc ? bh : c * bh;
        g.rowv = (int)(row_bytes / 16);
        g.pitch = (int)(pitch_bytes / 16);
        g.plane = (int)(plane_bytes / 16);
        g.img = (long long)c * h * w * esize / 16;
        g.colv = (int)(row_bytes / 16);
        g.span_bytes = (int)span;
        const int chunks = (g.rows * g.rowv + kCopyVecPerWG - 1) / kCopyVecPerWG;
        hipLaunchKernelGGL(k_frame_state16, dim3((unsigned)total * chunks), dim3(kCopyThreads), 0,
                           s, (const uint4 *)frame, (uint4 *)state, g, chunks, idx, count);
    } else {
        const int per_block = c * bh * bw;
        const long long work = (long long)total * per_block;
        const unsigned grid = (unsigned)((work + kCopyThreads - 1) / kCopyThreads < 65536
                                             ? (work + kCopyThreads - 1) / kCopyThreads
                                             : 65536);
        if (esize == 2)
            hipLaunchKernelGGL(k_frame_state_elem<uint16_t>, dim3(grid), dim3(kCopyThreads), 0, s,
                               (const uint16_t *)frame, (uint16_t *)state, n, c, h, w, gh, gw,
                               (int)nhwc, idx, count, per_block);
        else
            hipLaunchKernelGGL(k_frame_state_elem<uint32_t>, dim3(grid), dim3(kCopyThreads), 0, s,
                               (const uint32_t *)frame, (uint32_t *)state, n, c, h, w, gh, gw,
                               (int)nhwc, idx, count, per_block);
    }
    return hipGetLastError();
}

template <bool BF16>
static void launch_ig_nhwc16(const void *lt, const void *lp, const IgGeom &g, dim3 grid, float *ig,
                      hipStream_t s)
{
    const uint4 *a = (const uint4 *)lt, *b = (const uint4 *)lp;
    switch ((g.classes + 7) / 8) {
    case 1: hipLaunchKernelGGL((k_seg_kl_blockmax_nhwc16<BF16, 1>), grid, dim3(kIgThreads), 0, s, a, b, g, ig); break;
    case 2: hipLaunchKernelGGL((k_seg_kl_blockmax_nhwc16<BF16, 2>), grid, dim3(kIgThreads), 0, s, a, b, g, ig); break;
    case 3: hipLaunchKernelGGL((k_seg_kl_blockmax_nhwc16<BF16, 3>), grid, dim3(kIgThreads), 0, s, a, b, g, ig); break;
    default: hipLaunchKernelGGL((k_seg_kl_blockmax_nhwc16<BF16, 4>), grid, dim3(kIgThreads), 0, s, a, b, g, ig); break;
    }
}

hipError_t launch_seg_information_gain(const void *lt, const void *lp, int n, int c, int classes,
                                       int h, int w, int esize, bool nhwc, bool bf16, int gh,
                                       int gw, const uint8_t *mask, float *ig, hipStream_t s)
{
    const int blocks = n * gh * gw;
    IgGeom g;
    g.classes = classes; g.c = c; g.h = h; g.w = w; g.gh = gh; g.gw = gw;
    g.mask = mask;
    const int bh = h / gh, bw = w / gw;
    if (nhwc && bh * bw <= 4 * kIgPixPerWG) {
        // one workgroup per block (at most 16 pixels per thread, requested 4 at a time):
        // its maximum is stored, no zero fill and no atomics
        g.rows = bh;
    } else {
        // about kIgPixPerWG pixels per workgroup, a quarter of that below 2M pixels (a
        // quarter-resolution score map) so that the launch still has >= 512 workgroups
        const int per_wg = (long long)n * h * w >= (1LL << 21) ? kIgPixPerWG : kIgPixPerWG / 4;
        g.rows = per_wg / bw;
        g.rows = g.rows < 1 ? 1 : (g.rows > bh ? bh : g.rows);
    }
    g.strips = (bh + g.rows - 1) / g.rows;
    if (g.strips > 1)
        hipLaunchKernelGGL(k_fill_zero, dim3((blocks + 255) / 256), dim3(256), 0, s, ig, blocks);
    g.bytes = (int)((size_t)c * h * w * esize);   // one image's scores (checked < 2 GiB)
    const dim3 grid((unsigned)blocks * g.strips), block(kIgThreads);
    const float *a = (const float *)lt, *b = (const float *)lp;
    if (nhwc) {
        if (bf16) launch_ig_nhwc16<true>(lt, lp, g, grid, ig, s);
        else launch_ig_nhwc16<false>(lt, lp, g, grid, ig, s);
    } else if (classes == 19) {
        hipLaunchKernelGGL(k_seg_kl_blockmax<19>, grid, block, 0, s, a, b, g, ig);
    } else if (classes <= 8) {
        hipLaunchKernelGGL(k_seg_kl_blockmax<8>, grid, block, 0, s, a, b, g, ig);
    } else {
        hipLaunchKernelGGL(k_seg_kl_blockmax<32>, grid, block, 0, s, a, b, g, ig);
    }
    return hipGetLastError();
}

hipError_t launch_block_rewards(const float *ig, const uint8_t *mask, const float *prob, int n,
                                int blocks, float tau, float gamma, float mu, float *mavg,
                                float *reward, float *cost, float *loss, hipStream_t s)
{
    hipLaunchKernelGGL(k_block_rewards, dim3(n), dim3(kRwThreads), 0, s, ig, mask, prob, blocks,
                       tau, gamma, mu, mavg, reward, cost, loss);
    return hipGetLastError();
}

}  // namespace bc
