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
#include "bc_internal.h"

namespace bc {
namespace {

typedef short short8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int BK = 32;               // input channels per K step (one MFMA k)
constexpr int PITCH = BK * 2 + 16;   // bytes per LDS slot / weight row (64 data + 16 pad)
constexpr int kMaxAV = 12;           // halo slots per thread quarter: nslot <= 64 * kMaxAV
constexpr int EPITCH = 36;           // floats per epilogue scratch row (32 + 4 pad)
constexpr size_t kMaxLds = 64 * 1024;

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

// Active block of patch p of M tile mt; false when the patch lies beyond the count.
__device__ __forceinline__ bool patch_block(const MfmaArgs &a, int count, int mt, int p,
                                            int &img, int &oy0, int &ox0)
{
    int k, r0;
    if (a.P == 1) {
        k = mt / a.tpb;
        r0 = (mt - k * a.tpb) * a.R;
    } else {
        k = mt * a.P + p;
        r0 = 0;
    }
    if (k >= count) return false;
    const int bid = a.idx ? a.idx[k] : k;
    img = bid / (a.gh * a.gw);
    const int rem = bid - img * a.gh * a.gw;
    const int gy = rem / a.gw;
    oy0 = gy * a.bh + r0;
    ox0 = (rem - gy * a.gw) * a.bw;
    return true;
}

// Tile of this workgroup, XCD-first numbering over the T = mtiles * ntn live tiles.
__device__ __forceinline__ bool tile_of(const MfmaArgs &a, int &count, int &mt, int &nt)
{
    count = a.count ? *a.count : a.total_blocks;
    const int mtiles = (a.P == 1) ? count * a.tpb : (count + a.P - 1) / a.P;
    const int T = mtiles * a.ntn;
    const int L = blockIdx.x;
    if (L >= T) return false;
    const int xcd = L & 7, j = L >> 3, q8 = T >> 3, r8 = T & 7;
    const int logical = xcd * q8 + min(xcd, r8) + j;
    mt = logical / a.ntn;
    nt = logical - mt * a.ntn;
    return true;
}

// Fused epilogue: bias + residual + ReLU + rounding, 16-byte stores to block positions.
template <bool BF16, int BM, int BN>
__device__ __forceinline__ void epilogue(const MfmaArgs &a, f32x4 (&acc)[BM / 32][BN / 32],
                                         uint8_t *smem, int count, int mt, int n0)
{
    constexpr int WM = BM / 2, WN = BN / 2, MI = WM / 16;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    float *scr = (float *)smem + wave * (WM * EPITCH);
    const int rbw = a.R * a.bw;
#pragma unroll
    for (int np = 0; np < WN / 32; ++np) {
        __syncthreads();
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int nn = 0; nn < 2; ++nn)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    scr[(mi * 16 + 4 * (lane >> 4) + i) * EPITCH + nn * 16 + (lane & 15)] =
                        acc[mi][np * 2 + nn][i];
        __syncthreads();
#pragma unroll
        for (int u = 0; u < WM / 16; ++u) {
            const int item = lane + 64 * u;
            const int row = item >> 2, cv = item & 3;
            const int m = wm * WM + row;
            const int co = n0 + wn * WN + np * 32 + cv * 8;
            const int p = m / rbw;
            const int local = m - p * rbw;
            const int pr = local / a.bw, pc = local - (local / a.bw) * a.bw;
            int img, oy0, ox0;
            if (!patch_block(a, count, mt, p, img, oy0, ox0)) continue;
            const size_t pix = ((size_t)img * a.hout + oy0 + pr) * a.wout + ox0 + pc;
            const float4 s0 = *(const float4 *)(scr + row * EPITCH + cv * 8);
            const float4 s1 = *(const float4 *)(scr + row * EPITCH + cv * 8 + 4);
            float z[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
            if (a.bias) {
                const float4 b0 = *(const float4 *)(a.bias + co);
                const float4 b1 = *(const float4 *)(a.bias + co + 4);
                z[0] += b0.x; z[1] += b0.y; z[2] += b0.z; z[3] += b0.w;
                z[4] += b1.x; z[5] += b1.y; z[6] += b1.z; z[7] += b1.w;
            }
            if (a.res) {
                const uint4 r = *(const uint4 *)(a.res + pix * a.cout + co);
                const uint32_t rw[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    z[2 * t] += to_f32<BF16>(rw[t] & 0xFFFFu);
                    z[2 * t + 1] += to_f32<BF16>(rw[t] >> 16);
                }
            }
            uint32_t o[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                float z0 = z[2 * t], z1 = z[2 * t + 1];
                if (a.relu) {
                    z0 = (z0 > 0.f || z0 != z0) ? z0 : 0.f;
                    z1 = (z1 > 0.f || z1 != z1) ? z1 : 0.f;
                }
                o[t] = to_h16<BF16>(z0) | (to_h16<BF16>(z1) << 16);
            }
            *(uint4 *)(a.y + pix * a.cout + co) = make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
}

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

    int count, mt, nt;
    if (!tile_of(a, count, mt, nt)) return;
    const int n0 = nt * BN;
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
            int img, oy0, ox0;
            if (patch_block(a, count, mt, p, img, oy0, ox0)) {
                const int iy = oy0 * S - a.pad + ra * SS, ix = ox0 * S - a.pad + rb * SS;
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
    epilogue<BF16, BM, BN>(a, acc, smem, count, mt, n0);
}

// ------------------------------------------------------------------ stem form

template <bool BF16, int BM, int BN, int KS, int S>
__global__ __launch_bounds__(kThreads) void k_conv_mfma_stem(MfmaArgs a)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int MI = WM / 16, NI = WN / 16;
    constexpr int BKP = 40;  // elements per LDS weight row (32 + 8 pad)
    extern __shared__ __align__(16) uint8_t smem[];

    int count, mt, nt;
    if (!tile_of(a, count, mt, nt)) return;
    const int n0 = nt * BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int kwc = KS * a.cin;            // values per kernel row, <= 32
    const int rp = a.rowpitch;             // elements per halo row (>= HC*cin + 32)
    uint16_t *sA = (uint16_t *)smem;                       // [P][HR][rp]
    uint16_t *sB = sA + (size_t)a.P * a.HR * rp;           // [KS][BN][BKP]

    // stage halo rows: raw channels-last runs, zero outside the image and in the tail
    const int rowvals = a.HC * a.cin;
    const int nrows = a.P * a.HR;
    for (int e = tid; e < nrows * rp; e += kThreads) {
        const int row = e / rp, t = e - (e / rp) * rp;
        const int p = row / a.HR, ra = row - (row / a.HR) * a.HR;
        uint16_t v = 0;
        int img, oy0, ox0;
        if (t < rowvals && patch_block(a, count, mt, p, img, oy0, ox0)) {
            const int rb = t / a.cin, ch = t - (t / a.cin) * a.cin;
            const int iy = oy0 * S - a.pad + ra, ix = ox0 * S - a.pad + rb;
            if (iy >= 0 && iy < a.hin && ix >= 0 && ix < a.win)
                v = a.x[(((size_t)img * a.hin + iy) * a.win + ix) * a.cin + ch];
        }
        sA[e] = v;
    }
    // stage weights: B[i][n][kk] = W[n0 + n][i][kk] for kk < kw*cin, else 0
    for (int e = tid; e < KS * BN * BKP; e += kThreads) {
        const int i = e / (BN * BKP);
        const int r = e - i * BN * BKP;
        const int n = r / BKP, kk = r - (r / BKP) * BKP;
        sB[e] = kk < kwc ? a.w[((size_t)(n0 + n) * KS + i) * kwc + kk] : (uint16_t)0;
    }
    __syncthreads();

    const int rbw = a.R * a.bw;
    int arow[MI], acol[MI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int m = wm * WM + mi * 16 + (lane & 15);
        const int p = m / rbw;
        const int local = m - p * rbw;
        const int pr = local / a.bw, pc = local - (local / a.bw) * a.bw;
        arow[mi] = (p * a.HR + pr * S) * rp;
        acol[mi] = pc * S * a.cin + (lane >> 4) * 8;
    }
    f32x4 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int i = 0; i < KS; ++i) {
        short8 af[MI], bf[NI];
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            const uint16_t *src = sA + arow[mi] + i * rp + acol[mi];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                af[mi][j] = ((lane >> 4) * 8 + j < kwc) ? (short)src[j] : (short)0;
        }
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            bf[ni] = *(const short8 *)(sB + ((size_t)i * BN + wn * WN + ni * 16 + (lane & 15)) * BKP +
                                       (lane >> 4) * 8);
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = mfma<BF16>(af[mi], bf[ni], acc[mi][ni]);
    }
    epilogue<BF16, BM, BN>(a, acc, smem, count, mt, n0);
}

// ------------------------------------------------------------------ planning

struct Plan {
    int BM, BN;
    bool stem;
    MfmaArgs a;
    size_t lds;
    unsigned grid;
};

size_t epi_lds(int BM) { return (size_t)4 * (BM / 2) * EPITCH * sizeof(float); }

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
    a.R = R;
    a.P = P;
    a.tpb = (P == 1) ? g.bh / R : 1;
    return true;
}

bool make_plan(const LayerGeom &g, int BM, int BN, Plan &pl)
{
    MfmaArgs &a = pl.a;
    if (g.cout % BN) return false;
    if (!tile_rows(g, BM, a)) return false;
    const int KS = g.kh, S = g.stride;
    pl.stem = (g.cin % 8) != 0;
    if (pl.stem) {
        if (KS * g.cin > 32 || BN != 64) return false;
        a.HR = (a.R - 1) * S + KS;
        a.HC = (g.bw - 1) * S + KS;
        a.rowpitch = ((a.HC * g.cin + 32) + 7) / 8 * 8;
        a.nslot = 0;
        const size_t main = (size_t)a.P * a.HR * a.rowpitch * 2 + (size_t)KS * BN * 40 * 2;
        pl.lds = main > epi_lds(BM) ? main : epi_lds(BM);
    } else {
        if (KS == 1) {
            a.HR = a.R;
            a.HC = g.bw;
        } else {
            a.HR = (a.R - 1) * S + KS;
            a.HC = (g.bw - 1) * S + KS;
        }
        a.nslot = a.P * a.HR * a.HC;
        if (a.nslot > 64 * kMaxAV) return false;
        a.rowpitch = 0;
        const size_t main = (size_t)a.nslot * PITCH + (size_t)2 * BN * PITCH;
        pl.lds = main > epi_lds(BM) ? main : epi_lds(BM);
    }
    if (pl.lds > kMaxLds) return false;
    pl.BM = BM;
    pl.BN = BN;
    a.ntn = g.cout / BN;
    const int mt_full = (a.P == 1) ? g.total_blocks * a.tpb : (g.total_blocks + a.P - 1) / a.P;
    pl.grid = (unsigned)mt_full * a.ntn;
    return true;
}

// Largest tiles that still give the full frame >= 1024 workgroups (about 300 at the
// 30 % active fraction of the sparse frames), falling back to whatever fits.
bool choose_plan(const LayerGeom &g, Plan &best)
{
    static const int cand[4][2] = {{128, 128}, {128, 64}, {64, 128}, {64, 64}};
    bool have = false;
    for (const auto &c : cand) {
        Plan p;
        if (!make_plan(g, c[0], c[1], p)) continue;
        if (!have) {
            best = p;
            have = true;
        }
        if (p.grid >= 1024) {
            best = p;
            return true;
        }
        if (p.grid > best.grid) best = p;
    }
    return have;
}

template <bool BF16, int BM, int BN, int KS, int S>
void launch_one(const Plan &p, hipStream_t s)
{
    if (p.stem)
        hipLaunchKernelGGL((k_conv_mfma_stem<BF16, BM, BN, KS, S>), dim3(p.grid), dim3(kThreads),
                           p.lds, s, p.a);
    else
        hipLaunchKernelGGL((k_conv_mfma<BF16, BM, BN, KS, S>), dim3(p.grid), dim3(kThreads), p.lds,
                           s, p.a);
}

template <bool BF16, int KS, int S>
void launch_tiles(const Plan &p, hipStream_t s)
{
    if (p.BM == 128 && p.BN == 128) launch_one<BF16, 128, 128, KS, S>(p, s);
    else if (p.BM == 128) launch_one<BF16, 128, 64, KS, S>(p, s);
    else if (p.BN == 128) launch_one<BF16, 64, 128, KS, S>(p, s);
    else launch_one<BF16, 64, 64, KS, S>(p, s);
}

template <bool BF16>
void launch_geom(const Plan &p, int ks, int stride, hipStream_t s)
{
    if (ks == 1) stride == 1 ? launch_tiles<BF16, 1, 1>(p, s) : launch_tiles<BF16, 1, 2>(p, s);
    else if (ks == 3) stride == 1 ? launch_tiles<BF16, 3, 1>(p, s) : launch_tiles<BF16, 3, 2>(p, s);
    else if (ks == 5) stride == 1 ? launch_tiles<BF16, 5, 1>(p, s) : launch_tiles<BF16, 5, 2>(p, s);
    else stride == 1 ? launch_tiles<BF16, 7, 1>(p, s) : launch_tiles<BF16, 7, 2>(p, s);
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
    if (g.cin % 8 && g.kw * g.cin > 32) {
        *why = "matrix-core path: Cin must be a multiple of 8, or kw*Cin <= 32 (stem form)";
        return false;
    }
    if ((double)g.n * g.hin * g.win * g.cin >= 2147483647.0 ||
        (double)g.cout * g.kh * g.kw * g.cin >= 2147483647.0) {
        *why = "matrix-core path: tensor larger than 2^31 elements";
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

hipError_t launch_conv_nhwc_mfma(const uint16_t *x, const uint16_t *w, const float *bias,
                                 const uint16_t *res, uint16_t *y, int relu, Half16 fmt,
                                 const LayerGeom &g, hipStream_t s, const char **why)
{
    if (!conv_nhwc_mfma_supported(g, why)) return hipErrorInvalidValue;
    Plan p;
    choose_plan(g, p);
    MfmaArgs &a = p.a;
    a.x = x; a.w = w; a.bias = bias; a.res = res; a.y = y;
    a.idx = g.idx; a.count = g.count;
    a.hin = g.hin; a.win = g.win; a.cin = g.cin;
    a.hout = g.hout; a.wout = g.wout; a.cout = g.cout;
    a.pad = g.pad; a.relu = relu;
    a.gh = g.gh; a.gw = g.gw; a.bh = g.bh; a.bw = g.bw; a.total_blocks = g.total_blocks;
    if (p.grid == 0) return hipSuccess;
    if (fmt == Half16::BF16) launch_geom<true>(p, g.kh, g.stride, s);
    else launch_geom<false>(p, g.kh, g.stride, s);
    return hipGetLastError();
}

}  // namespace bc
