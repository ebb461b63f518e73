// Execution grid -> active-block index (Section 3.5: a_b = 1 executes block b).
//
// One workgroup of 1024 threads (16 wave64s) walks the mask in rounds of 1024
// entries. Within a wave, a ballot of the "execute" predicate and a masked
// popcount (mbcnt) give each lane its rank among the active lanes; the 16 wave
// totals are prefix-summed through LDS. Ranks are therefore stable, so the index
// comes out in ascending raster order without any sort, and the result does not
// depend on scheduling. Masks of up to 2^20 blocks are accepted by the ABI layer.
#include "bc_internal.h"

namespace bc {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__global__ __launch_bounds__(kThreads) void k_block_index(const uint8_t *__restrict__ mask,
                                                           int total, int32_t *__restrict__ idx,
                                                           int32_t *__restrict__ count)
{
    __shared__ int wave_total[kWaves];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int running = 0;
    for (int base = 0; base < total; base += kThreads) {
        const int i = base + tid;
        const bool act = (i < total) && (mask[i] != 0);
        const unsigned long long b = __ballot(act);
        const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0));
        if (lane == 0) wave_total[wave] = __popcll(b);
        __syncthreads();
        int before = 0, round_total = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int t = wave_total[w];
            before += (w < wave) ? t : 0;
            round_total += t;
        }
        if (act) idx[running + before + rank] = i;
        running += round_total;
        __syncthreads();  // wave_total is rewritten next round
    }
    if (tid == 0) *count = running;
}

}  // namespace

hipError_t launch_block_index(const uint8_t *mask, int total, int32_t *idx, int32_t *count,
                              hipStream_t s)
{
    hipLaunchKernelGGL(k_block_index, dim3(1), dim3(kThreads), 0, s, mask, total, idx, count);
    return hipGetLastError();
}

}  // namespace bc
