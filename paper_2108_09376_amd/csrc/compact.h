// Stable stream compaction shared by the kernels that turn per-block decisions into
// the active-block index (the execution grid of Section 3.5 -> ascending ids).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

constexpr int kCompactThreads = 1024;                 // one workgroup, 16 wave64s
constexpr int kCompactWaves = kCompactThreads / 64;

// One round of the compaction: every thread of the workgroup passes its predicate
// `act` for position i; an active thread writes i to idx[running + rank], where rank
// counts the active threads before it in thread order (a wave ballot and a masked
// popcount within the wave, the 16 wave totals prefix-summed through LDS). Ranks are
// therefore stable: ids come out in ascending order without a sort, independent of
// scheduling. Returns the round's total, the same in every thread. wave_total is
// kCompactWaves ints of LDS; the call holds two barriers, so all threads must call it.
__device__ __forceinline__ int compact_round(bool act, int i, int32_t *__restrict__ idx, int running,
                                             int *wave_total)
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const unsigned long long b = __ballot(act);
    const int rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32),
                                               __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0));
    if (lane == 0) wave_total[wave] = __popcll(b);
    __syncthreads();
    int before = 0, round_total = 0;
#pragma unroll
    for (int w = 0; w < kCompactWaves; ++w) {
        const int t = wave_total[w];
        before += (w < wave) ? t : 0;
        round_total += t;
    }
    if (act) idx[running + before + rank] = i;
    __syncthreads();                                  // wave_total is rewritten next round
    return round_total;
}

}  // namespace bc
