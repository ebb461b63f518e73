// Execution grid -> active-block index (Section 3.5: a_b = 1 executes block b).
//
// One workgroup of 1024 threads (16 wave64s) walks the mask in rounds of 1024
// entries with the stable ballot compaction of compact.h, so the index comes out in
// ascending raster order without any sort, and the result does not depend on
// scheduling. Masks of up to 2^20 blocks are accepted by the ABI layer.
#include "bc_internal.h"
#include "compact.h"

namespace bc {
namespace {

__global__ __launch_bounds__(kCompactThreads) void k_block_index(const uint8_t *__restrict__ mask,
                                                                  int total, int32_t *__restrict__ idx,
                                                                  int32_t *__restrict__ count)
{
    __shared__ int wave_total[kCompactWaves];
    int running = 0;
    for (int base = 0; base < total; base += kCompactThreads) {
        const int i = base + (int)threadIdx.x;
        const bool act = (i < total) && (mask[i] != 0);
        running += compact_round(act, i, idx, running, wave_total);
    }
    if (threadIdx.x == 0) *count = running;
}

}  // namespace

hipError_t launch_block_index(const uint8_t *mask, int total, int32_t *idx, int32_t *count,
                              hipStream_t s)
{
    hipLaunchKernelGGL(k_block_index, dim3(1), dim3(kCompactThreads), 0, s, mask, total, idx, count);
    return hipGetLastError();
}

}  // namespace bc
