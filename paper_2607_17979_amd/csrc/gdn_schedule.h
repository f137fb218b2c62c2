// Longest-first order of the sequences of a packed batch, the work order of
// the chunk kernels (the longest chains start first, so the last workgroups to
// finish are short ones).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdn_index.h"

namespace gdn {

// Run by one whole workgroup: order[rank] = sequence index, ranks by decreasing
// length with ties by index.  len: kSortMax ints of LDS.
__device__ __forceinline__ void schedule_longest_first(const int32_t* __restrict__ cu, int N,
                                                       int32_t* __restrict__ order, int* len) {
    if (N > kSortMax) {
        for (int i = threadIdx.x; i < N; i += blockDim.x) order[i] = i;
        return;
    }
    for (int i = threadIdx.x; i < N; i += blockDim.x) len[i] = cu[i + 1] - cu[i];
    __syncthreads();
    for (int i = threadIdx.x; i < N; i += blockDim.x) order[longest_first_rank(len, N, i)] = i;
}

}  // namespace gdn
