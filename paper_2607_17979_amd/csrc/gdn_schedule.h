// Longest-first order of the sequences of a packed batch, the work order of
// the chunk kernels (the longest chains start first, so the last workgroups to
// finish are short ones).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gdn_index.h"

namespace gdn {

// Run by one whole workgroup: order[rank] = sequence index, ranks by decreasing
// length with ties by index (lengths of the clamped spans, seq_span).  Also
// checks cu_seqlens: returns, in every thread, the number of sequences longer
// than recur_max and whether cu_seqlens is malformed (*bad).  len: kSortMax
// ints of LDS; cnt: two ints of LDS.
__device__ __forceinline__ int schedule_longest_first(const int32_t* __restrict__ cu, int N, int T,
                                                      int32_t* __restrict__ order, int* len, int* cnt,
                                                      int recur_max, bool* bad) {
    if (threadIdx.x == 0) cnt[0] = cnt[1] = 0;
    __syncthreads();
    int nl = 0, nb = 0;
    for (int i = threadIdx.x; i < N; i += blockDim.x) {
        const int li = seq_span(cu, i, T).len;
        if (N <= kSortMax) len[i] = li;
        nl += li > recur_max;
        nb += cu_seqlens_breaks(cu, N, T, i);
    }
    if (nl) atomicAdd(&cnt[0], nl);
    if (nb) atomicAdd(&cnt[1], nb);
    __syncthreads();
    if (order != nullptr) {
        if (N > kSortMax) {
            for (int i = threadIdx.x; i < N; i += blockDim.x) order[i] = i;
        } else {
            for (int i = threadIdx.x; i < N; i += blockDim.x) order[longest_first_rank(len, N, i)] = i;
        }
    }
    *bad = cnt[1] != 0;
    return cnt[0];
}

}  // namespace gdn
