// Host-side launch interface between the C ABI layer (argument checks) and
// the kernel files.  Arguments reaching these functions are already checked.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gdn {

struct DecodeArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    float* state;
    void* o;
    int B, H_qk, H_v, D;
    float scale;
    const int32_t* state_idx;  // NULL: state b is batch entry b; else a pool slot per entry
    int P;                     // pool slots (with state_idx)
    int flags;                 // input prologue: kFlagQkL2Norm | kFlagGateLogits (gdn_device.h)
};

struct PrefillArgs {
    const void* q;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    const int32_t* cu_seqlens;
    const float* initial_state;
    float* final_state;
    void* o;
    int N, T, H_qk, H_v, D, chunk;
    float scale;
    void* workspace;
    const int32_t* state_idx;  // NULL: state n is sequence n; else a pool slot per sequence
    int P;                     // pool slots (with state_idx)
    bool short_only;           // the caller's promise that no sequence exceeds kRecurMax:
                               // only the token-by-token launch runs, and a longer sequence
                               // is skipped and flagged (wait-fault word bit 1)
    int flags;                 // input prologue: kFlagQkL2Norm | kFlagGateLogits (gdn_device.h)
};

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_prefill(const PrefillArgs& a, hipStream_t stream);
// d = 128: sequences of at most kRecurMax tokens run token by token
// (gdn_recur.hip), longer ones in chunks; the route depends only on a
// sequence's own length.  The recurrent launch also writes the schedule.
// Measured on 64 sequences x 32 heads: token by token is faster up to about
// 10 tokens, the chunk kernel beyond.
constexpr int kRecurMax = 8;
hipError_t launch_prefill_recur(const PrefillArgs& a, int32_t* order, hipStream_t stream);
// d = 128, chunk 64: the pipelined kernel (gdn_prefill_pipe.hip); `order` is the
// workspace, holding the longest-first schedule already written (the kernel
// sets its wait-fault word).
hipError_t launch_prefill_pipe(const PrefillArgs& a, int32_t* order, hipStream_t stream);
// Compute units of the current device (queried once per device).
int device_compute_units();

// Workspace layout of the prefill: int32 order[N] (sequence indices sorted by
// length, longest first, ties by index), then (d = 128) int32 order[N] = the
// number of sequences longer than kRecurMax, then int32 order[N + 1] = the
// fault word (written by the call's first launch; bit 0 set by any wave of the
// chunk kernel whose counter wait ran out of its bound, bit 1 by a short-only
// call that met a longer sequence, bit 2 by a malformed cu_seqlens); rounded up
// to 256 bytes.
size_t prefill_workspace_bytes(int N);

}  // namespace gdn
