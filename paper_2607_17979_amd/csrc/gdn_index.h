// Index arithmetic of the kernels' work walks: which workgroup takes which
// (sequence, value head, column or row block) item, and the fields of an
// item.  Plain integer functions, compiled for the host as well as the
// device, so that a host build (with the address and undefined-behaviour
// sanitizers) can enumerate every walk and compare it with an independent
// enumeration.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

constexpr int kSortMax = 4096;  // larger batches keep their given order

// blockIdx -> logical work index.  The P consecutive work items P j .. P j +
// P - 1 (items that read the same q/k rows: the two value heads of a q/k head,
// times the value-column blocks of each) go to workgroups 8 apart, which the
// dispatcher places on the same XCD, so their reads share that L2.  A last
// partial group of 8 P items keeps the identity mapping.  A bijection of
// [0, total).
template <int P = 2>
__host__ __device__ inline int logical_item(int bid, int total) {
    constexpr int G = 8 * P;
    const int grp = bid / G;
    if (grp * G + G > total) return bid;
    const int r = bid - grp * G;
    return grp * G + P * (r & 7) + (r >> 3);
}

// Tokens [beg, beg + len) of sequence n, its offsets clamped into [0, T]: beg =
// clamp(cu[n], 0, T), end = clamp(cu[n + 1], beg, T).  For a valid cu_seqlens
// (cu[0] = 0, non-decreasing, cu[N] = T) this is cu[n] and cu[n + 1] - cu[n];
// for any other it still names no token outside [0, T), so a malformed
// cu_seqlens gives meaningless results but no access outside the buffers.
struct SeqSpan {
    int beg, len;
};
__host__ __device__ inline SeqSpan seq_span(const int32_t* cu, int n, int T) {
    int a = cu[n], b = cu[n + 1];
    a = a < 0 ? 0 : (a > T ? T : a);
    b = b < a ? a : (b > T ? T : b);
    return SeqSpan{a, b - a};
}
// Whether entry i of cu_seqlens breaks validity: cu[0] != 0, cu[N] != T, or
// cu[i + 1] < cu[i] (i in [0, N)); cu_seqlens is valid iff no i breaks it.
__host__ __device__ inline bool cu_seqlens_breaks(const int32_t* cu, int N, int T, int i) {
    return cu[i + 1] < cu[i] || (i == 0 && cu[0] != 0) || (i == N - 1 && cu[N] != T);
}

// Rank of sequence i when sequences are ordered by decreasing length, ties by
// index (len: the N lengths).
__host__ __device__ inline int longest_first_rank(const int* len, int N, int i) {
    const int li = len[i];
    int rank = 0;
    for (int j = 0; j < N; ++j) {
        const int lj = len[j];
        rank += (lj > li) || (lj == li && j < i);
    }
    return rank;
}

// ---- token-by-token kernel: units (sequence n, value head h, row block blk),
// u = (n H_v + h) BPH + blk.  Workgroup w (w >= 1) walks the slots w - 1,
// w - 1 + stride, ... and slot s holds unit recur_slot_unit(s).

// Whether unit u runs in the token-by-token kernel: its sequence has at most
// recur_max tokens and its state lies inside the pool (with state_idx).
__host__ __device__ inline bool recur_unit_runs(long u, int bph, int H_v, const int32_t* cu, int T,
                                                const int32_t* state_idx, int P, int recur_max) {
    const int n = (int)(u / bph / H_v);
    if (seq_span(cu, n, T).len > recur_max) return false;
    if (state_idx != nullptr) {
        const int slot = state_idx[n];
        if (slot < 0 || slot >= P) return false;
    }
    return true;
}

// Unit of slot s.  The grp consecutive units grp j .. grp j + grp - 1 (the
// units that read the same q/k rows: the row blocks of the value heads of one
// q/k head) sit in slots 8 apart; with a stride that is a multiple of 8 (or a
// single pass) they run on workgroups 8 apart, which the dispatcher places on
// one XCD, so those reads share its L2.  A last partial block of 8 grp slots
// keeps the identity.  A bijection of [0, units).
__host__ __device__ inline long recur_slot_unit(long s, long units, int grp) {
    const long G = 8L * grp;
    const long blk = s / G;
    if (blk * G + G > units) return s;
    const long r = s - blk * G;
    return blk * G + grp * (r & 7) + (r >> 3);
}

// The first slot at or after s (stepping by stride) whose unit runs here, or
// a value >= units.
__host__ __device__ inline long recur_next_slot(long s, long stride, long units, int grp, int bph, int H_v,
                                                const int32_t* cu, int T, const int32_t* state_idx, int P,
                                                int recur_max) {
    while (s < units && !recur_unit_runs(recur_slot_unit(s, units, grp), bph, H_v, cu, T, state_idx, P, recur_max))
        s += stride;
    return s;
}

// Fields of a unit that runs: its head, q/k head, row block, tokens and state
// (state n H_v + h, or pool slot state_idx[n] H_v + h).
struct RecurUnit {
    long u, shead;
    int h, hq, blk, t0, len;
};
__host__ __device__ inline RecurUnit recur_unit_at(long u, int bph, int H_v, int H_qk, const int32_t* cu, int T,
                                                   const int32_t* state_idx) {
    RecurUnit r;
    const long head = u / bph;  // n H_v + h
    const int n = (int)(head / H_v);
    r.u = u;
    r.h = (int)(head - (long)n * H_v);
    r.hq = r.h / (H_v / H_qk);
    r.blk = (int)(u - head * bph);
    const SeqSpan sp = seq_span(cu, n, T);
    r.t0 = sp.beg;
    r.len = sp.len;
    r.shead = state_idx != nullptr ? (long)state_idx[n] * H_v + r.h : head;
    return r;
}

// ---- chunk kernel: items (rank, value head h, value block vb), item =
// (rank H_v + h) VSPLIT + vb, over G workgroups: on pass p workgroup b takes
// the virtual index p G + b (p even) or p G + G - 1 - b (p odd), mapped by
// logical_item<2 VSPLIT>; -1 past the last item.
template <int VSPLIT>
__host__ __device__ inline int pipe_item_at(int pass, int G, int bid, int items) {
    const int vb = pass * G + ((pass & 1) ? G - 1 - bid : bid);
    return vb < items ? logical_item<2 * VSPLIT>(vb, items) : -1;
}

// Fields of a chunk-kernel item: sequence (order[rank]), value head, q/k head,
// value block, tokens, chunk count (0: not the chunk kernel's, or outside the
// pool) and state (sequence n, or its pool slot).
struct PipeItem {
    int n, h, hq, vblock, seq_beg, seq_len, nch;
    long slot;
};
__host__ __device__ inline PipeItem pipe_item_fields(int item, int vsplit, int H_v, int H_qk,
                                                     const int32_t* order, const int32_t* cu, int T,
                                                     const int32_t* state_idx, int P, int chunk,
                                                     int recur_max) {
    PipeItem it;
    const int head_item = item / vsplit;
    it.vblock = item - head_item * vsplit;
    const int rank = head_item / H_v;
    it.h = head_item - rank * H_v;
    it.n = order[rank];
    it.hq = it.h / (H_v / H_qk);
    const SeqSpan sp = seq_span(cu, it.n, T);
    it.seq_beg = sp.beg;
    it.seq_len = sp.len;
    it.nch = it.seq_len <= recur_max ? 0 : (it.seq_len + chunk - 1) / chunk;
    it.slot = it.n;
    if (state_idx != nullptr) {
        it.slot = state_idx[it.n];
        if (it.slot < 0 || it.slot >= P) it.nch = 0;
    }
    return it;
}

}  // namespace gdn
