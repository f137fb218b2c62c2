// Host-only enumeration of the kernels' work walks for the sanitizer build:
// the token-by-token kernel's unit walk (as the kernel runs it, and a
// reconstruction of an earlier form that scanned for the next unit and
// returned every field of it from one function), the longest-first schedule
// and the chunk kernel's item walk, all through the functions the kernels
// call (gdn_index.h).  Reads a configuration from stdin, prints one line per
// visited unit or item; the test compares them with its own enumeration.
// Input starting with "spans": N, T and N + 1 raw cu_seqlens values, possibly
// malformed; prints each sequence's clamped span and each entry's validity
// check.
#include <cstdio>
#include <iostream>
#include <string>
#include <vector>

#include "gdn_index.h"

using namespace gdn;

namespace {

constexpr int kRecurMax = 8;  // sequences of at most this many tokens run token by token
constexpr int kBph = 4;       // workgroups (row blocks) per (sequence, head) in that kernel
constexpr int kChunk = 64;

// The earlier form of the walk, reconstructed: one function scans for the
// next slot whose unit runs and returns all of its fields (s is left at that
// slot).
RecurUnit legacy_next(long& s, long stride, long units, int H_v, int H_qk, const int32_t* cu, int T,
                      const int32_t* state_idx, int P) {
    RecurUnit r;
    const int grp = (H_v / H_qk) * kBph;
    for (; s < units; s += stride) {
        const long u = recur_slot_unit(s, units, grp);
        const long head = u / kBph;
        const int n = (int)(head / H_v);
        r.h = (int)(head - (long)n * H_v);
        const SeqSpan sp = seq_span(cu, n, T);
        r.t0 = sp.beg;
        r.len = sp.len;
        if (r.len > kRecurMax) continue;
        long shead = head;
        if (state_idx != nullptr) {
            const long slot = state_idx[n];
            if (slot < 0 || slot >= P) continue;
            shead = slot * H_v + r.h;
        }
        r.u = u;
        r.hq = r.h / (H_v / H_qk);
        r.blk = (int)(u - head * kBph);
        r.shead = shead;
        return r;
    }
    r = RecurUnit{units, 0, 0, 0, 0, 0, 0};
    return r;
}

template <int VSPLIT>
void pipe_walk(int G, int items, int H_v, int H_qk, const int32_t* order, const int32_t* cu, int T,
               const int32_t* state_idx, int P) {
    for (int b = 0; b < G; ++b)
        for (int pass = 0;; ++pass) {
            const int item = pipe_item_at<VSPLIT>(pass, G, b, items);
            if (item < 0) break;
            const PipeItem it = pipe_item_fields(item, VSPLIT, H_v, H_qk, order, cu, T, state_idx, P, kChunk, kRecurMax);
            std::printf("pipe %d %d %d %d %d %d %d %ld %d %d\n", b, pass, item, it.n, it.h, it.vblock, it.nch,
                        it.slot, it.seq_beg, it.seq_len);
        }
}

}  // namespace

int spans() {
    int N, T;
    std::cin >> N >> T;
    std::vector<int32_t> cu(N + 1);
    for (int i = 0; i <= N; ++i) std::cin >> cu[i];
    for (int n = 0; n < N; ++n) {
        const SeqSpan sp = seq_span(cu.data(), n, T);
        std::printf("span %d %d %d\n", n, sp.beg, sp.len);
    }
    for (int i = 0; i < N; ++i) std::printf("breaks %d %d\n", i, (int)cu_seqlens_breaks(cu.data(), N, T, i));
    return 0;
}

int main() {
    std::string first;
    std::cin >> first;
    if (first == "spans") return spans();
    int N = std::stoi(first), H_qk, H_v, P, grid_recur, grid_pipe, vsplit, use_idx;
    std::cin >> H_qk >> H_v >> P >> grid_recur >> grid_pipe >> vsplit >> use_idx;
    std::vector<int32_t> len(N), cu(N + 1, 0), idx(N, 0);
    for (int i = 0; i < N; ++i) {
        std::cin >> len[i];
        cu[i + 1] = cu[i] + len[i];
    }
    if (use_idx)
        for (int i = 0; i < N; ++i) std::cin >> idx[i];
    const int32_t* sidx = use_idx ? idx.data() : nullptr;
    const int T = cu[N];
    // token-by-token walk, as the kernel runs it: workgroups 1 .. grid - 1
    const long units = (long)N * H_v * kBph, stride = grid_recur - 1;
    const int grp = (H_v / H_qk) * kBph;
    for (int b = 1; b < grid_recur; ++b) {
        long s = recur_next_slot(b - 1, stride, units, grp, kBph, H_v, cu.data(), T, sidx, P, kRecurMax);
        while (s < units) {
            const RecurUnit r = recur_unit_at(recur_slot_unit(s, units, grp), kBph, H_v, H_qk, cu.data(), T, sidx);
            std::printf("recur %d %ld %d %d %d %ld %d %d\n", b, r.u, r.h, r.hq, r.blk, r.shead, r.t0, r.len);
            s = recur_next_slot(s + stride, stride, units, grp, kBph, H_v, cu.data(), T, sidx, P, kRecurMax);
        }
        long ls = b - 1;
        for (RecurUnit r = legacy_next(ls, stride, units, H_v, H_qk, cu.data(), T, sidx, P); ls < units;
             ls += stride, r = legacy_next(ls, stride, units, H_v, H_qk, cu.data(), T, sidx, P))
            std::printf("legacy %d %ld %d %d %d %ld %d %d\n", b, r.u, r.h, r.hq, r.blk, r.shead, r.t0, r.len);
    }
    // longest-first schedule (identity beyond kSortMax sequences)
    std::vector<int32_t> order(N);
    for (int i = 0; i < N; ++i) order[N > kSortMax ? i : longest_first_rank(len.data(), N, i)] = i;
    for (int r = 0; r < N; ++r) std::printf("order %d %d\n", r, order[r]);
    // chunk-kernel item walk
    const int items = N * H_v * vsplit;
    if (vsplit == 1) pipe_walk<1>(grid_pipe, items, H_v, H_qk, order.data(), cu.data(), T, sidx, P);
    if (vsplit == 2) pipe_walk<2>(grid_pipe, items, H_v, H_qk, order.data(), cu.data(), T, sidx, P);
    if (vsplit == 4) pipe_walk<4>(grid_pipe, items, H_v, H_qk, order.data(), cu.data(), T, sidx, P);
    // logical_item: bijections
    for (int total : {1, 7, 16, 31, 32, 33, 100, 257}) {
        for (int bid = 0; bid < total; ++bid)
            std::printf("logical2 %d %d %d\n", total, bid, logical_item<2>(bid, total));
        for (int bid = 0; bid < total; ++bid)
            std::printf("logical8 %d %d %d\n", total, bid, logical_item<8>(bid, total));
    }
    return 0;
}
