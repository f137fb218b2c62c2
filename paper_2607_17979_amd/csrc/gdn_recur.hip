// Short sequences of the prefill regime, token by token (paper: appendix
// "Operator Background and Mathematical Definitions", subsection "Gated Delta
// Net": the recurrence applied to each new token in turn), for d = 128.
//
// For a sequence of a few tokens the chunk kernel pays a whole chunk (the
// producer's start-up, a state load, one pass of the state chain) and its
// per-item costs dominate; token by token such a sequence costs one pass over
// its state plus a few rank-1 updates.  This kernel runs every sequence of
// 0 .. kRecurMax tokens and the chunk kernel skips them, so the route of a
// sequence depends only on its own length, never on the rest of the batch.
// With initial_state == final_state this is also the multi-token decode of a
// batch (each sequence a few new tokens, states updated in place).
//
// Per (sequence, value head), state row i and token t, alpha_t = exp(g_t):
//     kv_i = S_i . k_t,  sq_i = S_i . q_t                  (row before the token)
//     u_i  = beta_t (v_{t,i} - alpha_t kv_i)
//     S_i  = alpha_t S_i + u_i k_t^T
//     o_{t,i} = scale (alpha_t sq_i + u_i (k_t . q_t))      (= scale S_t q_t)
// Rows are independent, so a workgroup keeps 32 rows of one (sequence, head)
// in registers for the whole sequence, in the decode kernel's layout (a row of
// 128 fp32 over 8 consecutive lanes, 16 values per lane; S k and S q are sums
// over those 8 lanes).  The sequence's token inputs are staged in LDS first.
//
// Block 0 writes the longest-first schedule of the chunk kernel, which runs
// after this one on the same stream (the schedule costs no launch of its
// own), and the number of sequences left to it, so that it exits at once
// when every sequence is short.
#include <algorithm>

#include "gdn_device.h"
#include "gdn_index.h"
#include "gdn_launch.h"
#include "gdn_schedule.h"

namespace gdn {
namespace recur {

constexpr int D = 128;
constexpr int LPR = 8;                        // lanes per state row
constexpr int J = D / (4 * LPR);              // float4 slots per lane
constexpr int ROWS_PER_WAVE = 64 / LPR;
constexpr int NWAVE = 4;
constexpr int BPH = D / (NWAVE * ROWS_PER_WAVE);  // workgroups per (sequence, head)

// A unit's token inputs, staged in LDS once (their latency paid once per
// unit, not per token): k and q rows of the q/k head widened to fp32, this
// workgroup's 32 values of v, alpha = exp(g), beta and k . q per token.  Block
// 0 uses the same LDS for the schedule.
union Smem {
    int sched_len[kSortMax];
    struct {
        alignas(16) float k[kRecurMax][D];
        alignas(16) float q[kRecurMax][D];
        uint16_t v[kRecurMax][NWAVE * ROWS_PER_WAVE];
        float alpha[kRecurMax], b[kRecurMax], kq[kRecurMax];
    } tok;
};

__global__ __launch_bounds__(256) void prefill_recur_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const float* __restrict__ g, const float* __restrict__ beta, const int32_t* __restrict__ cu,
    int32_t* __restrict__ order, const float* initial_state, float* final_state,
    uint16_t* __restrict__ o, int N, int T, int H_qk, int H_v, float scale,
    const int32_t* __restrict__ state_idx, int P, int short_only, int flags) {
    __shared__ Smem sm;
    __shared__ int cnt[2];
    if (blockIdx.x == 0) {
        // the chunk kernel's schedule (not needed when no chunk kernel
        // follows), the number of sequences it runs and the check of
        // cu_seqlens, from one read of it
        bool bad = false;
        const int nlong =
            schedule_longest_first(cu, N, T, short_only ? nullptr : order, sm.sched_len, cnt, kRecurMax, &bad);
        if (threadIdx.x == 0) {
            order[N] = nlong;
            // the fault word: a short-only call that met a longer sequence
            // (skipped) sets bit 1, a malformed cu_seqlens bit 2; the chunk
            // kernel may set bit 0 later
            order[N + 1] = ((short_only && nlong > 0) ? 2 : 0) | (bad ? 4 : 0);
        }
        return;
    }
    constexpr int ROWS = NWAVE * ROWS_PER_WAVE;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int sub = lane / LPR, c = lane % LPR;
    const long units = (long)N * H_v * BPH;
    const size_t qk_stride = (size_t)H_qk * D, v_stride = (size_t)H_v * D;
    // A unit runs here if its sequence has at most kRecurMax tokens and its
    // state lies inside the pool; a workgroup walks slots s, s + stride, ...
    // (the units of one q/k head on one XCD).
    const long stride = gridDim.x - 1;
    const int grp = (H_v / H_qk) * BPH;
    auto next_unit = [&](long s) -> long {
        return recur_next_slot(s, stride, units, grp, BPH, H_v, cu, T, state_idx, P, kRecurMax);
    };
    // The fields of the unit in slot s: its state (state n, or pool slot
    // state_idx[n]), head, row block and tokens.
    typedef RecurUnit Unit;
    auto unit_at = [&](long s) -> Unit {
        return recur_unit_at(recur_slot_unit(s, units, grp), BPH, H_v, H_qk, cu, T, state_idx);
    };
    auto state_row = [&](const Unit& x) {
        const int row = x.blk * ROWS + wave * ROWS_PER_WAVE + sub;
        return ((size_t)x.shead * D + row) * D;
    };
    auto load_rows = [&](const Unit& x, f32x4_t (&r)[J]) {
        const size_t srow = state_row(x);
#pragma unroll
        for (int j = 0; j < J; ++j) {
            if (initial_state != nullptr)
                r[j] = __builtin_nontemporal_load(
                    reinterpret_cast<const f32x4_t*>(initial_state + srow + (j * LPR + c) * 4));
            else
                r[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
    };
    long ucur = next_unit(blockIdx.x - 1);
    f32x4_t s[J];
    if (ucur < units) load_rows(unit_at(ucur), s);
    while (ucur < units) {
        const Unit cur = unit_at(ucur);
        const long unxt = next_unit(ucur + stride);
        const int h = cur.h, hq = cur.hq, t0 = cur.t0, len = cur.len;
        const int row0 = cur.blk * ROWS;
        const int row = row0 + wave * ROWS_PER_WAVE + sub;
        // stage the tokens: 16 segments of 8 values per k or q row, 4 per v slice
        if (tid < len * (D / 8)) {
            const int t = tid / (D / 8), seg = tid - t * (D / 8);
            const size_t row = (size_t)(t0 + t) * qk_stride + (size_t)hq * D;
            const size_t src = row + seg * 8;
            uint4 kk = *reinterpret_cast<const uint4*>(k + src);
            uint4 qq = *reinterpret_cast<const uint4*>(q + src);
            if (flags & kFlagQkL2Norm) {
                kk = scale_bf16x8(kk, row_inv_norm<D>(k + row));
                qq = scale_bf16x8(qq, row_inv_norm<D>(q + row));
            }
            const uint32_t kw[4] = {kk.x, kk.y, kk.z, kk.w}, qw[4] = {qq.x, qq.y, qq.z, qq.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                sm.tok.k[t][seg * 8 + 2 * e] = bf16_to_f32(kw[e] & 0xFFFF);
                sm.tok.k[t][seg * 8 + 2 * e + 1] = bf16_to_f32(kw[e] >> 16);
                sm.tok.q[t][seg * 8 + 2 * e] = bf16_to_f32(qw[e] & 0xFFFF);
                sm.tok.q[t][seg * 8 + 2 * e + 1] = bf16_to_f32(qw[e] >> 16);
            }
        }
        if (tid < len * (ROWS / 8)) {
            const int t = tid / (ROWS / 8), seg = tid - t * (ROWS / 8);
            *reinterpret_cast<uint4*>(&sm.tok.v[t][seg * 8]) =
                *reinterpret_cast<const uint4*>(v + (size_t)(t0 + t) * v_stride + (size_t)h * D + row0 + seg * 8);
        }
        if (tid < len) {
            const float gi = g[(size_t)(t0 + tid) * H_v + h], bi = beta[(size_t)(t0 + tid) * H_v + h];
            const bool logits = (flags & kFlagGateLogits) != 0;
            sm.tok.alpha[tid] = fast_exp(logits ? gate_from_logit(gi) : gi);
            sm.tok.b[tid] = logits ? beta_from_logit(bi) : bi;
        }
        __syncthreads();
        // k . q per token, summed in the row layout below (8 tokens per wave)
        if (tid < 8 * len) {
            const int t = tid / LPR;
            float kq = 0.f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const f32x4_t kv4 = *reinterpret_cast<const f32x4_t*>(&sm.tok.k[t][(j * LPR + c) * 4]);
                const f32x4_t qv4 = *reinterpret_cast<const f32x4_t*>(&sm.tok.q[t][(j * LPR + c) * 4]);
#pragma unroll
                for (int e = 0; e < 4; ++e) kq = fmaf(kv4[e], qv4[e], kq);
            }
            kq = group_sum<LPR>(kq);
            if (c == 0) sm.tok.kq[t] = kq;
        }
        __syncthreads();
        // the next unit's state rows, in flight during this unit's token loop
        // (issued after the staging loads, which the counters retire in order)
        f32x4_t sn[J];
        if (unxt < units) load_rows(unit_at(unxt), sn);
        for (int t = 0; t < len; ++t) {
            f32x4_t kf[J], qf[J];
#pragma unroll
            for (int j = 0; j < J; ++j) {
                kf[j] = *reinterpret_cast<const f32x4_t*>(&sm.tok.k[t][(j * LPR + c) * 4]);
                qf[j] = *reinterpret_cast<const f32x4_t*>(&sm.tok.q[t][(j * LPR + c) * 4]);
            }
            const float alpha = sm.tok.alpha[t], bt = sm.tok.b[t], kq = sm.tok.kq[t];
            float kv = 0.f, sq = 0.f;
#pragma unroll
            for (int j = 0; j < J; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    kv = fmaf(s[j][e], kf[j][e], kv);
                    sq = fmaf(s[j][e], qf[j][e], sq);
                }
            kv = group_sum<LPR>(kv);
            sq = group_sum<LPR>(sq);
            const float uu = bt * (bf16_to_f32(sm.tok.v[t][row - row0]) - alpha * kv);
#pragma unroll
            for (int j = 0; j < J; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) s[j][e] = fmaf(alpha, s[j][e], uu * kf[j][e]);
            if (c == 0)
                o[(size_t)(t0 + t) * v_stride + (size_t)h * D + row] = f32_to_bf16(scale * fmaf(alpha, sq, uu * kq));
        }
        const size_t srow = state_row(cur);
#pragma unroll
        for (int j = 0; j < J; ++j)
            __builtin_nontemporal_store(s[j], reinterpret_cast<f32x4_t*>(final_state + srow + (j * LPR + c) * 4));
        if (unxt < units) {
#pragma unroll
            for (int j = 0; j < J; ++j) s[j] = sn[j];
        }
        ucur = unxt;
        __syncthreads();  // the staged tokens are read; the next unit may overwrite them
    }
}

}  // namespace recur

// Up to eight workgroups per compute unit, each walking (sequence, head, row
// block) units; block 0 writes the schedule.
hipError_t launch_prefill_recur(const PrefillArgs& a, int32_t* order, hipStream_t stream) {
    const long units = (long)a.N * a.H_v * recur::BPH;
    const long grid = 1 + std::max<long>(1, std::min<long>(units, 8L * device_compute_units()));
    hipLaunchKernelGGL(recur::prefill_recur_kernel, dim3((unsigned)grid), dim3(64 * recur::NWAVE), 0, stream,
                       (const uint16_t*)a.q, (const uint16_t*)a.k, (const uint16_t*)a.v, a.g, a.beta,
                       a.cu_seqlens, order, a.initial_state, a.final_state, (uint16_t*)a.o, a.N, a.T, a.H_qk,
                       a.H_v, a.scale, a.state_idx, a.P, a.short_only ? 1 : 0, a.flags);
    return hipGetLastError();
}

}  // namespace gdn
