// Pipelined chunk kernel of the prefill regime for d = 128, chunk 64 (the
// chunked form and its notation are described in gdn_prefill.hip).
//
// The per-chunk work splits into a state-independent part (stage q/k/v/g/beta,
// the gate prefix, the lower-triangular tiles of K K^T and Q K^T, masks and
// decays, T = (I + A)^-1 and T diag(beta), K^T) and a state-dependent part
// (K S0^T, Q S0^T, W, U, O and the state update).  Only the second part is
// sequential along a sequence.  One workgroup per (sequence, value head) runs
// both as a two-stage pipeline over chunks:
//
//   * 4 state waves: wave w owns value columns [32 w, 32 w + 32) of S^T in
//     fp32 MFMA accumulators and, in iteration c, runs the state-dependent
//     part of chunk c;
//   * 4 producer waves: in iteration c they build K^T of chunk c (which the
//     state waves need last) and then prepare every state-independent input of
//     chunk c + 1, loading chunk c + 2 into registers meanwhile.
//
// One workgroup barrier ends each iteration.  Inside an iteration the roles
// meet only through LDS counters: producers count "K^T of chunk c written",
// state waves count "done reading Q of chunk c" and "done reading V of chunk c"
// (Q and V have a single LDS buffer), and producers synchronise among
// themselves with a counter barrier.  Buffers written by producers for chunk
// c + 1 while state waves read chunk c (K, T diag(beta) hi/lo, the masked
// scores, the decays) are double-buffered by chunk parity.  Every wait is a
// bounded spin; LDS operations of a wave execute in order, so a counter
// increment issued after a wave's LDS stores (or reads) is observed only after
// those have executed.
#include "gdn_launch.h"
#include "gdn_mfma.h"

namespace gdn {
namespace pipe {

constexpr int D = 128, C = 64;
constexpr int NP = 4;                 // producer waves
constexpr int NDT = D / 16, NCT = C / 16;
constexpr int PD = D + 8;             // LDS pitch (bf16) of [C][D] and [D][C] arrays
constexpr int PC = C + 8;
constexpr int BP = 24;                // pitch (bf16) of a stored 16 x 16 block
constexpr int FP = 17;                // pitch (fp32) of a stored 16 x 16 block
constexpr int NBLK = NCT * (NCT + 1) / 2;   // lower-triangular 16 x 16 blocks (10)
constexpr int SEGS = D / 8;                 // 16-byte segments per q/k/v row
constexpr int PITEMS = C * SEGS / (64 * NP);  // staged segments per producer thread
constexpr int kSpinLimit = 1 << 20;

__device__ __forceinline__ constexpr int bidx(int i, int j) { return i * (i + 1) / 2 + j; }
// Private slot of diagonal block b (b >= w) for producer wave w < 3: wave 0 uses
// slots 0-3, wave 1 slots 4-6, wave 2 slots 7-8.
__device__ __forceinline__ constexpr int dslot(int w, int b) { return 4 * w - w * (w - 1) / 2 + (b - w); }

struct Smem {
    uint16_t kb[2][C][PD];            // K rows, by chunk parity
    uint16_t qb[C][PD];               // Q rows
    uint16_t vb[C][PD];               // V rows
    uint16_t kt[D][PC];               // K^T of the chunk the state waves work on
    uint16_t th[2][NBLK][16][BP];     // T diag(beta), bf16 hi, lower blocks
    uint16_t tl[2][NBLK][16][BP];     // T diag(beta), bf16 lo
    uint16_t pm[2][NBLK][16][BP];     // (M o Q K^T), bf16
    uint16_t zero[16][BP];            // stands in for blocks above the diagonal
    float a[NBLK][16][FP];            // A (strictly lower), producers only
    float t[NBLK][16][FP];            // diagonal blocks of T, private slots per producer wave
    float gam[NP][C];                 // per producer wave: gate prefix of its chunk
    float bet[NP][C];                 // per producer wave: beta of its chunk
    alignas(16) float eg[2][C];       // exp(gamma), by chunk parity
    alignas(16) float egl[2][C];      // exp(gamma_last - gamma), by chunk parity
    unsigned cnt[4];                  // producer barrier, K^T ready, Q free, V free
};

enum { CNT_PBAR = 0, CNT_KT = 1, CNT_QFREE = 2, CNT_VFREE = 3 };

// Count this wave (lane 0) into *ctr.  The compiler fence keeps the wave's
// earlier LDS accesses before the increment; the LDS executes them in order.
__device__ __forceinline__ void signal(unsigned* ctr, int lane) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (lane == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Wait until *ctr >= target (bounded: never spins forever).
__device__ __forceinline__ void wait_ge(unsigned* ctr, unsigned target) {
    for (int it = 0; it < kSpinLimit; ++it) {
        if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= target) break;
        __builtin_amdgcn_s_sleep(1);
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// A operand from a stored lower-triangular block matrix (row tile ct,
// contraction columns kc..kc+31, permuted order); blocks above the diagonal
// read the zero block.
__device__ __forceinline__ bf16x8_t blk_frag(const uint16_t (*blocks)[16][BP], const uint16_t (*zero)[BP],
                                             int ct, int kc, int m, int g) {
    const int j0 = kc >> 4;
    const uint16_t* p0 = &blocks[bidx(ct, j0)][m][4 * g];
    const uint16_t* p1 = (j0 + 1 <= ct) ? &blocks[bidx(ct, j0 + 1)][m][4 * g] : &zero[m][4 * g];
    const uint2 lo = *reinterpret_cast<const uint2*>(p0);
    const uint2 hi = *reinterpret_cast<const uint2*>(p1);
    uint4 u = {lo.x, lo.y, hi.x, hi.y};
    return __builtin_bit_cast(bf16x8_t, u);
}

// NS state waves (4 or 8), each owning D / NS value columns.
template <int NS>
__global__ __launch_bounds__(64 * (NS + NP)) void prefill_pipe_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const float* __restrict__ g, const float* __restrict__ beta, const int32_t* __restrict__ cu,
    const int32_t* __restrict__ order, const float* initial_state, float* final_state,
    uint16_t* __restrict__ o, int N, int H_qk, int H_v, float scale) {
    constexpr int NT = 64 * (NS + NP);  // threads per workgroup
    constexpr int VW = D / NS;          // value columns per state wave
    constexpr int NVT = VW / 16;        // 16-wide value tiles per state wave
    __shared__ Smem sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int m = lane & 15;
    const int gq = lane >> 4;

    const int item = logical_item(blockIdx.x, N * H_v);
    const int rank = item / H_v;
    const int h = item - rank * H_v;
    const int n = order[rank];
    const int hq = h / (H_v / H_qk);
    const int seq_beg = cu[n];
    const int seq_len = cu[n + 1] - seq_beg;
    const int nch = (seq_len + C - 1) / C;
    const size_t qk_stride = (size_t)H_qk * D;
    const size_t v_stride = (size_t)H_v * D;
    const size_t state_off = ((size_t)n * H_v + h) * D * D;

    if (tid < 4) sm.cnt[tid] = 0;
    for (int i = tid; i < 16 * BP; i += NT) (&sm.zero[0][0])[i] = 0;
    __syncthreads();

    if (wave < NS) {
        // ======================= state waves ===================================
        const int vcol0 = wave * VW;
        f32x4_t st[NDT][NVT];  // st[dt][vt][i] = S[v][d], v = vcol0 + 16 vt + m, d = 16 dt + 4 gq + i
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int vt = 0; vt < NVT; ++vt) {
                if (initial_state != nullptr) {
                    const float4 s4 = *reinterpret_cast<const float4*>(
                        initial_state + state_off + (size_t)(vcol0 + 16 * vt + m) * D + 16 * dt + 4 * gq);
                    st[dt][vt] = f32x4_t{s4.x, s4.y, s4.z, s4.w};
                } else {
                    st[dt][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                }
            }
        __syncthreads();  // producers have prepared chunk 0

        for (int c = 0; c < nch; ++c) {
            const int par = c & 1;
            const int L = min(C, seq_len - c * C);
            const int t0 = seq_beg + c * C;
            // K S0^T (S0 hi + lo) and Q S0^T (S0 hi)
            f32x4_t ks[NCT][NVT], qs[NCT][NVT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) {
                    ks[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                    qs[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
            for (int kk = 0; kk < D; kk += 32) {
                bf16x8_t bh[NVT], bl[NVT];
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) acc_frag<32>(st[kk / 16][vt], st[kk / 16 + 1][vt], bh[vt], bl[vt]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const bf16x8_t ak = lds_frag_perm<32>(&sm.kb[par][16 * ct + m][0], kk, gq);
                    const bf16x8_t aq = lds_frag_perm<32>(&sm.qb[16 * ct + m][0], kk, gq);
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        ks[ct][vt] = mma(ak, bh[vt], ks[ct][vt]);
                        ks[ct][vt] = mma(ak, bl[vt], ks[ct][vt]);
                        qs[ct][vt] = mma(aq, bh[vt], qs[ct][vt]);
                    }
                }
            }
            signal(&sm.cnt[CNT_QFREE], lane);
            // W = V - diag(exp(gamma)) K S0^T (in ks); O starts as diag(exp(gamma)) Q S0^T (in qs)
            f32x4_t egr[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) egr[ct] = *reinterpret_cast<const f32x4_t*>(&sm.eg[par][16 * ct + 4 * gq]);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float vv = bf16_to_f32(sm.vb[16 * ct + 4 * gq + i][vcol0 + 16 * vt + m]);
                        ks[ct][vt][i] = fmaf(-egr[ct][i], ks[ct][vt][i], vv);
                        qs[ct][vt][i] *= egr[ct][i];
                    }
            signal(&sm.cnt[CNT_VFREE], lane);
            // U = T diag(beta) W  (hi*hi + hi*lo + lo*hi)
            f32x4_t uu[NCT][NVT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) uu[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < C; kc += 32) {
                bf16x8_t wh[NVT], wl[NVT];
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) acc_frag<32>(ks[kc / 16][vt], ks[kc / 16 + 1][vt], wh[vt], wl[vt]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    if (kc > 16 * ct + 15) continue;
                    const bf16x8_t ah = blk_frag(sm.th[par], sm.zero, ct, kc, m, gq);
                    const bf16x8_t al = blk_frag(sm.tl[par], sm.zero, ct, kc, m, gq);
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        uu[ct][vt] = mma(ah, wh[vt], uu[ct][vt]);
                        uu[ct][vt] = mma(ah, wl[vt], uu[ct][vt]);
                        uu[ct][vt] = mma(al, wh[vt], uu[ct][vt]);
                    }
                }
            }
            // O += (M o Q K^T) U  (U hi), then store
#pragma unroll
            for (int kc = 0; kc < C; kc += 32) {
                bf16x8_t uh[NVT];
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) uh[vt] = acc_frag_hi<32>(uu[kc / 16][vt], uu[kc / 16 + 1][vt]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    if (kc > 16 * ct + 15) continue;
                    const bf16x8_t ap = blk_frag(sm.pm[par], sm.zero, ct, kc, m, gq);
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) qs[ct][vt] = mma(ap, uh[vt], qs[ct][vt]);
                }
            }
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = 16 * ct + 4 * gq + i;
                    if (row < L) {
                        uint16_t* orow = o + (size_t)(t0 + row) * v_stride + (size_t)h * D + vcol0 + m;
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt) orow[16 * vt] = f32_to_bf16(scale * qs[ct][vt][i]);
                    }
                }
            // S^T = exp(gamma_last) S^T + K^T (diag(exp(gamma_last - gamma)) U)   (hi + lo)
            f32x4_t eglv[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) eglv[ct] = *reinterpret_cast<const f32x4_t*>(&sm.egl[par][16 * ct + 4 * gq]);
            const float eg_last = sm.eg[par][C - 1];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) st[dt][vt] *= eg_last;
            wait_ge(&sm.cnt[CNT_KT], (unsigned)(NP * (c + 1)));
#pragma unroll
            for (int kc = 0; kc < C; kc += 32) {
                bf16x8_t uth[NVT], utl[NVT];
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt)
                    acc_frag<32>(uu[kc / 16][vt] * eglv[kc / 16], uu[kc / 16 + 1][vt] * eglv[kc / 16 + 1], uth[vt], utl[vt]);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    const bf16x8_t a = lds_frag_perm<32>(&sm.kt[16 * dt + m][0], kc, gq);
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        st[dt][vt] = mma(a, uth[vt], st[dt][vt]);
                        st[dt][vt] = mma(a, utl[vt], st[dt][vt]);
                    }
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int vt = 0; vt < NVT; ++vt) {
                const float4 s4 = {st[dt][vt][0], st[dt][vt][1], st[dt][vt][2], st[dt][vt][3]};
                *reinterpret_cast<float4*>(final_state + state_off + (size_t)(vcol0 + 16 * vt + m) * D +
                                           16 * dt + 4 * gq) = s4;
            }
    } else {
        // ======================= producer waves ================================
        const int pw = wave - NS;
        const int ptid = tid - 64 * NS;
        unsigned pbar_gen = 0;
        auto pbar = [&]() {
            ++pbar_gen;
            signal(&sm.cnt[CNT_PBAR], lane);
            wait_ge(&sm.cnt[CNT_PBAR], (unsigned)(NP * pbar_gen));
        };
        // chunk inputs held in registers until staged
        uint4 rk[PITEMS], rq[PITEMS], rv[PITEMS];
        float rg = 0.f, rb = 0.f;
        auto load_chunk = [&](int x) {
            const int Lx = min(C, seq_len - x * C);
            const int tb = seq_beg + x * C;
#pragma unroll
            for (int it = 0; it < PITEMS; ++it) {
                const int i = ptid + it * 64 * NP;
                const int r = i / SEGS, seg = i - r * SEGS;
                rk[it] = rq[it] = rv[it] = uint4{0, 0, 0, 0};
                if (r < Lx) {
                    const size_t tq = (size_t)(tb + r) * qk_stride + (size_t)hq * D + seg * 8;
                    rk[it] = *reinterpret_cast<const uint4*>(k + tq);
                    rq[it] = *reinterpret_cast<const uint4*>(q + tq);
                    rv[it] = *reinterpret_cast<const uint4*>(v + (size_t)(tb + r) * v_stride + (size_t)h * D + seg * 8);
                }
            }
            const bool in = lane < Lx;
            rg = in ? g[(size_t)(tb + lane) * H_v + h] : 0.f;
            rb = in ? beta[(size_t)(tb + lane) * H_v + h] : 0.f;
        };
        auto build_kt = [&](int par) {
            for (int i = ptid; i < (C / 2) * SEGS; i += 64 * NP) {
                const int p = i % (C / 2), seg = i / (C / 2);
                const uint4 r0 = *reinterpret_cast<const uint4*>(&sm.kb[par][2 * p][seg * 8]);
                const uint4 r1 = *reinterpret_cast<const uint4*>(&sm.kb[par][2 * p + 1][seg * 8]);
                const uint32_t a[4] = {r0.x, r0.y, r0.z, r0.w};
                const uint32_t b[4] = {r1.x, r1.y, r1.z, r1.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    *reinterpret_cast<uint32_t*>(&sm.kt[seg * 8 + 2 * j][2 * p]) = (a[j] & 0xFFFFu) | (b[j] << 16);
                    *reinterpret_cast<uint32_t*>(&sm.kt[seg * 8 + 2 * j + 1][2 * p]) = (a[j] >> 16) | (b[j] & 0xFFFF0000u);
                }
            }
        };
        // Prepare every state-independent input of chunk x from the registers;
        // `free_target` is what the Q-free / V-free counters must reach before
        // the single Q and V buffers may be overwritten.
        auto prepare = [&](int x, unsigned free_target) {
            const int par = x & 1;
            // stage K, gate prefix, beta
#pragma unroll
            for (int it = 0; it < PITEMS; ++it) {
                const int i = ptid + it * 64 * NP;
                const int r = i / SEGS, seg = i - r * SEGS;
                *reinterpret_cast<uint4*>(&sm.kb[par][r][seg * 8]) = rk[it];
            }
            float gx = rg;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const float y = __shfl_up(gx, d);
                if (lane >= d) gx += y;
            }
            const float glast = __shfl(gx, C - 1);
            sm.gam[pw][lane] = gx;
            sm.bet[pw][lane] = rb;
            if (pw == 0) {
                sm.eg[par][lane] = fast_exp(gx);
                sm.egl[par][lane] = fast_exp(glast - gx);
            }
            pbar();  // K of chunk x complete
            // G = K K^T tiles -> A (fp32)
            for (int tri = pw; tri < NBLK; tri += NP) {
                int ti = 0;
                while ((ti + 1) * (ti + 2) / 2 <= tri) ++ti;
                const int tj = tri - ti * (ti + 1) / 2;
                f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
                const uint16_t* arow = &sm.kb[par][16 * ti + m][0];
                const uint16_t* brow = &sm.kb[par][16 * tj + m][0];
#pragma unroll
                for (int kk = 0; kk < D; kk += 32)
                    acc = mma(lds_frag_nat<32>(arow, kk, gq), lds_frag_nat<32>(brow, kk, gq), acc);
                const int col = 16 * tj + m;
                const float gcol = sm.gam[pw][col];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = 16 * ti + 4 * gq + i;
                    const float dec = fast_exp(sm.gam[pw][row] - gcol);
                    sm.a[tri][4 * gq + i][m] = col < row ? sm.bet[pw][row] * dec * acc[i] : 0.f;
                }
            }
            pbar();  // A complete
            // T = (I + A)^-1.  Every producer wave inverts all four diagonal blocks
            // at once (lane 16 b + m: column m of block b, forward substitution
            // with each row sum split over two chains), writes T diag(beta) of
            // block pw, and keeps the diagonal blocks its own sweep needs in a
            // private LDS slot.  Wave j < 3 then forms the blocks below the
            // diagonal of block column j one after another,
            //     T_bj = -D_b sum_{kb=j}^{b-1} A_{b,kb} T_{kb,j},   T_jj = D_j,
            // keeping each result in its accumulator (as a B operand it supplies
            // contraction row 4 gq + s at step s).  A is complete and each wave
            // reads only its own slots, so no producer barrier is needed here.
            {
                const int b = lane >> 4;
                const int bb = bidx(b, b);
                float xs[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float a0 = (r == m) ? 1.f : 0.f, a1 = 0.f;
#pragma unroll
                    for (int i = 0; i < r; ++i) {
                        if (i & 1) a1 = fmaf(-sm.a[bb][r][i], xs[i], a1);
                        else a0 = fmaf(-sm.a[bb][r][i], xs[i], a0);
                    }
                    xs[r] = a0 + a1;
                }
                if (b == pw) {
                    const float bcol = sm.bet[pw][16 * b + m];
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        split_bf16(xs[r] * bcol, sm.th[par][bb][r][m], sm.tl[par][bb][r][m]);
                }
                if (pw < NCT - 1 && b >= pw) {
                    float (*slot)[FP] = sm.t[dslot(pw, b)];
#pragma unroll
                    for (int r = 0; r < 16; ++r) slot[r][m] = xs[r];
                }
            }
            if (pw < NCT - 1) {
                const int j = pw;
                const float bcol = sm.bet[pw][16 * j + m];
                const float (*dj)[FP] = sm.t[dslot(j, j)];
                f32x4_t tz[NCT];
#pragma unroll
                for (int bi = 1; bi < NCT; ++bi) {
                    tz[bi] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                    if (bi <= j) continue;
                    f32x4_t y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        y = mma_f32(sm.a[bidx(bi, j)][m][4 * gq + s], dj[4 * gq + s][m], y);
#pragma unroll
                    for (int kb = 1; kb < bi; ++kb) {
                        if (kb <= j) continue;
#pragma unroll
                        for (int s = 0; s < 4; ++s) y = mma_f32(sm.a[bidx(bi, kb)][m][4 * gq + s], tz[kb][s], y);
                    }
                    const float (*db)[FP] = sm.t[dslot(j, bi)];
                    f32x4_t z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int s = 0; s < 4; ++s) z = mma_f32(-db[m][4 * gq + s], y[s], z);
                    tz[bi] = z;
                    const int ob = bidx(bi, j);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        split_bf16(z[i] * bcol, sm.th[par][ob][4 * gq + i][m], sm.tl[par][ob][4 * gq + i][m]);
                }
            }
            // stage Q and V once the state waves are done with the previous chunk's
            wait_ge(&sm.cnt[CNT_QFREE], free_target);
#pragma unroll
            for (int it = 0; it < PITEMS; ++it) {
                const int i = ptid + it * 64 * NP;
                const int r = i / SEGS, seg = i - r * SEGS;
                *reinterpret_cast<uint4*>(&sm.qb[r][seg * 8]) = rq[it];
            }
            wait_ge(&sm.cnt[CNT_VFREE], free_target);
#pragma unroll
            for (int it = 0; it < PITEMS; ++it) {
                const int i = ptid + it * 64 * NP;
                const int r = i / SEGS, seg = i - r * SEGS;
                *reinterpret_cast<uint4*>(&sm.vb[r][seg * 8]) = rv[it];
            }
            pbar();  // Q of chunk x complete
            // P = Q K^T tiles -> masked scores (bf16)
            for (int tri = pw; tri < NBLK; tri += NP) {
                int ti = 0;
                while ((ti + 1) * (ti + 2) / 2 <= tri) ++ti;
                const int tj = tri - ti * (ti + 1) / 2;
                f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
                const uint16_t* arow = &sm.qb[16 * ti + m][0];
                const uint16_t* brow = &sm.kb[par][16 * tj + m][0];
#pragma unroll
                for (int kk = 0; kk < D; kk += 32)
                    acc = mma(lds_frag_nat<32>(arow, kk, gq), lds_frag_nat<32>(brow, kk, gq), acc);
                const int col = 16 * tj + m;
                const float gcol = sm.gam[pw][col];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = 16 * ti + 4 * gq + i;
                    const float dec = fast_exp(sm.gam[pw][row] - gcol);
                    sm.pm[par][tri][4 * gq + i][m] = f32_to_bf16(col <= row ? dec * acc[i] : 0.f);
                }
            }
        };

        if (nch > 0) {
            load_chunk(0);
            prepare(0, 0u);
            if (nch > 1) load_chunk(1);
        }
        __syncthreads();  // chunk 0 prepared
        for (int c = 0; c < nch; ++c) {
            build_kt(c & 1);
            signal(&sm.cnt[CNT_KT], lane);
            if (c + 1 < nch) {
                prepare(c + 1, (unsigned)(NS * (c + 1)));
                if (c + 2 < nch) load_chunk(c + 2);
            }
            __syncthreads();
        }
    }
}

}  // namespace pipe

#ifndef GDN_PIPE_STATE_WAVES
#define GDN_PIPE_STATE_WAVES 4
#endif

hipError_t launch_prefill_pipe(const PrefillArgs& a, const int32_t* order, hipStream_t stream) {
    constexpr int NS = GDN_PIPE_STATE_WAVES;
    hipLaunchKernelGGL(pipe::prefill_pipe_kernel<NS>, dim3((unsigned)(a.N * a.H_v)), dim3(64 * (NS + pipe::NP)),
                       0, stream, (const uint16_t*)a.q, (const uint16_t*)a.k, (const uint16_t*)a.v, a.g,
                       a.beta, a.cu_seqlens, order, a.initial_state, a.final_state, (uint16_t*)a.o,
                       a.N, a.H_qk, a.H_v, a.scale);
    return hipGetLastError();
}

}  // namespace gdn
