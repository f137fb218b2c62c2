// Prefill regime of the gated delta rule (paper: appendix "Operator Background
// and Mathematical Definitions", subsection "Gated Delta Net": the whole
// sequence is evaluated and both outputs and the final state are returned, by
// chunked matrix operations that apply the log-domain gate consistently).
//
// Chunked form used here (an exact regrouping of the token recurrence).  For a
// chunk of rows r = 0..C-1 of one (sequence, value head), gamma_r = running sum
// of g inside the chunk, S0 = state entering the chunk (d_v x d_k):
//     A_ri = beta_r exp(gamma_r - gamma_i) (k_r . k_i)   (i < r, else 0)
//     T    = (I + A)^-1                                  (unit lower triangular)
//     W    = V - diag(exp(gamma)) K S0^T
//     U    = T diag(beta) W
//     O    = scale (diag(exp(gamma)) Q S0^T + (M o Q K^T) U),
//            M_ri = exp(gamma_r - gamma_i) for i <= r, else 0
//     S    = exp(gamma_{C-1}) S0 + (diag(exp(gamma_{C-1} - gamma)) U)^T K
// Chunks start at each sequence's first token; the ragged last chunk is padded
// with q = k = v = 0, g = 0, beta = 0 rows, which contribute exactly nothing.
//
// Work decomposition (gfx950, one workgroup per (sequence, value head)):
//   * NW waves; wave w owns value columns [w VW, (w+1) VW) of the state, held
//     transposed (S^T, d x v) in fp32 MFMA accumulators across all chunks.
//   * Per chunk: stage Q, K, V rows in LDS (row-major bf16) and K^T; the gate
//     prefix sum; the lower-triangular tiles of K K^T and Q K^T on bf16 MFMA
//     (exact bf16 operands); masks and decays in fp32; T by 16 x 16 diagonal
//     forward substitution plus fp32-MFMA block levels; T diag(beta) stored as
//     a bf16 hi + lo pair.
//   * State-dependent part per wave on bf16 MFMA with fp32 accumulation.
//     Operands that are computed fp32 values feeding the state are split into
//     hi + lo bf16 (x = hi + lo to ~2^-17): S0 in K S0^T, W and T diag(beta)
//     in U (hi*hi + hi*lo + lo*hi), and U in the state update.  The output-only
//     products (Q S0^T, (M o QK^T) U) use the hi parts.
//   * Accumulator tiles feed the next MFMA directly as B operands: for a
//     32-deep contraction slice, lane group g holds accumulator rows 4g..4g+3
//     of two 16-row tiles, and the matching A operand is read from LDS in the
//     same permuted contraction order (two 8-byte reads per lane).
#include "gdn_launch.h"
#include "gdn_schedule.h"
#include "gdn_mfma.h"

namespace gdn {

// --- configuration -------------------------------------------------------------
template <int D, int C>
struct Cfg {
    static constexpr int NW = (D == 128) ? 8 : 1;  // waves per workgroup (2 per SIMD for D = 128)
    static constexpr int NT = 64 * NW;             // threads
    static constexpr int VW = D / NW;              // value columns per wave (16)
    static constexpr int NVT = VW / 16;            // 16-wide value tiles per wave
    static constexpr int NDT = D / 16;             // 16-row d tiles
    static constexpr int NCT = C / 16;             // 16-row chunk tiles
    static constexpr int KD = D >= 32 ? 32 : 16;   // contraction step over d
    static constexpr int KC = C >= 32 ? 32 : 16;   // contraction step over chunk rows
    static constexpr int PD = D + 8;               // LDS pitch (bf16) of [C][D] arrays
    static constexpr int PC = C + 8;               // LDS pitch (bf16) of [.][C] arrays
    static constexpr int PF = C + 4;               // LDS pitch (fp32) of [C][C] arrays
    static constexpr int SEGS = D / 8;             // 16-byte segments per q/k/v row
    static constexpr int ITEMS = (C * SEGS + NT - 1) / NT;  // staged segments per thread
    static_assert(NW >= NCT, "one wave per diagonal 16x16 block of T");
    static_assert(NVT >= 1, "value tile of 16 columns");
};

template <int D, int C>
struct Smem {
    typedef Cfg<D, C> P;
    uint16_t q[C][P::PD];
    uint16_t k[C][P::PD];
    uint16_t v[C][P::PD];
    uint16_t kt[D][P::PC];   // K^T
    uint16_t th[C][P::PC];   // T diag(beta), bf16 hi
    uint16_t tl[C][P::PC];   // T diag(beta), bf16 lo
    uint16_t pm[C][P::PC];   // (M o Q K^T), bf16
    union {
        struct {
            float a[C][P::PF];  // A (strictly lower)
            float t[C][P::PF];  // T (lower, unit diagonal)
        } f;
        uint16_t o[C][P::PD];   // output staging
    } u;
    alignas(16) float gam[C];   // gamma (running sum of g)
    alignas(16) float eg[C];    // exp(gamma)
    alignas(16) float egl[C];   // exp(gamma_last - gamma)
    float beta[C];
    float graw[C];
};

// --- schedule: sequences by length, longest first (ties by index) ---------------
__global__ __launch_bounds__(256) void prefill_schedule_kernel(const int32_t* __restrict__ cu,
                                                               int N, int T, int32_t* __restrict__ order) {
    __shared__ int len[kSortMax];
    __shared__ int cnt[2];
    bool bad = false;
    schedule_longest_first(cu, N, T, order, len, cnt, 0, &bad);
    // the fault word: no waits here, so only bit 2 (a malformed cu_seqlens)
    if (threadIdx.x == 0) order[N + 1] = bad ? 4 : 0;
}

// --- the chunk kernel ----------------------------------------------------------
template <int D, int C>
__global__ __launch_bounds__((Cfg<D, C>::NT)) void prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, const int32_t* __restrict__ cu,
    const int32_t* __restrict__ order, const float* initial_state, float* final_state,
    uint16_t* __restrict__ o, int N, int T, int H_qk, int H_v, float scale,
    const int32_t* __restrict__ state_idx, int P_slots, int flags) {
    typedef Cfg<D, C> P;
    constexpr int KD = P::KD, KC = P::KC;
    typedef typename Frag<KD>::type FD;
    typedef typename Frag<KC>::type FC;
    __shared__ Smem<D, C> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int m = lane & 15;  // row / column within a 16x16 tile
    const int gq = lane >> 4; // lane group (0..3)

    const int item = logical_item(blockIdx.x, N * H_v);
    const int rank = item / H_v;
    const int h = item - rank * H_v;
    const int n = order[rank];
    const int hq = h / (H_v / H_qk);
    const SeqSpan sp = seq_span(cu, n, T);
    const int seq_beg = sp.beg;
    const int seq_len = sp.len;
    const int vcol0 = wave * P::VW;
    // the state of sequence n: state n, or pool slot state_idx[n] (outside the
    // pool: the sequence is skipped)
    long slot = n;
    if (state_idx != nullptr) {
        slot = state_idx[n];
        if (slot < 0 || slot >= P_slots) return;
    }

    // State S^T (d x v) for this wave's value columns, fp32 accumulators:
    // st[dt][vt][i] = S[v][d], v = vcol0 + 16 vt + m, d = 16 dt + 4 gq + i.
    f32x4_t st[P::NDT][P::NVT];
    const size_t state_off = ((size_t)slot * H_v + h) * D * D;
#pragma unroll
    for (int dt = 0; dt < P::NDT; ++dt)
#pragma unroll
        for (int vt = 0; vt < P::NVT; ++vt) {
            if (initial_state != nullptr) {
                const float4 s4 = *reinterpret_cast<const float4*>(
                    initial_state + state_off + (size_t)(vcol0 + 16 * vt + m) * D + 16 * dt + 4 * gq);
                st[dt][vt] = f32x4_t{s4.x, s4.y, s4.z, s4.w};
            } else {
                st[dt][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
        }

    // Blocks strictly above the diagonal of T diag(beta) and of the masked
    // scores stay zero for the whole kernel; the diagonal blocks are rewritten
    // (upper part included) every chunk.
    for (int i = tid; i < C * C; i += P::NT) {
        const int r = i / C, cc = i - r * C;
        if ((cc >> 4) > (r >> 4)) { sm.th[r][cc] = 0; sm.tl[r][cc] = 0; sm.pm[r][cc] = 0; }
    }

    const size_t qk_stride = (size_t)H_qk * D;
    const size_t v_stride = (size_t)H_v * D;

    // Chunk inputs are loaded into registers one chunk ahead (the loads of chunk
    // c+1 are in flight while chunk c computes) and written to LDS at the top of
    // the next iteration.  Rows past the sequence end are zero, with g = beta = 0.
    uint4 pq[P::ITEMS], pk[P::ITEMS], pv[P::ITEMS];
    float pg = 0.f, pb = 0.f;
    auto load_chunk = [&](int cbeg) {
        const int Lc = min(C, seq_len - cbeg);
        const int tb = seq_beg + cbeg;
#pragma unroll
        for (int it = 0; it < P::ITEMS; ++it) {
            const int i = tid + it * P::NT;
            const int r = i / P::SEGS, seg = i - r * P::SEGS;
            pq[it] = pk[it] = pv[it] = uint4{0, 0, 0, 0};
            if (i < C * P::SEGS && r < Lc) {
                const size_t row = (size_t)(tb + r) * qk_stride + (size_t)hq * D;
                const size_t tq = row + seg * 8;
                pq[it] = *reinterpret_cast<const uint4*>(q + tq);
                pk[it] = *reinterpret_cast<const uint4*>(k + tq);
                if (flags & kFlagQkL2Norm) {
                    pq[it] = scale_bf16x8(pq[it], row_inv_norm<D>(q + row));
                    pk[it] = scale_bf16x8(pk[it], row_inv_norm<D>(k + row));
                }
                pv[it] = *reinterpret_cast<const uint4*>(v + (size_t)(tb + r) * v_stride + (size_t)h * D + seg * 8);
            }
        }
        if (tid < C) {
            const bool in = tid < Lc;
            pg = in ? g[(size_t)(tb + tid) * H_v + h] : 0.f;
            pb = in ? beta[(size_t)(tb + tid) * H_v + h] : 0.f;
            if (in && (flags & kFlagGateLogits)) {
                pg = gate_from_logit(pg);
                pb = beta_from_logit(pb);
            }
        }
    };
    if (seq_len > 0) load_chunk(0);

    for (int c0 = 0; c0 < seq_len; c0 += C) {
        const int L = min(C, seq_len - c0);
        const int t0 = seq_beg + c0;

        // ---- stage the chunk ---------------------------------------------------
        // No wave reads sm.q/k/v/graw/beta after the previous chunk's output
        // barrier, so they can be overwritten here.
#pragma unroll
        for (int it = 0; it < P::ITEMS; ++it) {
            const int i = tid + it * P::NT;
            const int r = i / P::SEGS, seg = i - r * P::SEGS;
            if (i < C * P::SEGS) {
                *reinterpret_cast<uint4*>(&sm.q[r][seg * 8]) = pq[it];
                *reinterpret_cast<uint4*>(&sm.k[r][seg * 8]) = pk[it];
                *reinterpret_cast<uint4*>(&sm.v[r][seg * 8]) = pv[it];
            }
        }
        if (tid < C) {
            sm.graw[tid] = pg;
            sm.beta[tid] = pb;
        }
        __syncthreads();
        if (c0 + C < seq_len) load_chunk(c0 + C);

        // ---- gate prefix, K^T, raw score tiles -----------------------------------
        if (wave == 0) {
            float x = lane < C ? sm.graw[lane] : 0.f;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const float y = __shfl_up(x, d);
                if (lane >= d) x += y;
            }
            const float last = __shfl(x, C - 1);
            if (lane < C) {
                sm.gam[lane] = x;
                sm.eg[lane] = fast_exp(x);
                sm.egl[lane] = fast_exp(last - x);
            }
        }
        for (int i = tid; i < (C / 2) * (D / 8); i += P::NT) {
            const int p = i % (C / 2), seg = i / (C / 2);
            const uint4 r0 = *reinterpret_cast<const uint4*>(&sm.k[2 * p][seg * 8]);
            const uint4 r1 = *reinterpret_cast<const uint4*>(&sm.k[2 * p + 1][seg * 8]);
            const uint32_t a[4] = {r0.x, r0.y, r0.z, r0.w};
            const uint32_t b[4] = {r1.x, r1.y, r1.z, r1.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                *reinterpret_cast<uint32_t*>(&sm.kt[seg * 8 + 2 * j][2 * p]) =
                    (a[j] & 0xFFFFu) | (b[j] << 16);
                *reinterpret_cast<uint32_t*>(&sm.kt[seg * 8 + 2 * j + 1][2 * p]) =
                    (a[j] >> 16) | (b[j] & 0xFFFF0000u);
            }
        }
        // lower-triangular 16x16 tiles of G = K K^T (job < NTRI) and P = Q K^T
        constexpr int NTRI = P::NCT * (P::NCT + 1) / 2;
        constexpr int NJOB = 2 * NTRI;
        constexpr int JPW = (NJOB + P::NW - 1) / P::NW;
        f32x4_t gp[JPW];
#pragma unroll
        for (int jj = 0; jj < JPW; ++jj) {
            gp[jj] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            const int job = wave + jj * P::NW;
            if (job < NJOB) {
                const int tri = job % NTRI;
                int ti = 0;
                while ((ti + 1) * (ti + 2) / 2 <= tri) ++ti;
                const int tj = tri - ti * (ti + 1) / 2;
                const uint16_t* arow = (job < NTRI ? &sm.k[0][0] : &sm.q[0][0]) + (16 * ti + m) * P::PD;
                const uint16_t* brow = &sm.k[16 * tj + m][0];
#pragma unroll
                for (int kk = 0; kk < D; kk += KD)
                    gp[jj] = mma(lds_frag_nat<KD>(arow, kk, gq), lds_frag_nat<KD>(brow, kk, gq), gp[jj]);
            }
        }
        __syncthreads();

        // ---- masks and decays: A (fp32) and M o Q K^T (bf16) ----------------------
#pragma unroll
        for (int jj = 0; jj < JPW; ++jj) {
            const int job = wave + jj * P::NW;
            if (job < NJOB) {
                const int tri = job % NTRI;
                int ti = 0;
                while ((ti + 1) * (ti + 2) / 2 <= tri) ++ti;
                const int tj = tri - ti * (ti + 1) / 2;
                const int col = 16 * tj + m;
                const float gcol = sm.gam[col];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = 16 * ti + 4 * gq + i;
                    const float dec = fast_exp(sm.gam[row] - gcol);
                    if (job < NTRI) {
                        sm.u.f.a[row][col] = col < row ? sm.beta[row] * dec * gp[jj][i] : 0.f;
                    } else {
                        sm.pm[row][col] = f32_to_bf16(col <= row ? dec * gp[jj][i] : 0.f);
                    }
                }
            }
        }
        __syncthreads();

        // ---- T = (I + A)^-1 -------------------------------------------------------
        // diagonal blocks by forward substitution: wave w, lane j < 16 -> column j
        // of block w.
        if (wave < P::NCT) {
            const int b = wave;
            float x[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float acc = (r == m) ? 1.f : 0.f;
#pragma unroll
                for (int i = 0; i < r; ++i) acc = fmaf(-sm.u.f.a[16 * b + r][16 * b + i], x[i], acc);
                x[r] = acc;
            }
            if (lane < 16) {
                const float bcol = sm.beta[16 * b + m];
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    sm.u.f.t[16 * b + r][16 * b + m] = x[r];
                    split_bf16(x[r] * bcol, sm.th[16 * b + r][16 * b + m], sm.tl[16 * b + r][16 * b + m]);
                }
            }
        }
        __syncthreads();
        // off-diagonal blocks, level by level: T_bj = -T_bb sum_{k=j}^{b-1} A_bk T_kj
#pragma unroll
        for (int lev = 1; lev < P::NCT; ++lev) {
            const int j = wave;
            const int b = j + lev;
            if (b < P::NCT) {  // waves j < NCT - lev; the others only meet the barrier
                f32x4_t y = {0.f, 0.f, 0.f, 0.f};
                for (int kb = j; kb < b; ++kb) {
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        y = mma_f32(sm.u.f.a[16 * b + m][16 * kb + 4 * s + gq],
                                    sm.u.f.t[16 * kb + 4 * s + gq][16 * j + m], y);
                }
                // y is an accumulator: lane (n = m, group gq) holds Y[4 gq + i][n].  As
                // the B operand of step s it supplies contraction row 4 gq + s.
                f32x4_t z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    z = mma_f32(-sm.u.f.t[16 * b + m][16 * b + 4 * gq + s], y[s], z);
                const float bcol = sm.beta[16 * j + m];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int row = 16 * b + 4 * gq + i;
                    sm.u.f.t[row][16 * j + m] = z[i];
                    split_bf16(z[i] * bcol, sm.th[row][16 * j + m], sm.tl[row][16 * j + m]);
                }
            }
            __syncthreads();
        }

        // ---- state-dependent part (per wave, its value columns) --------------------
        f32x4_t ks[P::NCT][P::NVT], qs[P::NCT][P::NVT];
#pragma unroll
        for (int ct = 0; ct < P::NCT; ++ct)
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt) {
                ks[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                qs[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
        // K S0^T (S0 hi + lo) and Q S0^T (S0 hi)
#pragma unroll
        for (int kk = 0; kk < D; kk += KD) {
            FD bh[P::NVT], bl[P::NVT];
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt)
                acc_frag<KD>(st[kk / 16][vt], st[(kk / 16) + (KD == 32 ? 1 : 0)][vt], bh[vt], bl[vt]);
#pragma unroll
            for (int ct = 0; ct < P::NCT; ++ct) {
                const FD ak = lds_frag_perm<KD>(&sm.k[16 * ct + m][0], kk, gq);
                const FD aq = lds_frag_perm<KD>(&sm.q[16 * ct + m][0], kk, gq);
#pragma unroll
                for (int vt = 0; vt < P::NVT; ++vt) {
                    ks[ct][vt] = mma(ak, bh[vt], ks[ct][vt]);
                    ks[ct][vt] = mma(ak, bl[vt], ks[ct][vt]);
                    qs[ct][vt] = mma(aq, bh[vt], qs[ct][vt]);
                }
            }
        }
        // W = V - diag(exp(gamma)) K S0^T   (in place of ks)
        // O starts as diag(exp(gamma)) Q S0^T (in place of qs)
        f32x4_t egr[P::NCT];
#pragma unroll
        for (int ct = 0; ct < P::NCT; ++ct) egr[ct] = *reinterpret_cast<const f32x4_t*>(&sm.eg[16 * ct + 4 * gq]);
#pragma unroll
        for (int ct = 0; ct < P::NCT; ++ct)
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float vv = bf16_to_f32(sm.v[16 * ct + 4 * gq + i][vcol0 + 16 * vt + m]);
                    ks[ct][vt][i] = fmaf(-egr[ct][i], ks[ct][vt][i], vv);
                    qs[ct][vt][i] *= egr[ct][i];
                }
        // U = T diag(beta) W   (three bf16 products: hi*hi + hi*lo + lo*hi)
        f32x4_t uu[P::NCT][P::NVT];
#pragma unroll
        for (int ct = 0; ct < P::NCT; ++ct)
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt) uu[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < C; kc += KC) {
            FC wh[P::NVT], wl[P::NVT];
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt)
                acc_frag<KC>(ks[kc / 16][vt], ks[(kc / 16) + (KC == 32 ? 1 : 0)][vt], wh[vt], wl[vt]);
#pragma unroll
            for (int ct = 0; ct < P::NCT; ++ct) {
                if (kc > 16 * ct + 15) continue;  // block above the diagonal: zero
                const FC ah = lds_frag_perm<KC>(&sm.th[16 * ct + m][0], kc, gq);
                const FC al = lds_frag_perm<KC>(&sm.tl[16 * ct + m][0], kc, gq);
#pragma unroll
                for (int vt = 0; vt < P::NVT; ++vt) {
                    uu[ct][vt] = mma(ah, wh[vt], uu[ct][vt]);
                    uu[ct][vt] = mma(ah, wl[vt], uu[ct][vt]);
                    uu[ct][vt] = mma(al, wh[vt], uu[ct][vt]);
                }
            }
        }
        // O += (M o Q K^T) U   (U hi); the state update operand diag(exp(gamma_last -
        // gamma)) U is split into hi + lo.
        f32x4_t eglv[P::NCT];
#pragma unroll
        for (int ct = 0; ct < P::NCT; ++ct)
            eglv[ct] = *reinterpret_cast<const f32x4_t*>(&sm.egl[16 * ct + 4 * gq]);
        const float eg_last = sm.eg[C - 1];
        FC uth[C / KC][P::NVT], utl[C / KC][P::NVT];
#pragma unroll
        for (int kc = 0; kc < C; kc += KC) {
            const int c1 = (kc / 16) + (KC == 32 ? 1 : 0);
            FC uh[P::NVT];
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt) {
                uh[vt] = acc_frag_hi<KC>(uu[kc / 16][vt], uu[c1][vt]);
                acc_frag<KC>(uu[kc / 16][vt] * eglv[kc / 16], uu[c1][vt] * eglv[c1], uth[kc / KC][vt],
                             utl[kc / KC][vt]);
            }
#pragma unroll
            for (int ct = 0; ct < P::NCT; ++ct) {
                if (kc > 16 * ct + 15) continue;
                const FC ap = lds_frag_perm<KC>(&sm.pm[16 * ct + m][0], kc, gq);
#pragma unroll
                for (int vt = 0; vt < P::NVT; ++vt) qs[ct][vt] = mma(ap, uh[vt], qs[ct][vt]);
            }
        }
        // S^T = exp(gamma_last) S^T + K^T (diag(exp(gamma_last - gamma)) U)   (hi + lo)
#pragma unroll
        for (int dt = 0; dt < P::NDT; ++dt) {
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt) st[dt][vt] *= eg_last;
#pragma unroll
            for (int kc = 0; kc < C; kc += KC) {
                const FC a = lds_frag_perm<KC>(&sm.kt[16 * dt + m][0], kc, gq);
#pragma unroll
                for (int vt = 0; vt < P::NVT; ++vt) {
                    st[dt][vt] = mma(a, uth[kc / KC][vt], st[dt][vt]);
                    st[dt][vt] = mma(a, utl[kc / KC][vt], st[dt][vt]);
                }
            }
        }
        // ---- outputs: stage in LDS, then coalesced 16-byte stores ------------------
        // sm.u.o overlays the T scratch, which no wave reads after the last level
        // barrier.  The barrier below also guarantees every wave has finished the
        // state-dependent part before the next chunk is staged.
#pragma unroll
        for (int ct = 0; ct < P::NCT; ++ct)
#pragma unroll
            for (int vt = 0; vt < P::NVT; ++vt)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    sm.u.o[16 * ct + 4 * gq + i][vcol0 + 16 * vt + m] = f32_to_bf16(scale * qs[ct][vt][i]);
        __syncthreads();
        for (int i = tid; i < L * (D / 8); i += P::NT) {
            const int r = i / (D / 8), seg = i - r * (D / 8);
            *reinterpret_cast<uint4*>(o + (size_t)(t0 + r) * v_stride + (size_t)h * D + seg * 8) =
                *reinterpret_cast<const uint4*>(&sm.u.o[r][seg * 8]);
        }
        // No barrier: the next staging writes only q, k, v, graw and beta; sm.u is
        // next written after the staging barrier.
    }

    // final state
#pragma unroll
    for (int dt = 0; dt < P::NDT; ++dt)
#pragma unroll
        for (int vt = 0; vt < P::NVT; ++vt) {
            const float4 s4 = {st[dt][vt][0], st[dt][vt][1], st[dt][vt][2], st[dt][vt][3]};
            *reinterpret_cast<float4*>(final_state + state_off + (size_t)(vcol0 + 16 * vt + m) * D +
                                       16 * dt + 4 * gq) = s4;
        }
}


hipError_t launch_prefill(const PrefillArgs& a, hipStream_t stream) {
    int32_t* order = static_cast<int32_t*>(a.workspace);
    if (a.D == 128) {
        // short sequences token by token (that launch also writes the
        // schedule), the rest in chunks; with T <= kRecurMax every sequence is short
        hipError_t e = launch_prefill_recur(a, order, stream);
        if (e != hipSuccess || a.T <= kRecurMax || a.short_only) return e;
        return launch_prefill_pipe(a, order, stream);
    }
    hipLaunchKernelGGL(prefill_schedule_kernel, dim3(1), dim3(256), 0, stream, a.cu_seqlens, a.N, a.T, order);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    typedef Cfg<16, 16> P16;
    hipLaunchKernelGGL((prefill_kernel<16, 16>), dim3((unsigned)(a.N * a.H_v)), dim3(P16::NT), 0,
                       stream, (const uint16_t*)a.q, (const uint16_t*)a.k, (const uint16_t*)a.v, a.g,
                       a.beta, a.cu_seqlens, (const int32_t*)order, a.initial_state, a.final_state,
                       (uint16_t*)a.o, a.N, a.T, a.H_qk, a.H_v, a.scale, a.state_idx, a.P, a.flags);
    return hipGetLastError();
}

}  // namespace gdn
