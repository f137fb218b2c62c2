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
//   * 4 producer waves: in iteration c they prepare every state-independent
//     input of chunk c + 1, loading chunk c + 2 into registers meanwhile.
//
// One workgroup barrier ends each iteration.  Inside an iteration the roles
// meet only through LDS counters: state waves count "K^T of chunk c written"
// (each builds a part at the start of the iteration; all parts are needed by
// the state update at its end), "done reading Q of chunk c" and "done reading
// V of chunk c"
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
constexpr int FB = 20;                // row pitch (fp32) of a stored 16 x 16 block (16-byte rows)
constexpr int FS = 16 * FB + 8;       // block stride (fp32): successive blocks start 8 banks apart
constexpr int NBLK = NCT * (NCT + 1) / 2;   // lower-triangular 16 x 16 blocks (10)
constexpr int SEGS = D / 8;                 // 16-byte segments per q/k/v row
constexpr int PITEMS = C * SEGS / (64 * NP);  // staged segments per producer thread
constexpr int kSpinLimit = 1 << 20;

__device__ __forceinline__ constexpr int bidx(int i, int j) { return i * (i + 1) / 2 + j; }


struct Smem {
    uint16_t kb[2][C][PD];            // K rows, by chunk parity
    uint16_t qb[C][PD];               // Q rows
    uint16_t vb[C][PD];               // V rows
    uint16_t kt[D][PC];               // K^T of the chunk the state waves work on
    uint16_t th[2][NBLK][16][BP];     // T diag(beta), bf16 hi, lower blocks
    uint16_t tl[2][NBLK][16][BP];     // T diag(beta), bf16 lo
    uint16_t pm[2][NBLK][16][BP];     // (M o Q K^T), bf16
    uint16_t zero[16][BP];            // stands in for blocks above the diagonal
    float at[NBLK][FS];               // A^T by lower blocks: at[blk][c * FB + r] = A[r][c] (producers)
    float dtr[NCT][FS];               // D_b^T of the diagonal blocks of T (producers)
    alignas(16) float gam[NP][C];     // per producer wave: gate prefix of its chunk
    alignas(16) float bet[NP][C];     // per producer wave: beta of its chunk
    alignas(16) float eg[2][C];       // exp(gamma), by chunk parity
    alignas(16) float egl[2][C];      // exp(gamma_last - gamma), by chunk parity
    unsigned cnt[4];                  // producer barrier, K^T written, Q free, V free
};

enum { CNT_PBAR = 0, CNT_KT = 1, CNT_QFREE = 2, CNT_VFREE = 3 };

// Inclusive prefix sum over the 64 lanes of a wave (DPP row shifts, then row
// broadcasts across the four rows of 16 lanes).
template <int CTRL, int ROWMASK, bool BOUND>
__device__ __forceinline__ float dpp_src(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWMASK, 0xF, BOUND));
}
__device__ __forceinline__ float wave_prefix_sum(float x) {
    x += dpp_src<0x111, 0xF, true>(x);  // row_shr:1
    x += dpp_src<0x112, 0xF, true>(x);  // row_shr:2
    x += dpp_src<0x114, 0xF, true>(x);  // row_shr:4
    x += dpp_src<0x118, 0xF, true>(x);  // row_shr:8
    x += dpp_src<0x142, 0xA, false>(x); // row_bcast:15 into rows 1 and 3
    x += dpp_src<0x143, 0xC, false>(x); // row_bcast:31 into rows 2 and 3
    return x;
}

// Row / column block of the lower-triangular block with linear index tri.
__device__ __forceinline__ int tri_row(int tri) { return tri >= 6 ? 3 : tri >= 3 ? 2 : tri >= 1 ? 1 : 0; }

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

// Block column J of T below the diagonal (producer wave J):
//     T_bJ = -D_b sum_{kb=J}^{b-1} A_{b,kb} T_{kb,J},   T_JJ = D_J,
// each result kept in its accumulator, which as a B operand supplies
// contraction row 4 g + s at step s.  All LDS operands are loaded first; the
// results go out as T diag(beta) hi / lo.
// 16 x 16 x 16 product of fp32 operands on bf16 MFMA with each operand split
// into hi + lo (hi*hi + hi*lo + lo*hi; relative error ~2^-16).  a[j] is the A
// operand (row m, contraction 4 g + j), b[j] the B operand (contraction 4 g + j,
// column m); an accumulator holding X is the B operand of X and, read as
// a[j], the A operand of X^T.
__device__ __forceinline__ f32x4_t prod3(const f32x4_t& a, const f32x4_t& b, f32x4_t acc) {
    uint2 ah, al, bh, bl;
    split_pair(a[0], a[1], ah.x, al.x);
    split_pair(a[2], a[3], ah.y, al.y);
    split_pair(b[0], b[1], bh.x, bl.x);
    split_pair(b[2], b[3], bh.y, bl.y);
    const s16x4_t ahf = __builtin_bit_cast(s16x4_t, ah), alf = __builtin_bit_cast(s16x4_t, al);
    const s16x4_t bhf = __builtin_bit_cast(s16x4_t, bh), blf = __builtin_bit_cast(s16x4_t, bl);
    acc = mma(ahf, bhf, acc);
    acc = mma(ahf, blf, acc);
    return mma(alf, bhf, acc);
}

template <int J>
__device__ __forceinline__ void col_sweep(Smem& sm, int par, int m, int g) {
    const float bcol = sm.bet[J][16 * J + m];
    const f32x4_t djb = *reinterpret_cast<const f32x4_t*>(sm.dtr[J] + m * FB + 4 * g);
    f32x4_t aop[NCT][NCT];    // A_{bi,kb}[m][4 g + s]
    f32x4_t dop[NCT];         // -D_bi[m][4 g + s]
#pragma unroll
    for (int bi = J + 1; bi < NCT; ++bi) {
#pragma unroll
        for (int kb = J; kb < bi; ++kb) {
            const float* ab = sm.at[bidx(bi, kb)];
#pragma unroll
            for (int s = 0; s < 4; ++s) aop[bi][kb][s] = ab[(4 * g + s) * FB + m];
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) dop[bi][s] = -sm.dtr[bi][(4 * g + s) * FB + m];
    }
    f32x4_t tz[NCT];
#pragma unroll
    for (int bi = J + 1; bi < NCT; ++bi) {
        // one accumulator per term of the sum, added at the end
        const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
        f32x4_t yk[NCT];
#pragma unroll
        for (int kb = J; kb < bi; ++kb) yk[kb] = prod3(aop[bi][kb], kb == J ? djb : tz[kb], zero);
        f32x4_t y = yk[J];
#pragma unroll
        for (int kb = J + 1; kb < bi; ++kb) y += yk[kb];
        const f32x4_t z = prod3(dop[bi], y, zero);
        tz[bi] = z;
        const int ob = bidx(bi, J);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            split_bf16(z[i] * bcol, sm.th[par][ob][4 * g + i][m], sm.tl[par][ob][4 * g + i][m]);
    }
}

// D = (I + N)^-1 for a strictly lower 16 x 16 block N (N^16 = 0), as the
// product (I - N)(I + N^2)(I + N^4)(I + N^8) (the factors are polynomials in N
// and commute), each product on three bf16 MFMAs (prod3).  An accumulator
// holding X is the B operand of X and the A operand of X^T, so each power is
// formed both ways and every product reads registers only.
//   nat: A operand of N, N[m][4 g + s];  nb: B operand of N, N[4 g + s][m].
// Returns D in accumulator layout.
__device__ __forceinline__ f32x4_t block_inverse(const f32x4_t& nat, const f32x4_t& nb, int m, int g) {
    auto prod = [](const f32x4_t& a, const f32x4_t& b, const f32x4_t& acc) { return prod3(a, b, acc); };
    const f32x4_t zero = {0.f, 0.f, 0.f, 0.f};
    const f32x4_t n2 = prod(nat, nb, zero);    // N^2
    const f32x4_t n2t = prod(nb, nat, zero);   // (N^2)^T = N^T N^T
    const f32x4_t n3 = prod(nat, n2, zero);    // N^3 = N N^2
    const f32x4_t n4 = prod(n2t, n2, zero);    // N^4 = N^2 N^2
    const f32x4_t n4t = prod(n2, n2t, zero);   // (N^4)^T
    f32x4_t p1;                                // (I - N)(I + N^2) = I - N + N^2 - N^3
#pragma unroll
    for (int i = 0; i < 4; ++i) p1[i] = ((4 * g + i == m) ? 1.f : 0.f) - nb[i] + n2[i] - n3[i];
    const f32x4_t p2 = prod(n4t, p1, p1);      // (I + N^4) P1
    const f32x4_t n8t = prod(n4, n4t, zero);   // (N^8)^T
    return prod(n8t, p2, p2);                  // (I + N^8) P2
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
            // K^T of chunk c (read only by the state update at the end of this
            // iteration, after every state wave has written its part)
            for (int i = tid; i < (C / 2) * SEGS; i += 64 * NS) {
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
            signal(&sm.cnt[CNT_KT], lane);
            // K S0^T (S0 hi + lo) and Q S0^T (S0 hi)
            f32x4_t ks[NCT][NVT], qs[NCT][NVT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) {
                    ks[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                    qs[ct][vt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                }
            bf16x8_t ak[2][NCT], aq[2][NCT];  // operands of two contraction steps in flight
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                ak[0][ct] = lds_frag_perm<32>(&sm.kb[par][16 * ct + m][0], 0, gq);
                aq[0][ct] = lds_frag_perm<32>(&sm.qb[16 * ct + m][0], 0, gq);
            }
#pragma unroll
            for (int kq = 0; kq < D / 32; ++kq) {
                const int cur = kq & 1;
                if (kq + 1 < D / 32) {
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        ak[cur ^ 1][ct] = lds_frag_perm<32>(&sm.kb[par][16 * ct + m][0], 32 * (kq + 1), gq);
                        aq[cur ^ 1][ct] = lds_frag_perm<32>(&sm.qb[16 * ct + m][0], 32 * (kq + 1), gq);
                    }
                }
                bf16x8_t bh[NVT], bl[NVT];
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) acc_frag<32>(st[2 * kq][vt], st[2 * kq + 1][vt], bh[vt], bl[vt]);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        ks[ct][vt] = mma(ak[cur][ct], bh[vt], ks[ct][vt]);
                        ks[ct][vt] = mma(ak[cur][ct], bl[vt], ks[ct][vt]);
                        qs[ct][vt] = mma(aq[cur][ct], bh[vt], qs[ct][vt]);
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
            // Outputs: a 4 x 4 transpose inside each quad of lanes turns "4 rows of
            // one column" into "4 columns of one row", stored as 8 bytes.
            {
                const int kq = m & 3;
                const bool odd = (kq & 1) != 0, hi2 = (kq & 2) != 0;
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        const f32x4_t a0 = qs[ct][vt] * scale;
                        const float x0 = dpp<DPP_QUAD_XOR1>(a0[1]), x1 = dpp<DPP_QUAD_XOR1>(a0[0]);
                        const float x2 = dpp<DPP_QUAD_XOR1>(a0[3]), x3 = dpp<DPP_QUAD_XOR1>(a0[2]);
                        const f32x4_t a1 = {odd ? x0 : a0[0], odd ? a0[1] : x1, odd ? x2 : a0[2], odd ? a0[3] : x3};
                        const float u0 = dpp<DPP_QUAD_XOR2>(a1[2]), u1 = dpp<DPP_QUAD_XOR2>(a1[3]);
                        const float u2 = dpp<DPP_QUAD_XOR2>(a1[0]), u3 = dpp<DPP_QUAD_XOR2>(a1[1]);
                        const f32x4_t a2 = {hi2 ? u0 : a1[0], hi2 ? u1 : a1[1], hi2 ? a1[2] : u2, hi2 ? a1[3] : u3};
                        const int row = 16 * ct + 4 * gq + kq;
                        if (row < L) {
                            const uint2 pk = {cvt_pk(a2[0], a2[1]), cvt_pk(a2[2], a2[3])};
                            *reinterpret_cast<uint2*>(o + (size_t)(t0 + row) * v_stride + (size_t)h * D + vcol0 +
                                                      16 * vt + 4 * (m >> 2)) = pk;
                        }
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
            wait_ge(&sm.cnt[CNT_KT], (unsigned)(NS * (c + 1)));
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
            const float gx = wave_prefix_sum(rg);
            const float glast = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gx), C - 1));
            sm.gam[pw][lane] = gx;
            sm.bet[pw][lane] = rb;
            if (pw == 0) {
                sm.eg[par][lane] = fast_exp(gx);
                sm.egl[par][lane] = fast_exp(glast - gx);
            }
            pbar();  // K of chunk x complete
            // G = K K^T tiles pw, pw + 4, pw + 8 -> A^T (fp32); all operand loads
            // are issued before the products.
            {
                constexpr int NJ = 3;
                bf16x8_t fa[NJ][D / 32], fb[NJ][D / 32];
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj) {
                    const int tri = min(pw + NP * jj, NBLK - 1);
                    const int ti = tri_row(tri), tj = tri - ti * (ti + 1) / 2;
#pragma unroll
                    for (int kq = 0; kq < D / 32; ++kq) {
                        fa[jj][kq] = lds_frag_nat<32>(&sm.kb[par][16 * ti + m][0], 32 * kq, gq);
                        fb[jj][kq] = lds_frag_nat<32>(&sm.kb[par][16 * tj + m][0], 32 * kq, gq);
                    }
                }
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj) {
                    const int tri = pw + NP * jj;
                    if (tri >= NBLK) break;
                    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kq = 0; kq < D / 32; ++kq) acc = mma(fa[jj][kq], fb[jj][kq], acc);
                    const int ti = tri_row(tri), tj = tri - ti * (ti + 1) / 2;
                    const int col = 16 * tj + m;
                    const float gcol = sm.gam[pw][col];
                    const f32x4_t grow = *reinterpret_cast<const f32x4_t*>(&sm.gam[pw][16 * ti + 4 * gq]);
                    const f32x4_t brow = *reinterpret_cast<const f32x4_t*>(&sm.bet[pw][16 * ti + 4 * gq]);
                    f32x4_t val;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int row = 16 * ti + 4 * gq + i;
                        val[i] = col < row ? brow[i] * fast_exp(grow[i] - gcol) * acc[i] : 0.f;
                    }
                    *reinterpret_cast<f32x4_t*>(&sm.at[tri][m * FB + 4 * gq]) = val;
                }
            }
            pbar();  // A complete
            // T = (I + A)^-1.  Wave pw inverts diagonal block pw on the matrix
            // cores, writes its T diag(beta) and shares D^T with the other
            // producers; after one producer barrier, wave j < 3 sweeps block
            // column j below the diagonal.
            {
                const int bb = bidx(pw, pw);
                const float* atb = sm.at[bb];
                const f32x4_t nat = {atb[(4 * gq) * FB + m], atb[(4 * gq + 1) * FB + m],
                                     atb[(4 * gq + 2) * FB + m], atb[(4 * gq + 3) * FB + m]};
                const f32x4_t nb = *reinterpret_cast<const f32x4_t*>(atb + m * FB + 4 * gq);
                const f32x4_t dacc = block_inverse(nat, nb, m, gq);
                const float bcol = sm.bet[pw][16 * pw + m];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    split_bf16(dacc[i] * bcol, sm.th[par][bb][4 * gq + i][m], sm.tl[par][bb][4 * gq + i][m]);
                *reinterpret_cast<f32x4_t*>(sm.dtr[pw] + m * FB + 4 * gq) = dacc;
            }
            pbar();  // diagonal blocks of T complete
            // Block column sweep of wave pw < 3 (below the diagonal of T).
            if (pw == 0) col_sweep<0>(sm, par, m, gq);
            else if (pw == 1) col_sweep<1>(sm, par, m, gq);
            else if (pw == 2) col_sweep<2>(sm, par, m, gq);
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
            // P = Q K^T tiles -> masked scores (bf16); operands loaded first
            {
                constexpr int NJ = 3;
                bf16x8_t fa[NJ][D / 32], fb[NJ][D / 32];
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj) {
                    const int tri = min(pw + NP * jj, NBLK - 1);
                    const int ti = tri_row(tri), tj = tri - ti * (ti + 1) / 2;
#pragma unroll
                    for (int kq = 0; kq < D / 32; ++kq) {
                        fa[jj][kq] = lds_frag_nat<32>(&sm.qb[16 * ti + m][0], 32 * kq, gq);
                        fb[jj][kq] = lds_frag_nat<32>(&sm.kb[par][16 * tj + m][0], 32 * kq, gq);
                    }
                }
#pragma unroll
                for (int jj = 0; jj < NJ; ++jj) {
                    const int tri = pw + NP * jj;
                    if (tri >= NBLK) break;
                    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kq = 0; kq < D / 32; ++kq) acc = mma(fa[jj][kq], fb[jj][kq], acc);
                    const int ti = tri_row(tri), tj = tri - ti * (ti + 1) / 2;
                    const int col = 16 * tj + m;
                    const float gcol = sm.gam[pw][col];
                    const f32x4_t grow = *reinterpret_cast<const f32x4_t*>(&sm.gam[pw][16 * ti + 4 * gq]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int row = 16 * ti + 4 * gq + i;
                        sm.pm[par][tri][4 * gq + i][m] = f32_to_bf16(col <= row ? fast_exp(grow[i] - gcol) * acc[i] : 0.f);
                    }
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
