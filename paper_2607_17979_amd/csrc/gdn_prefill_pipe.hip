// Pipelined chunk kernel of the prefill regime for d = 128, chunk 64 (the
// chunked form and its notation are described in gdn_prefill.hip).
//
// The per-chunk work splits into a state-independent part (the gate prefix,
// the Gram and score tiles K K^T and Q K^T with their masks and decays,
// T = (I + A)^-1 and T diag(beta)) and a state-dependent part (K S0^T, Q S0^T,
// W, U, O and the state update).  Only the second part is sequential along a
// sequence.  One workgroup per (sequence, value head) runs them in two kinds
// of waves that never share a barrier inside the chunk loop:
//
//   * NS state waves: wave w owns value columns [w D/NS, (w + 1) D/NS) of S^T in
//     fp32 MFMA accumulators and runs the state-dependent part chunk by chunk;
//   * NP = 4 producer waves: producer p owns the chunks x = p (mod 4).  For each
//     it loads K, Q, g and beta straight from global memory into MFMA operand
//     registers, computes every state-independent input of the chunk on its
//     own (block inverses, block column sweep and masked scores all stay in
//     registers), writes them to its result slot once the state waves are done
//     with the slot's previous chunk, and finally stages the chunk's K, Q, V
//     rows into LDS (K double-buffered by chunk parity, Q and V single) once
//     the state waves have released the buffers: K and the second half of Q
//     from the operand registers it still holds, the first half of Q and V
//     read from memory.  A producer therefore has
//     about four state iterations to prepare a chunk, and none of its latency
//     is on the state waves' path.
//
// Operands that run along a column of a row-major LDS array (K^T for the state
// update, V for W) come from the gfx950 transpose read, so no transposed copy
// is ever built.  Waves meet only through counters in LDS (chunks staged,
// buffers released, slot results ready, slots released).  Every wait is a
// bounded spin; LDS operations of a wave execute in order, so a counter
// increment issued after a wave's LDS stores (or reads) is observed only after
// those have executed.
#include <algorithm>

#include "gdn_launch.h"
#include "gdn_mfma.h"

namespace gdn {
namespace pipe {

constexpr int D = 128, C = 64;
constexpr int NP = 4;                 // producer waves = result slots
constexpr int NDT = D / 16, NCT = C / 16;
// LDS pitch (bf16) of the [C][D] row buffers: 72 dwords, so eight
// consecutive rows start 8 banks apart.  Columns are stored swizzled,
// column c of row r at c ^ (r & 8) (8-byte units stay whole): the transposed
// reads (8 consecutive rows x 4 eight-byte units per half wave) and the row
// reads (16 rows x 2 units per half wave, rows r and r + 8 now 4 banks apart)
// both touch 64 distinct banks.
constexpr int PD = D + 16;
// Swizzled column of row r of a row buffer or a P block.  Only bit 3 of the
// column changes, so for c = c16 + c_lane with c16 a multiple of 16 the
// swizzle applies to c_lane alone and c16 stays an address immediate.
__device__ __forceinline__ int swz(int r, int c) { return c ^ (r & 8); }
constexpr int NBLK = NCT * (NCT + 1) / 2;   // lower-triangular 16 x 16 blocks (10)
constexpr int SEGS = D / 8;                 // 16-byte segments per q/k/v row
constexpr int SITEMS = C * SEGS / 64;       // staged segments per producer lane (16)
constexpr int SP = 20;                      // row pitch (fp32) of the producers' 16 x 16 scratch blocks
// Block pitch (fp32) of that scratch: 4 words of padding, so that the four
// lane groups, each reading a row of its own block, hit different banks.
constexpr int SBS = 16 * SP + 4;
constexpr int kSpinLimit = 1 << 20;
// K S0^T takes the lo half of S0 only when the chunk's total decay
// exp(gamma_last) exceeds this (see the state waves' first phase).
constexpr float kS0LoDecay = 1.f / 256;

__device__ __forceinline__ constexpr int bidx(int i, int j) { return i * (i + 1) / 2 + j; }

// Column of the 4-element unit u of row r in a stored 16 x 16 bf16 block: the
// units of a row rotate with r / 4.  The 8-byte stores of one unit column
// (16 lanes, rows 0..15) then cover all 128 bytes of banks a store cycle
// serves, and the 8-byte reads of 32 lanes all 256 bytes of a read cycle.
__device__ __forceinline__ int bsw(int r, int u) { return 4 * (u ^ ((r >> 2) & 3)); }

// Results of the state-independent part of one chunk.
struct Slot {
    // 16 x 16 blocks, the 4-element units of each row placed by bsw
    uint16_t th[NBLK][16][16];   // T diag(beta) by lower blocks, transposed [col][row], bf16 hi
    uint16_t tl[NBLK][16][16];   // bf16 lo
    uint16_t pm[NBLK][16][16];   // scale (M o Q K^T) by lower blocks [row t][col s], bf16
    alignas(16) float eg[C];     // exp(gamma)
    alignas(16) float egl[C];    // exp(gamma_last - gamma)
};

enum {
    CNT_STG = 0,      // chunks whose K, Q and V rows are staged
    CNT_QVFREE,       // releases of the Q and V row buffers (state waves after W,
                      // output waves after (Q S0^T)^T)
    CNT_DONE,         // chunk completions (state and output waves): the chunk's
                      // K buffer and result slot are free
    CNT_READY0,       // + p: chunks written to slot p
    CNT_HAND0 = CNT_READY0 + NP,  // + 4 w + {0, 1, 2, 3}: S0 hi operands of state
                      // wave w written / read, U hi operands written / read
    NCNT = CNT_HAND0 + 4 * 2
};

// VB: value columns of the workgroup (the V rows it stages); NO: output waves,
// each finishing (Q S0^T)^T, the output products and the stores for one state
// wave, fed through the hand-over arrays.
template <int VB, int NO, int NVT>
struct Smem {
    uint16_t kb[2][C][PD];            // K rows, by chunk parity
    uint16_t qb[C][PD];               // Q rows of the chunk in flight
    uint16_t vb[C][VB + 16];          // V rows, the workgroup's columns (swizzled, see PD)
    Slot slot[NP];
    alignas(16) float scr[NP][NCT * SBS];  // per producer: diagonal blocks of A, then of T
    alignas(16) float gam[NP][C];     // per producer: gate prefix of its chunk
    alignas(16) float bet[NP][C];     // per producer: beta of its chunk
    uint16_t zero[16][16];            // stands in for blocks above the diagonal
    uint4 hs[NO][D / 32][NVT][64];    // per state wave: S0 hi operands of the chunk
    uint4 hu[NO][C / 32][NVT][64];    // per state wave: U hi operands of the chunk
    unsigned cnt[NCNT];
    alignas(16) float rn[NP][2][C];   // per producer, with the q/k L2 norm: 1 / |row| of its K, Q rows
};

template <int CTRL, int ROWMASK, bool BOUND>
__device__ __forceinline__ float dpp_src(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWMASK, 0xF, BOUND));
}
// Terms of one row of the diagonal-block solve: acc + sum_i n_i(R) y_i over
// the CNT (1 to 4) elements of n and y in order, where n_i(R) is n_i in lane R
// of this lane's row of 16 lanes: v_fmac_f32 with a DPP row broadcast
// (row_newbcast, gfx90a and later) on n_i, one instruction per term.  The
// block starts with two wait states, so the DPP reads are safe even if the
// compiler has just written n's registers with a vector instruction.
template <int R, int CNT>
__device__ __forceinline__ float fmac_bcast(float acc, const f32x4_t& n, const float* y) {
    static_assert(R >= 1 && R < 16 && CNT >= 1 && CNT <= 4, "lane and term count");
    if constexpr (CNT == 4)
        asm("s_nop 1\n"
            "v_fmac_f32_dpp %0, %1, %5 row_newbcast:%9 row_mask:0xf bank_mask:0xf\n"
            "v_fmac_f32_dpp %0, %2, %6 row_newbcast:%9 row_mask:0xf bank_mask:0xf\n"
            "v_fmac_f32_dpp %0, %3, %7 row_newbcast:%9 row_mask:0xf bank_mask:0xf\n"
            "v_fmac_f32_dpp %0, %4, %8 row_newbcast:%9 row_mask:0xf bank_mask:0xf"
            : "+v"(acc)
            : "v"(n[0]), "v"(n[1]), "v"(n[2]), "v"(n[3]), "v"(y[0]), "v"(y[1]), "v"(y[2]), "v"(y[3]), "i"(R));
    else if constexpr (CNT == 3)
        asm("s_nop 1\n"
            "v_fmac_f32_dpp %0, %1, %4 row_newbcast:%7 row_mask:0xf bank_mask:0xf\n"
            "v_fmac_f32_dpp %0, %2, %5 row_newbcast:%7 row_mask:0xf bank_mask:0xf\n"
            "v_fmac_f32_dpp %0, %3, %6 row_newbcast:%7 row_mask:0xf bank_mask:0xf"
            : "+v"(acc) : "v"(n[0]), "v"(n[1]), "v"(n[2]), "v"(y[0]), "v"(y[1]), "v"(y[2]), "i"(R));
    else if constexpr (CNT == 2)
        asm("s_nop 1\n"
            "v_fmac_f32_dpp %0, %1, %3 row_newbcast:%5 row_mask:0xf bank_mask:0xf\n"
            "v_fmac_f32_dpp %0, %2, %4 row_newbcast:%5 row_mask:0xf bank_mask:0xf"
            : "+v"(acc) : "v"(n[0]), "v"(n[1]), "v"(y[0]), "v"(y[1]), "i"(R));
    else
        asm("s_nop 1\n"
            "v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
            : "+v"(acc) : "v"(n[0]), "v"(y[0]), "i"(R));
    return acc;
}
// Row R of the solve: acc + sum_{i < R} nrow_i(R) xs_i, terms in order of i.
template <int R>
__device__ __forceinline__ float fsolve_row(const f32x4_t (&nrow)[4], const float (&xs)[16], float acc) {
    acc = fmac_bcast<R, (R < 4 ? R : 4)>(acc, nrow[0], &xs[0]);
    if constexpr (R > 4) acc = fmac_bcast<R, (R - 4 < 4 ? R - 4 : 4)>(acc, nrow[1], &xs[4]);
    if constexpr (R > 8) acc = fmac_bcast<R, (R - 8 < 4 ? R - 8 : 4)>(acc, nrow[2], &xs[8]);
    if constexpr (R > 12) acc = fmac_bcast<R, R - 12>(acc, nrow[3], &xs[12]);
    return acc;
}
// Inclusive prefix sum over the 64 lanes of a wave (DPP row shifts, then row
// broadcasts across the four rows of 16 lanes).
__device__ __forceinline__ float wave_prefix_sum(float x) {
    x += dpp_src<0x111, 0xF, true>(x);  // row_shr:1
    x += dpp_src<0x112, 0xF, true>(x);  // row_shr:2
    x += dpp_src<0x114, 0xF, true>(x);  // row_shr:4
    x += dpp_src<0x118, 0xF, true>(x);  // row_shr:8
    x += dpp_src<0x142, 0xA, false>(x); // row_bcast:15 into rows 1 and 3
    x += dpp_src<0x143, 0xC, false>(x); // row_bcast:31 into rows 2 and 3
    return x;
}

// Count this wave (lane 0) into *ctr.  The compiler fence keeps the wave's
// earlier LDS accesses before the increment; the LDS executes them in order.
__device__ __forceinline__ void signal(unsigned* ctr, int lane) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (lane == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Wait until *ctr >= target (bounded: never spins forever).  A wait that runs
// out of its bound (a broken synchronisation, never expected) sets *fault, so
// that the caller can tell that the call's results are invalid.
__device__ __forceinline__ void wait_ge(unsigned* ctr, unsigned target, int* fault) {
    int it = 0;
    for (; it < kSpinLimit; ++it) {
        if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= target) break;
        __builtin_amdgcn_s_sleep(1);
    }
    if (it == kSpinLimit) __hip_atomic_fetch_or(fault, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// A counter's value now, for a later wait_seen: the LDS round trip of the
// read overlaps the work in between.
__device__ __forceinline__ unsigned peek(unsigned* ctr) {
    return __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// wait_ge for a counter read earlier as `seen`: counters only grow, so a seen
// value at the target needs no further read.
__device__ __forceinline__ void wait_seen(unsigned* ctr, unsigned target, unsigned seen, int* fault) {
    if (__builtin_amdgcn_readfirstlane(seen) < target) wait_ge(ctr, target, fault);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));

// An 8-byte LDS read that stays a ds_read_b64 of its own.  Two 8-byte reads
// off one base would otherwise become one ds_read2_b64, which serves 16 lanes
// per cycle and word over 128 bytes of banks; a ds_read_b64 serves 32 lanes
// per cycle over 256 bytes, so the pair costs 4 LDS cycles instead of 8, and
// the operand patterns here, laid out for 256 bytes, stay conflict-free.
// (The volatile access is what keeps the compiler from pairing the two.)
__device__ __forceinline__ u32x2_t lds_ld8_alone(const uint16_t* p) {
    return *(const volatile __attribute__((address_space(3))) u32x2_t*)p;
}

// A (or B) operand from a stored lower-triangular block matrix (block row ct,
// contraction columns kc..kc+31 in the permuted order); blocks above the
// diagonal read the zero block.
__device__ __forceinline__ bf16x8_t blk_frag(const uint16_t (*blocks)[16][16], const uint16_t (*zero)[16],
                                             int ct, int kc, int m, int g) {
    const int j0 = kc >> 4;
    const uint16_t* p0 = &blocks[bidx(ct, j0)][m][bsw(m, g)];
    const uint16_t* p1 = (j0 + 1 <= ct) ? &blocks[bidx(ct, j0 + 1)][m][bsw(m, g)] : &zero[m][bsw(m, g)];
    const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(p0);
    const u32x2_t hi = lds_ld8_alone(p1);
    uint4 u = {lo[0], lo[1], hi[0], hi[1]};
    return __builtin_bit_cast(bf16x8_t, u);
}

typedef short tr16x4_t __attribute__((ext_vector_type(4)));

// gfx950 transpose read (ds_read_b64_tr_b16): within each group of 16 lanes,
// lane i receives element i % 4 of the 8-byte words addressed by lanes
// i / 4 + 4 e, e = 0..3.  With lane l addressing row r0 + l / 4, column
// c0 + 4 (l % 4) of a row-major array, lane i therefore gets rows r0..r0+3 of
// column c0 + i.
__device__ __forceinline__ uint2 lds_tr4(const uint16_t* p) {
    const tr16x4_t r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) tr16x4_t*)p);
    return __builtin_bit_cast(uint2, r);
}

// A operand whose rows are columns c0..c0+15 (c0 a multiple of 16) of a
// swizzled row buffer, contraction over rows r0..r0+31 (r0 a multiple of 16)
// in the permuted order (slot j < 4: row r0 + 4 g + j; slot j >= 4: row
// r0 + 16 + 4 g + (j - 4)).
__device__ __forceinline__ bf16x8_t lds_frag_tr(const uint16_t (*a)[PD], int r0, int c0, int m, int g) {
    const int r = 4 * g + (m >> 2), cl = swz(r, 4 * (m & 3));
    const uint2 lo = lds_tr4(&a[r0 + r][c0 + cl]);
    const uint2 hi = lds_tr4(&a[r0 + 16 + r][c0 + cl]);
    uint4 u = {lo.x, lo.y, hi.x, hi.y};
    return __builtin_bit_cast(bf16x8_t, u);
}

// A operand from a stored lower-triangular block matrix kept transposed
// ([col][row] per block): block row ct, contraction columns kc..kc+31 in the
// permuted order; blocks above the diagonal read the zero block.
__device__ __forceinline__ bf16x8_t blk_frag_t(const uint16_t (*blocks)[16][16], const uint16_t (*zero)[16],
                                               int ct, int kc, int m, int g) {
    const int j0 = kc >> 4;
    const int r = 4 * g + (m >> 2), cc = bsw(r, m & 3);
    const uint2 lo = lds_tr4(&blocks[bidx(ct, j0)][r][cc]);
    const uint2 hi = lds_tr4((j0 + 1 <= ct) ? &blocks[bidx(ct, j0 + 1)][r][cc] : &zero[r][cc]);
    uint4 u = {lo.x, lo.y, hi.x, hi.y};
    return __builtin_bit_cast(bf16x8_t, u);
}

// In the 16 x 16 block products below an accumulator holding X (lane m + 16 g,
// element i = X[4 g + i][m]) is the B operand of X and the A operand of X^T
// (contraction index 4 g + i), so prod(acc(X), acc(Y)) = acc(X^T Y).

// An accumulator-layout block split into bf16 hi and lo (four values per lane).
struct Split16 {
    uint2 h, l;
};
__device__ __forceinline__ Split16 split16(const f32x4_t& x) {
    Split16 r;
    split_pair(x[0], x[1], r.h.x, r.l.x);
    split_pair(x[2], x[3], r.h.y, r.l.y);
    return r;
}
// prod(acc(X), acc(Y)) = acc(X^T Y) on split bf16 operands: hi.hi, hi.lo and
// lo.hi as three 16x16x16 MFMAs, each accumulating in fp32.  (Packing hi.hi
// and hi.lo into one 16x16x32 MFMA lost the small terms within the
// instruction's own sum and failed parity.)  Relative error about 2^-16.
__device__ __forceinline__ f32x4_t prods(const Split16& a, const Split16& b, const f32x4_t& acc) {
    f32x4_t t = mma(__builtin_bit_cast(s16x4_t, a.h), __builtin_bit_cast(s16x4_t, b.h), acc);
    t = mma(__builtin_bit_cast(s16x4_t, a.h), __builtin_bit_cast(s16x4_t, b.l), t);
    return mma(__builtin_bit_cast(s16x4_t, a.l), __builtin_bit_cast(s16x4_t, b.h), t);
}

__device__ __forceinline__ bf16x8_t as_frag(const uint4& u) { return __builtin_bit_cast(bf16x8_t, u); }

// Block X in accumulator layout, times scale, stored transposed as bf16 hi / lo:
// element [m][4 g + i] of the stored block is X[4 g + i][m].
__device__ __forceinline__ void store_split_t(uint16_t (*th)[16], uint16_t (*tl)[16], const f32x4_t& x,
                                              float scale, int m, int g) {
    uint2 hi, lo;
    split_pair(x[0] * scale, x[1] * scale, hi.x, lo.x);
    split_pair(x[2] * scale, x[3] * scale, hi.y, lo.y);
    *reinterpret_cast<uint2*>(&th[m][bsw(m, g)]) = hi;
    *reinterpret_cast<uint2*>(&tl[m][bsw(m, g)]) = lo;
}

// Context of a producer wave: values fixed for the whole sequence.
struct ProdCtx {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const float* g;
    const float* beta;
    size_t qk_stride, v_stride;
    int seq_beg, seq_len, hq, h, H_v, pw;
    int vcb0;   // first value column of the workgroup
    float scale;
    int* fault; // set by a wait that runs out of its bound
};

// A/B operand from row r of a swizzled row buffer, contraction columns
// k0..k0+31 (k0 a multiple of 32) in the permuted order of the accumulator
// tiles (slot j < 4: column k0 + 4 g + j, slot j >= 4: k0 + 16 + 4 g + j - 4).
__device__ __forceinline__ bf16x8_t row_frag(const uint16_t (*a)[PD], int r, int k0, int g) {
    const int cl = swz(r, 4 * g);
    const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(&a[r][k0 + cl]);
    const u32x2_t hi = lds_ld8_alone(&a[r][k0 + 16 + cl]);
    uint4 u = {lo[0], lo[1], hi[0], hi[1]};
    return __builtin_bit_cast(bf16x8_t, u);
}

// 16-byte global load at a wave-uniform base plus a 32-bit per-lane
// byte offset (scalar base + vector offset addressing: no 64-bit lane math).
__device__ __forceinline__ uint4 ld16(const void* base, unsigned byte_off) {
    return *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(base) + byte_off);
}
// Streaming load of the V rows (read once), marked non-temporal so that it
// does not push out of L2 the Q rows 0..31 of a chunk, which the producers
// read twice (operand fragments, then staging a few chunks later).
typedef unsigned u32x4v_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_stream(const void* base, unsigned byte_off) {
    const u32x4v_t r =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4v_t*>(reinterpret_cast<const char*>(base) + byte_off));
    return uint4{r[0], r[1], r[2], r[3]};
}

// Producer work for chunk lc of the work item described by pc, which is chunk
// x of the workgroup's chunk stream (the chunks of its work items in order;
// buffers and counters follow x).  The lane indices m, gq are passed in per
// chunk (opaque to the compiler), so the addresses and masks derived from them
// are recomputed per chunk instead of being kept live across the producer loop.
// NSIG: waves that count each chunk done and each Q/V release (state plus
// output waves); VB: value columns staged.
// PRO: the input prologue (kFlagQkL2Norm, kFlagGateLogits).
template <int NSIG, int VB, int PRO, class SM>
__device__ __forceinline__ void produce_chunk(SM& sm, const ProdCtx& pc, int x, int lc, int m, int gq) {
    constexpr bool NORM = (PRO & kFlagQkL2Norm) != 0;
    const int lane = m + 16 * gq;
    Slot& sl = sm.slot[pc.pw];
    float* scr = sm.scr[pc.pw];
    float* gam = sm.gam[pc.pw];
    float* bet = sm.bet[pc.pw];
    const int L = min(C, pc.seq_len - lc * C);
    const int tb = pc.seq_beg + lc * C;
    // ---- inputs: gates and the K operand fragments of the chunk
    //      (fk[b][kq]: row 16 b + m, columns 32 kq + 8 gq .. + 7); the Q
    //      fragments of block row b are loaded one block row ahead
    // Uniform chunk bases with 32-bit lane offsets.  Rows past the end of a
    // short last chunk read row L - 1 instead of zeros: those rows have
    // g = beta = 0, so T diag(beta) is exactly zero in their rows and columns,
    // and their scores and outputs are never used; the values only need to be
    // finite.
    const uint16_t* kc0 = pc.k + (size_t)tb * pc.qk_stride + (size_t)pc.hq * D;
    const uint16_t* qc0 = pc.q + (size_t)tb * pc.qk_stride + (size_t)pc.hq * D;
    const unsigned qks = (unsigned)pc.qk_stride;
    const bool in = lane < L;
    float gl = in ? pc.g[(size_t)(tb + lane) * pc.H_v + pc.h] : 0.f;
    float bl = in ? pc.beta[(size_t)(tb + lane) * pc.H_v + pc.h] : 0.f;
    if ((PRO & kFlagGateLogits) && in) {
        gl = gate_from_logit(gl);
        bl = beta_from_logit(bl);
    }
    // With the q/k L2 norm: 1 / |row| of K and Q row `lane` (rows past the end
    // repeat row L - 1, as the loads below do), for the fragments and the
    // staged rows alike, so that both use the same bf16 values.
    float* rnk = sm.rn[pc.pw][0];
    float* rnq = sm.rn[pc.pw][1];
    if constexpr (NORM) {
        const unsigned roff = (unsigned)min(lane, L - 1) * qks;
        rnk[lane] = row_inv_norm<D>(kc0 + roff);
        rnq[lane] = row_inv_norm<D>(qc0 + roff);
    }
    auto load_frags = [&](const uint16_t* base, const float* rn, int b, uint4 (&f)[4]) {
        const unsigned off = (unsigned)min(16 * b + m, L - 1) * qks + 8u * gq;
#pragma unroll
        for (int kq = 0; kq < 4; ++kq) f[kq] = ld16(base, 2u * off + 64u * kq);
        if constexpr (NORM) {
            const float r = rn[16 * b + m];
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) f[kq] = scale_bf16x8(f[kq], r);
        }
    };
    uint4 fk[NCT][4], fq[2][4];
#pragma unroll
    for (int b = 0; b < NCT; ++b) load_frags(kc0, rnk, b, fk[b]);
    load_frags(qc0, rnq, 0, fq[0]);
    const float gx = wave_prefix_sum(gl);
    const float glast = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gx), C - 1));
    gam[lane] = gx;
    bet[lane] = bl;
    float gr[NCT], br[NCT];  // gamma, beta of row 16 b + m
#pragma unroll
    for (int b = 0; b < NCT; ++b) {
        gr[b] = gam[16 * b + m];
        br[b] = bet[16 * b + m];
    }
    // ---- masked scores: tile (b, jt) of (M o Q K^T)^T, t = 16 b + m,
    //      s = 16 jt + 4 gq + i, packed to bf16 as row t of the block
    uint2 pk[NBLK];
#pragma unroll
    for (int b = 0; b < NCT; ++b) {
        if (b + 1 < NCT) load_frags(qc0, rnq, b + 1, fq[(b + 1) & 1]);
#pragma unroll
        for (int jt = 0; jt <= b; ++jt) {
            f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) acc = mma(as_frag(fk[jt][kq]), as_frag(fq[b & 1][kq]), acc);
            const f32x4_t gc = *reinterpret_cast<const f32x4_t*>(&gam[16 * jt + 4 * gq]);
            float val[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                val[i] = (jt < b || 4 * gq + i <= m) ? fast_exp(gr[b] - gc[i]) * (acc[i] * pc.scale) : 0.f;
            pk[bidx(b, jt)] = uint2{cvt_pk(val[0], val[1]), cvt_pk(val[2], val[3])};
        }
    }
    // ---- A = beta_r exp(gamma_r - gamma_c) (K K^T)_rc, c < r.
    //      Diagonal blocks: acc(-N_b^T) from the (symmetric) Gram tile;
    //      below the diagonal: acc(A_bk^T).
    f32x4_t nt[NCT], at[NBLK];
#pragma unroll
    for (int b = 0; b < NCT; ++b) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kq = 0; kq < 4; ++kq) acc = mma(as_frag(fk[b][kq]), as_frag(fk[b][kq]), acc);
        const f32x4_t gc = *reinterpret_cast<const f32x4_t*>(&gam[16 * b + 4 * gq]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            nt[b][i] = (4 * gq + i < m) ? -(br[b] * fast_exp(gr[b] - gc[i]) * acc[i]) : 0.f;
#pragma unroll
        for (int kb = 0; kb < b; ++kb) {
            f32x4_t ag = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) ag = mma(as_frag(fk[kb][kq]), as_frag(fk[b][kq]), ag);
            const f32x4_t gk = *reinterpret_cast<const f32x4_t*>(&gam[16 * kb + 4 * gq]);
#pragma unroll
            for (int i = 0; i < 4; ++i) at[bidx(b, kb)][i] = br[b] * fast_exp(gr[b] - gk[i]) * ag[i];
        }
    }
    // ---- T = (I + A)^-1: diagonal blocks D_b = (I + N_b)^-1 by forward
    //      substitution in fp32, lane 16 b + j solving column j of block b;
    //      then block columns T_bJ = -D_b sum_{kb=J}^{b-1} A_{b,kb} T_{kb,J}
    //      (b > J) on split-bf16 MFMA.
    // Lane 16 b + m holds row m of -N_b in registers (through the scratch
    // block, which transposes the accumulator layout); the solve takes
    // element i of row r from lane 16 b + r with a DPP row broadcast, so its
    // 120 multiply-adds wait on no LDS access.
    float* scb = scr + gq * SBS;  // this lane's block b = gq
#pragma unroll
    for (int b = 0; b < NCT; ++b)     // row m of -N_b, columns 4 gq .. 4 gq + 3
        *reinterpret_cast<f32x4_t*>(&scr[b * SBS + m * SP + 4 * gq]) = nt[b];
    f32x4_t nrow[4];
#pragma unroll
    for (int i4 = 0; i4 < 4; ++i4) nrow[i4] = *reinterpret_cast<const f32x4_t*>(&scb[m * SP + 4 * i4]);
    float xs[16];
    xs[0] = (m == 0) ? 1.f : 0.f;
#define GDN_SOLVE_ROW(R) xs[R] = fsolve_row<R>(nrow, xs, (R == m) ? 1.f : 0.f);
    GDN_SOLVE_ROW(1) GDN_SOLVE_ROW(2) GDN_SOLVE_ROW(3) GDN_SOLVE_ROW(4) GDN_SOLVE_ROW(5)
    GDN_SOLVE_ROW(6) GDN_SOLVE_ROW(7) GDN_SOLVE_ROW(8) GDN_SOLVE_ROW(9) GDN_SOLVE_ROW(10)
    GDN_SOLVE_ROW(11) GDN_SOLVE_ROW(12) GDN_SOLVE_ROW(13) GDN_SOLVE_ROW(14) GDN_SOLVE_ROW(15)
#undef GDN_SOLVE_ROW
#pragma unroll
    for (int r4 = 0; r4 < 16; r4 += 4)  // row m of the scratch block = column m of D_b
        *reinterpret_cast<f32x4_t*>(&scb[m * SP + r4]) = f32x4_t{xs[r4], xs[r4 + 1], xs[r4 + 2], xs[r4 + 3]};
    f32x4_t dd[NCT], ddt[NCT], tt[NBLK];
#pragma unroll
    for (int b = 0; b < NCT; ++b) {     // acc(D_b): D_b[4 gq + i][m]
        dd[b] = *reinterpret_cast<const f32x4_t*>(&scr[b * SBS + m * SP + 4 * gq]);
        if (b > 0) {                    // -acc(D_b^T): -D_b[m][4 gq + i]
#pragma unroll
            for (int i = 0; i < 4; ++i) ddt[b][i] = -scr[b * SBS + (4 * gq + i) * SP + m];
        }
    }
    {
        // block-column sweep on split bf16 products; every operand is split once
        const f32x4_t zero4 = {0.f, 0.f, 0.f, 0.f};
        Split16 sat[NBLK], sdd[NCT - 1], sdt[NCT], stt[NBLK];
#pragma unroll
        for (int bi = 1; bi < NCT; ++bi) {
            sdt[bi] = split16(ddt[bi]);
#pragma unroll
            for (int kb = 0; kb < bi; ++kb) sat[bidx(bi, kb)] = split16(at[bidx(bi, kb)]);
        }
#pragma unroll
        for (int J = 0; J + 1 < NCT; ++J) sdd[J] = split16(dd[J]);
#pragma unroll
        for (int bi = 1; bi < NCT; ++bi)
#pragma unroll
            for (int J = 0; J < bi; ++J) {
                f32x4_t y = prods(sat[bidx(bi, J)], sdd[J], zero4);
#pragma unroll
                for (int kb = J + 1; kb < bi; ++kb) y = prods(sat[bidx(bi, kb)], stt[bidx(kb, J)], y);
                tt[bidx(bi, J)] = prods(sdt[bi], split16(y), zero4);
                if (bi + 1 < NCT) stt[bidx(bi, J)] = split16(tt[bidx(bi, J)]);
            }
    }
    // ---- publish to the slot once the state waves are done with its
    //      previous chunk
    wait_ge(&sm.cnt[CNT_DONE], (unsigned)(x >= 4 ? NSIG * (x - 3) : 0), pc.fault);   // chunk x - 4 done
#pragma unroll
    for (int b = 0; b < NCT; ++b)
#pragma unroll
        for (int jt = 0; jt <= b; ++jt)
            *reinterpret_cast<uint2*>(&sl.pm[bidx(b, jt)][m][bsw(m, gq)]) = pk[bidx(b, jt)];
#pragma unroll
    for (int b = 0; b < NCT; ++b) {
        store_split_t(sl.th[bidx(b, b)], sl.tl[bidx(b, b)], dd[b], br[b], m, gq);
#pragma unroll
        for (int J = 0; J < b; ++J) store_split_t(sl.th[bidx(b, J)], sl.tl[bidx(b, J)], tt[bidx(b, J)], br[J], m, gq);
    }
    sl.eg[lane] = fast_exp(gx);
    sl.egl[lane] = fast_exp(glast - gx);
    signal(&sm.cnt[CNT_READY0 + pc.pw], lane);
    // ---- stage the chunk's K, Q, V rows once the state waves have
    //      released the previous chunk's (Q rows 0..31 read again: row 4 it +
    //      gq, segment m; rows 32..63 are the fragments of block rows 2 and 3
    //      the scores left in registers); stream chunk 0 was staged by the
    //      whole workgroup
    if (x == 0) return;
    // (The zero stores before the loads are dead; without them the compiler
    // kept these arrays in scratch memory across the waits below.)
    uint4 sq[SITEMS / 2];
#pragma unroll
    for (int it = 0; it < SITEMS / 2; ++it) {
        const unsigned off = (unsigned)min(4 * it + gq, L - 1) * qks + 8u * m;
        sq[it] = uint4{0, 0, 0, 0};
        sq[it] = ld16(qc0, 2u * off);
        if constexpr (NORM) sq[it] = scale_bf16x8(sq[it], rnq[min(4 * it + gq, L - 1)]);
    }
    // K buffer x & 1 was last read by the update of chunk x - 2.  The K rows
    // are the operand fragments loaded at the start (lane m + 16 gq holds
    // columns 32 kq + 8 gq .. + 7 of row 16 b + m), so they are written from
    // registers rather than read from memory a second time.
    wait_ge(&sm.cnt[CNT_DONE], (unsigned)(x >= 2 ? NSIG * (x - 1) : 0), pc.fault);
#pragma unroll
    for (int b = 0; b < NCT; ++b)
#pragma unroll
        for (int kq = 0; kq < 4; ++kq)
            *reinterpret_cast<uint4*>(&sm.kb[x & 1][16 * b + m][swz(16 * b + m, 32 * kq + 8 * gq)]) = fk[b][kq];
    // V rows of the workgroup's VB columns (VB / 8 lanes per row), loaded into
    // the registers the K rows held, so that their latency overlaps the wait
    // for the Q and V buffers
    // With 4 lanes per row, rows 2i + 1 and 2i + 2 swap their lanes, so that
    // each 8 lanes (one store cycle) write two rows 192 bytes apart, which
    // share no banks.
    constexpr int VLR = VB / 8, VRI = 64 / VLR, VIT = C / VRI;
    const int vq = lane / VLR, vsg = lane - vq * VLR;
    const int vr = VLR == 4 ? (vq & ~3) | ((vq & 1) << 1) | ((vq >> 1) & 1) : vq;
    const uint16_t* vc0 = pc.v + (size_t)tb * pc.v_stride + (size_t)pc.h * D + pc.vcb0;
    uint4 sv[VIT];
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
        sv[it] = uint4{0, 0, 0, 0};
        sv[it] = ld16_stream(vc0, 2u * ((unsigned)min(VRI * it + vr, L - 1) * (unsigned)pc.v_stride + 8u * vsg));
    }
    wait_ge(&sm.cnt[CNT_QVFREE], (unsigned)(NSIG * x), pc.fault);
#pragma unroll
    for (int it = 0; it < SITEMS / 2; ++it) *reinterpret_cast<uint4*>(&sm.qb[4 * it + gq][swz(4 * it + gq, m * 8)]) = sq[it];
#pragma unroll
    for (int b = 2; b < NCT; ++b)
#pragma unroll
        for (int kq = 0; kq < 4; ++kq)
            *reinterpret_cast<uint4*>(&sm.qb[16 * b + m][swz(16 * b + m, 32 * kq + 8 * gq)]) = fq[b & 1][kq];
#pragma unroll
    for (int it = 0; it < VIT; ++it)
        *reinterpret_cast<uint4*>(&sm.vb[VRI * it + vr][swz(VRI * it + vr, 8 * vsg)]) = sv[it];
    signal(&sm.cnt[CNT_STG], lane);
}

// NS state waves, each owning NVT 16-wide tiles of value columns; a workgroup
// covers NS * NVT * 16 of the D value columns of its head, so a head is split
// over VSPLIT = D / (16 NS NVT) workgroups (each repeating the producer work of
// the head), which spreads few long sequences over more compute units.
template <int NS, int NVT, int NO, int PRO>
__global__ __launch_bounds__(64 * (NS + NO + NP)) void prefill_pipe_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const float* __restrict__ g, const float* __restrict__ beta, const int32_t* __restrict__ cu,
    const int32_t* __restrict__ order, const float* initial_state, float* final_state,
    uint16_t* __restrict__ o, int N, int T, int H_qk, int H_v, float scale,
    const int32_t* __restrict__ state_idx, int P, int* fault) {
    constexpr bool NORM = (PRO & kFlagQkL2Norm) != 0;
    constexpr int VW = 16 * NVT;        // value columns per state wave
    constexpr int VB = NS * VW;         // value columns per workgroup
    constexpr int VSPLIT = D / VB;
    constexpr int NW = NS + NO + NP;    // waves per workgroup
    static_assert(VSPLIT * VB == D, "value columns must tile D");
    static_assert(NO == 0 || NO == NS, "one output wave per state wave");
    __shared__ Smem<VB, NO, NVT> sm;

    // no sequence longer than kRecurMax: all of them ran token by token
    if (order[N] == 0) return;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar chunk and address math
    const int m = lane & 15;
    const int gq = lane >> 4;

    // Work items of this workgroup: on pass p the virtual index p G + b (b, or
    // G - 1 - b on odd passes, which pairs long and short items) mapped to a
    // logical item; -1 past the last item.
    const int items = N * H_v * VSPLIT;
    const int G = gridDim.x;
    const int bid = blockIdx.x;
    auto item_at = [&](int pass) -> int { return pipe_item_at<VSPLIT>(pass, G, bid, items); };
    typedef PipeItem Item;
    auto decode = [&](int item) -> Item {
        return pipe_item_fields(item, VSPLIT, H_v, H_qk, order, cu, T, state_idx, P, C, kRecurMax);
    };
    const size_t qk_stride = (size_t)H_qk * D;
    const size_t v_stride = (size_t)H_v * D;

    // Every wave stages chunk 0 of the first non-empty item (chunk 0 of the
    // stream) before the roles split, so the state waves can start on it while
    // producer 0 prepares the rest.
    Item first = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int pass = 0;; ++pass) {
        const int item = item_at(pass);
        if (item < 0) break;
        first = decode(item);
        if (first.nch > 0) break;
    }
    if (tid < NCNT) sm.cnt[tid] = (tid == CNT_STG && first.nch > 0) ? 1u : 0u;
    for (int i = tid; i < 16 * 16; i += 64 * NW) (&sm.zero[0][0])[i] = 0;
    if (first.nch > 0) {
        const int L0 = min(C, first.seq_len);
        for (int i = tid; i < C * SEGS; i += 64 * NW) {
            const int r = i / SEGS, seg = i - r * SEGS;
            uint4 rk = {0, 0, 0, 0}, rq = {0, 0, 0, 0};
            if (r < L0) {
                const size_t row = (size_t)(first.seq_beg + r) * qk_stride + (size_t)first.hq * D;
                const size_t tq = row + seg * 8;
                rk = *reinterpret_cast<const uint4*>(k + tq);
                rq = *reinterpret_cast<const uint4*>(q + tq);
                if constexpr (NORM) {
                    rk = scale_bf16x8(rk, row_inv_norm<D>(k + row));
                    rq = scale_bf16x8(rq, row_inv_norm<D>(q + row));
                }
            }
            *reinterpret_cast<uint4*>(&sm.kb[0][r][swz(r, seg * 8)]) = rk;
            *reinterpret_cast<uint4*>(&sm.qb[r][swz(r, seg * 8)]) = rq;
        }
        for (int i = tid; i < C * (VB / 8); i += 64 * NW) {
            const int r = i / (VB / 8), seg = i - r * (VB / 8);
            uint4 rv = {0, 0, 0, 0};
            if (r < L0)
                rv = *reinterpret_cast<const uint4*>(v + (size_t)(first.seq_beg + r) * v_stride + (size_t)first.h * D +
                                                     first.vblock * VB + seg * 8);
            *reinterpret_cast<uint4*>(&sm.vb[r][swz(r, seg * 8)]) = rv;
        }
    }
    __syncthreads();

    if (wave < NS) {
        // ======================= state waves ===================================
        const SplitMasks spm = split_masks();
        int xs = 0;  // stream index of the next chunk
        // The counters chunk xs waits for, read at the end of chunk xs - 1
        // (their LDS round trip overlaps that chunk's output stores); a wait
        // reads again only if the value seen was short.  0: nothing seen yet.
        unsigned seen_stg = 0, seen_hs = 0, seen_rdy = 0, seen_hu = 0;
        float seen_egl = 0.f;  // the next chunk's exp(gamma_last), valid once seen_rdy says ready
        for (int pass = 0;; ++pass) {
        const int item = item_at(pass);
        if (item < 0) break;
        const Item it = decode(item);
        if (it.nch == 0) continue;  // a short sequence: the recurrent kernel's
        const int h = it.h, seq_beg = it.seq_beg, seq_len = it.seq_len, nch = it.nch;
        const size_t state_off = ((size_t)it.slot * H_v + h) * D * D;
        const int vcol0 = (it.vblock * NS + wave) * VW;
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

        for (int c = 0; c < nch; ++c, ++xs) {
            const int par = xs & 1;
            const int L = min(C, seq_len - c * C);
            const int t0 = seq_beg + c * C;
            const Slot& sl = sm.slot[xs % NP];
            const uint16_t (*kb)[PD] = sm.kb[par];
            // (uniform values, held in scalar registers through the chunk)
            const unsigned rdy_seen = __builtin_amdgcn_readfirstlane(seen_rdy);
            const unsigned hu_seen = __builtin_amdgcn_readfirstlane(seen_hu);
            wait_seen(&sm.cnt[CNT_STG], (unsigned)(xs + 1), seen_stg, fault);
            // with output waves: the previous chunk's S0 hi operands were read
            if constexpr (NO > 0) wait_seen(&sm.cnt[CNT_HAND0 + 4 * wave + 1], (unsigned)xs, seen_hs, fault);
            // K S0^T (S0 hi + lo, or hi alone), rows t; (Q S0^T)^T (S0 hi), rows
            // v, unless an output wave takes it (it gets the S0 hi operands
            // instead).
            // The lo half of S0 matters in K S0^T only while the state persists:
            // every term of the chunk's new state that depends on S0 carries
            // the chunk's total decay exp(gamma_last), so dropping S0 lo there
            // changes the state by about 2^-9 exp(gamma_last) of its size per
            // chunk, which later chunks decay further.  With exp(gamma_last) <=
            // kS0LoDecay the product takes S0 hi alone (uniform branches around
            // the lo split and products).  The decay comes from the chunk's
            // result slot, which for stream chunks after the first is ready
            // once the chunk is staged (a producer publishes before it
            // stages); stream chunk 0 waits for it here.  The choice depends
            // on the chunk's own gates only, never on the batch around it.
            // (The decay was read with the ready counter at the end of the
            // previous chunk; read again only if the slot was not ready then.)
            bool s0lo;
            {
                const unsigned target = (unsigned)(xs / NP + 1);
                float egl = seen_egl;
                if (rdy_seen < target) {
                    wait_ge(&sm.cnt[CNT_READY0 + xs % NP], target, fault);
                    egl = sl.eg[C - 1];
                }
                s0lo = __builtin_amdgcn_readfirstlane((int)(egl > kS0LoDecay)) != 0;
            }
            f32x4_t ks[NCT][NVT], ot[NVT][NCT];
            const f32x4_t zero4 = {0.f, 0.f, 0.f, 0.f};
            // Software pipeline over the contraction: the operand reads of step
            // kq + 1 are issued ahead of the products of step kq (the barrier
            // keeps the scheduler from sinking them towards their use), and
            // the split of step kq + 1 is interleaved with those products.  The
            // lo halves (split and products) sit in uniform branches of their
            // own; each accumulator still takes hi then lo of every step.
            bf16x8_t ak[2][NCT], aq[2][NCT], bh[2][NVT], bl[2][NVT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
                ak[0][ct] = row_frag(kb, 16 * ct + m, 0, gq);
                if constexpr (NO == 0) aq[0][ct] = row_frag(sm.qb, 16 * ct + m, 0, gq);
            }
            auto split_s0 = [&](int kq, int buf) {
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) {
                    bh[buf][vt] = acc_frag_hi<32>(st[2 * kq][vt], st[2 * kq + 1][vt]);
                    if constexpr (NO > 0)
                        sm.hs[wave % (NO > 0 ? NO : 1)][kq][vt][lane] = __builtin_bit_cast(uint4, bh[buf][vt]);
                }
                if (s0lo) {
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt)
                        bl[buf][vt] = acc_frag_lo32(st[2 * kq][vt], st[2 * kq + 1][vt], bh[buf][vt]);
                }
            };
            split_s0(0, 0);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kq = 0; kq < D / 32; ++kq) {
                const int cur = kq & 1;
                if (kq + 1 < D / 32) {
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        ak[cur ^ 1][ct] = row_frag(kb, 16 * ct + m, 32 * (kq + 1), gq);
                        if constexpr (NO == 0) aq[cur ^ 1][ct] = row_frag(sm.qb, 16 * ct + m, 32 * (kq + 1), gq);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        ks[ct][vt] = mma(ak[cur][ct], bh[cur][vt], kq == 0 ? zero4 : ks[ct][vt]);
                        if constexpr (NO == 0) ot[vt][ct] = mma(bh[cur][vt], aq[cur][ct], kq == 0 ? zero4 : ot[vt][ct]);
                    }
                if (kq + 1 < D / 32) {
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        bh[cur ^ 1][vt] = acc_frag_hi<32>(st[2 * kq + 2][vt], st[2 * kq + 3][vt]);
                        if constexpr (NO > 0)
                            sm.hs[wave % (NO > 0 ? NO : 1)][kq + 1][vt][lane] = __builtin_bit_cast(uint4, bh[cur ^ 1][vt]);
                    }
                }
#pragma unroll
                for (int i = 0; i < 12 * NVT; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
                    __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);   // VALU
                }
                __builtin_amdgcn_sched_barrier(0);
                if (s0lo) {
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt) ks[ct][vt] = mma(ak[cur][ct], bl[cur][vt], ks[ct][vt]);
                    if (kq + 1 < D / 32) {
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt)
                            bl[cur ^ 1][vt] = acc_frag_lo32(st[2 * kq + 2][vt], st[2 * kq + 3][vt], bh[cur ^ 1][vt]);
                    }
#pragma unroll
                    for (int i = 0; i < NCT * NVT; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
                        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);   // VALU
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (NO > 0) signal(&sm.cnt[CNT_HAND0 + 4 * wave + 0], lane);
            // W = V - diag(exp(gamma)) K S0^T (in ks)
            // T operands of U = T diag(beta) W, read now so that their latency
            // hides behind the vector work of W
            bf16x8_t tah[NCT][2], tal[NCT][2];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int hb = 0; hb < 2; ++hb) {
                    if (32 * hb > 16 * ct + 15) continue;
                    tah[ct][hb] = blk_frag_t(sl.th, sm.zero, ct, 32 * hb, m, gq);
                    tal[ct][hb] = blk_frag_t(sl.tl, sm.zero, ct, 32 * hb, m, gq);
                }
            f32x4_t egr[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) egr[ct] = *reinterpret_cast<const f32x4_t*>(&sl.eg[16 * ct + 4 * gq]);
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) {
                    // V[16 ct + 4 gq + i][vcol0 + 16 vt + m], i = 0..3
                    const int vr = 4 * gq + (m >> 2);
                    const uint2 vv = lds_tr4(&sm.vb[16 * ct + vr][wave * VW + 16 * vt + swz(vr, 4 * (m & 3))]);
                    const float vf[4] = {bf16_to_f32(vv.x & 0xFFFFu), bf16_to_f32(vv.x >> 16),
                                         bf16_to_f32(vv.y & 0xFFFFu), bf16_to_f32(vv.y >> 16)};
#pragma unroll
                    for (int i = 0; i < 4; ++i) ks[ct][vt][i] = fmaf(-egr[ct][i], ks[ct][vt][i], vf[i]);
                }
            signal(&sm.cnt[CNT_QVFREE], lane);
            // U = T diag(beta) W  (hi*hi + hi*lo + lo*hi); the split of the
            // second half of W overlaps the products of the first.
            f32x4_t uu[NCT][NVT];
            bf16x8_t wh[2][NVT], wl[2][NVT];
#pragma unroll
            for (int vt = 0; vt < NVT; ++vt) acc_frag(ks[0][vt], ks[1][vt], wh[0][vt], wl[0][vt], spm);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kc = 0; kc < C; kc += 32) {
                const int hb = kc / 32;
                if (hb == 0) {
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) acc_frag(ks[2][vt], ks[3][vt], wh[1][vt], wl[1][vt], spm);
                }
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    if (kc > 16 * ct + 15) continue;
                    const bf16x8_t& ah = tah[ct][hb];
                    const bf16x8_t& al = tal[ct][hb];
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) {
                        const f32x4_t u0 = (kc == 0) ? zero4 : uu[ct][vt];
                        uu[ct][vt] = mma(ah, wh[hb][vt], u0);
                        uu[ct][vt] = mma(ah, wl[hb][vt], uu[ct][vt]);
                        uu[ct][vt] = mma(al, wh[hb][vt], uu[ct][vt]);
                    }
                }
                if (hb == 0) {
                    // groups of one MFMA and two vector instructions with
                    // output waves, of three and six without (each measured
                    // the faster of the two for its variant)
                    constexpr int GM = NO > 0 ? 1 : 3;
#pragma unroll
                    for (int i = 0; i < 12 * NVT / GM; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, GM, 0);       // MFMA
                        __builtin_amdgcn_sched_group_barrier(0x002, 2 * GM, 0);   // VALU
                    }
                }
            }
            if constexpr (NO > 0) {
                // the previous chunk's U hi operands were read
                wait_seen(&sm.cnt[CNT_HAND0 + 4 * wave + 3], (unsigned)xs, hu_seen, fault);
#pragma unroll
                for (int kc = 0; kc < C; kc += 32)
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt)
                        sm.hu[wave % (NO > 0 ? NO : 1)][kc / 32][vt][lane] =
                            __builtin_bit_cast(uint4, acc_frag_hi<32>(uu[kc / 16][vt], uu[kc / 16 + 1][vt]));
                signal(&sm.cnt[CNT_HAND0 + 4 * wave + 2], lane);
            }
            // S^T = exp(gamma_last) S^T + K^T (diag(exp(gamma_last - gamma)) U)   (hi + lo),
            // block row by block row of S^T so that the scaling of one overlaps
            // the products of the previous
            f32x4_t eglv[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) eglv[ct] = *reinterpret_cast<const f32x4_t*>(&sl.egl[16 * ct + 4 * gq]);
            const float eg_last = sl.eg[C - 1];
            // P operands of the output products, read ahead of the update
            bf16x8_t pf[NCT][2];
            if constexpr (NO == 0) {
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int hb = 0; hb < 2; ++hb) {
                        if (32 * hb > 16 * ct + 15) continue;
                        pf[ct][hb] = blk_frag(sl.pm, sm.zero, ct, 32 * hb, m, gq);
                    }
            }
            bf16x8_t uth[2][NVT], utl[2][NVT];
#pragma unroll
            for (int hb = 0; hb < 2; ++hb)
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt)
                    acc_frag(uu[2 * hb][vt] * eglv[2 * hb], uu[2 * hb + 1][vt] * eglv[2 * hb + 1], uth[hb][vt], utl[hb][vt], spm);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                const bf16x8_t a0 = lds_frag_tr(kb, 0, 16 * dt, m, gq);
                const bf16x8_t a1 = lds_frag_tr(kb, 32, 16 * dt, m, gq);
#pragma unroll
                for (int vt = 0; vt < NVT; ++vt) {
                    st[dt][vt] *= eg_last;
                    st[dt][vt] = mma(a0, uth[0][vt], st[dt][vt]);
                    st[dt][vt] = mma(a0, utl[0][vt], st[dt][vt]);
                    st[dt][vt] = mma(a1, uth[1][vt], st[dt][vt]);
                    st[dt][vt] = mma(a1, utl[1][vt], st[dt][vt]);
                }
            }
            if constexpr (NO == 0) {
                // scale O^T = scale diag(exp(gamma)) (Q S0^T)^T + U^T (scale M o Q K^T)^T
                // (U hi); its vector work overlaps the update's products
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const float e = sl.eg[16 * ct + m] * scale;
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) ot[vt][ct] *= e;
                }
#pragma unroll
                for (int kc = 0; kc < C; kc += 32) {
                    bf16x8_t uh[NVT];
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) uh[vt] = acc_frag_hi<32>(uu[kc / 16][vt], uu[kc / 16 + 1][vt]);
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        if (kc > 16 * ct + 15) continue;
                        const bf16x8_t& bp = pf[ct][kc / 32];
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt) ot[vt][ct] = mma(uh[vt], bp, ot[vt][ct]);
                    }
                }
            }
            // all LDS reads of chunk c are done: its K buffer and result slot are free
            signal(&sm.cnt[CNT_DONE], lane);
            seen_stg = peek(&sm.cnt[CNT_STG]);
            seen_rdy = peek(&sm.cnt[CNT_READY0 + (xs + 1) % NP]);
            // read after the counter (the LDS serves a wave's operations in
            // order; the fence keeps the compiler from swapping them), so a
            // ready value seen means this is the published decay
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
            seen_egl = __hip_atomic_load(&sm.slot[(xs + 1) % NP].eg[C - 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            if constexpr (NO > 0) {
                seen_hs = peek(&sm.cnt[CNT_HAND0 + 4 * wave + 1]);
                seen_hu = peek(&sm.cnt[CNT_HAND0 + 4 * wave + 3]);
            }
            if constexpr (NO == 0) {
                // Outputs: lane m + 16 gq holds, in ot[vt][ct], token 16 ct + m and
                // value columns 16 vt + 4 gq .. + 3.  Two such tiles x, y are merged
                // by a swap between lane groups gq and gq ^ 1 (v_permlane16_swap:
                // group 2i ends with x of groups 2i, 2i + 1, group 2i + 1 with y of
                // both), so that each lane stores 8 consecutive columns (16 bytes):
                // x, y are the two value tiles when NVT is even, else token blocks
                // ct and ct + 1.
                const int odd = gq & 1, half = gq >> 1;
                auto store_pair = [&](const f32x4_t& x, const f32x4_t& y, int row, int col) {
                    const auto p0 = __builtin_amdgcn_permlane16_swap(cvt_pk(x[0], x[1]), cvt_pk(y[0], y[1]), false, false);
                    const auto p1 = __builtin_amdgcn_permlane16_swap(cvt_pk(x[2], x[3]), cvt_pk(y[2], y[3]), false, false);
                    const uint4 pk = {p0[0], p1[0], p0[1], p1[1]};
                    if (row < L)
                        *reinterpret_cast<uint4*>(o + (size_t)(t0 + row) * v_stride + (size_t)h * D + vcol0 + col) = pk;
                };
                if constexpr (NVT % 2 == 0) {
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int vt = 0; vt < NVT; vt += 2)
                            store_pair(ot[vt][ct], ot[vt + 1][ct], 16 * ct + m, 16 * vt + 16 * odd + 8 * half);
                } else {
#pragma unroll
                    for (int ct = 0; ct < NCT; ct += 2)
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt)
                            store_pair(ot[vt][ct], ot[vt][ct + 1], 16 * (ct + odd) + m, 16 * vt + 8 * half);
                }
            }
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int vt = 0; vt < NVT; ++vt) {
                const float4 s4 = {st[dt][vt][0], st[dt][vt][1], st[dt][vt][2], st[dt][vt][3]};
                *reinterpret_cast<float4*>(final_state + state_off + (size_t)(vcol0 + 16 * vt + m) * D +
                                           16 * dt + 4 * gq) = s4;
            }
        }
    } else if (wave < NS + NO) {
        // ======================= output waves ==================================
        // Output wave w finishes the chunks of state wave w: (Q S0^T)^T from
        // the handed-over S0 hi operands, then the output products with the
        // handed-over U hi operands, then the stores.
        const int w = wave - NS;
        int xs = 0;
        for (int pass = 0;; ++pass) {
            const int item = item_at(pass);
            if (item < 0) break;
            const Item it = decode(item);
            const int vcol0 = (it.vblock * NS + w) * VW;
            for (int c = 0; c < it.nch; ++c, ++xs) {
                const int L = min(C, it.seq_len - c * C);
                const int t0 = it.seq_beg + c * C;
                const Slot& sl = sm.slot[xs % NP];
                const f32x4_t zero4 = {0.f, 0.f, 0.f, 0.f};
                // the chunk's Q operands go to registers at once, so that the Q
                // buffer is released before the S0 operands arrive
                wait_ge(&sm.cnt[CNT_STG], (unsigned)(xs + 1), fault);
                bf16x8_t aq[D / 32][NCT];
#pragma unroll
                for (int kq = 0; kq < D / 32; ++kq)
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) aq[kq][ct] = row_frag(sm.qb, 16 * ct + m, 32 * kq, gq);
                signal(&sm.cnt[CNT_QVFREE], lane);
                wait_ge(&sm.cnt[CNT_HAND0 + 4 * w + 0], (unsigned)(xs + 1), fault);
                bf16x8_t bh[D / 32][NVT];
#pragma unroll
                for (int kq = 0; kq < D / 32; ++kq)
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) bh[kq][vt] = __builtin_bit_cast(bf16x8_t, sm.hs[w % (NO > 0 ? NO : 1)][kq][vt][lane]);
                signal(&sm.cnt[CNT_HAND0 + 4 * w + 1], lane);
                f32x4_t ot[NVT][NCT];
#pragma unroll
                for (int kq = 0; kq < D / 32; ++kq)
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt) ot[vt][ct] = mma(bh[kq][vt], aq[kq][ct], kq == 0 ? zero4 : ot[vt][ct]);
                wait_ge(&sm.cnt[CNT_READY0 + xs % NP], (unsigned)(xs / NP + 1), fault);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const float e = sl.eg[16 * ct + m] * scale;
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) ot[vt][ct] *= e;
                }
                bf16x8_t pf[NCT][2];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                    for (int hb = 0; hb < 2; ++hb) {
                        if (32 * hb > 16 * ct + 15) continue;
                        pf[ct][hb] = blk_frag(sl.pm, sm.zero, ct, 32 * hb, m, gq);
                    }
                wait_ge(&sm.cnt[CNT_HAND0 + 4 * w + 2], (unsigned)(xs + 1), fault);
                bf16x8_t uh[C / 32][NVT];
#pragma unroll
                for (int kc = 0; kc < C / 32; ++kc)
#pragma unroll
                    for (int vt = 0; vt < NVT; ++vt) uh[kc][vt] = __builtin_bit_cast(bf16x8_t, sm.hu[w % (NO > 0 ? NO : 1)][kc][vt][lane]);
                signal(&sm.cnt[CNT_HAND0 + 4 * w + 3], lane);
#pragma unroll
                for (int kc = 0; kc < C; kc += 32)
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        if (kc > 16 * ct + 15) continue;
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt) ot[vt][ct] = mma(uh[kc / 32][vt], pf[ct][kc / 32], ot[vt][ct]);
                    }
                // all LDS reads of the chunk by this wave are done
                signal(&sm.cnt[CNT_DONE], lane);
                // outputs: token blocks ct and ct + 1 (or the value tiles) merged by
                // a swap between lane groups, 8 consecutive columns per lane
                const int odd = gq & 1, half = gq >> 1;
                auto store_pair = [&](const f32x4_t& x, const f32x4_t& y, int row, int col) {
                    const auto p0 = __builtin_amdgcn_permlane16_swap(cvt_pk(x[0], x[1]), cvt_pk(y[0], y[1]), false, false);
                    const auto p1 = __builtin_amdgcn_permlane16_swap(cvt_pk(x[2], x[3]), cvt_pk(y[2], y[3]), false, false);
                    const uint4 pk = {p0[0], p1[0], p0[1], p1[1]};
                    if (row < L)
                        *reinterpret_cast<uint4*>(o + (size_t)(t0 + row) * v_stride + (size_t)it.h * D + vcol0 + col) = pk;
                };
                if constexpr (NVT % 2 == 0) {
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
                        for (int vt = 0; vt < NVT; vt += 2)
                            store_pair(ot[vt][ct], ot[vt + 1][ct], 16 * ct + m, 16 * vt + 16 * odd + 8 * half);
                } else {
#pragma unroll
                    for (int ct = 0; ct < NCT; ct += 2)
#pragma unroll
                        for (int vt = 0; vt < NVT; ++vt)
                            store_pair(ot[vt][ct], ot[vt][ct + 1], 16 * (ct + odd) + m, 16 * vt + 8 * half);
                }
            }
        }
    } else {
        // ======================= producer waves ================================
        ProdCtx pc = {q, k, v, g, beta, qk_stride, v_stride, 0, 0, 0, 0, H_v, wave - NS - NO, 0, scale, fault};
        // stream chunks x = pw, pw + NP, ...: the work item holding chunk x
        // starts at stream index xbeg
        int pass = 0, xbeg = 0;
        int item = item_at(0);
        Item it = item >= 0 ? decode(item) : first;
        for (int x = wave - NS - NO; item >= 0; x += NP) {
            while (item >= 0 && x >= xbeg + it.nch) {
                xbeg += it.nch;
                item = item_at(++pass);
                if (item >= 0) it = decode(item);
            }
            if (item < 0) break;
            pc.seq_beg = it.seq_beg;
            pc.seq_len = it.seq_len;
            pc.hq = it.hq;
            pc.h = it.h;
            pc.vcb0 = it.vblock * VB;
            int mo = m, go = gq;
            asm volatile("" : "+v"(mo), "+v"(go));
            produce_chunk<NS + NO, VB, PRO>(sm, pc, x, x - xbeg, mo, go);
        }
    }
}

}  // namespace pipe

int device_compute_units() {
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
    if (dev < 64 && cache[dev] > 0) return cache[dev];
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    if (dev < 64) cache[dev] = n;
    return n;
}

// One workgroup per compute unit (the LDS use admits one), each walking its
// work items; fewer items than compute units give one item per workgroup.
template <int NS, int NVT, int NO, int PRO>
static hipError_t launch_pipe_pro(const PrefillArgs& a, int32_t* order, hipStream_t stream) {
    constexpr int VSPLIT = pipe::D / (16 * NS * NVT);
    const long items = (long)a.N * a.H_v * VSPLIT;
    const long grid = std::min<long>(items, device_compute_units());
    hipLaunchKernelGGL((pipe::prefill_pipe_kernel<NS, NVT, NO, PRO>), dim3((unsigned)grid),
                       dim3(64 * (NS + NO + pipe::NP)), 0, stream, (const uint16_t*)a.q, (const uint16_t*)a.k,
                       (const uint16_t*)a.v, a.g, a.beta, a.cu_seqlens, order, a.initial_state, a.final_state,
                       (uint16_t*)a.o, a.N, a.T, a.H_qk, a.H_v, a.scale, a.state_idx, a.P, order + a.N + 1);
    return hipGetLastError();
}

// The kernel instantiated for the requested prologue (none: the plain kernel).
template <int NS, int NVT, int NO>
static hipError_t launch_pipe(const PrefillArgs& a, int32_t* order, hipStream_t stream) {
    switch (a.flags & (kFlagQkL2Norm | kFlagGateLogits)) {
        case kFlagQkL2Norm: return launch_pipe_pro<NS, NVT, NO, kFlagQkL2Norm>(a, order, stream);
        case kFlagGateLogits: return launch_pipe_pro<NS, NVT, NO, kFlagGateLogits>(a, order, stream);
        case kFlagQkL2Norm | kFlagGateLogits:
            return launch_pipe_pro<NS, NVT, NO, kFlagQkL2Norm | kFlagGateLogits>(a, order, stream);
        default: return launch_pipe_pro<NS, NVT, NO, 0>(a, order, stream);
    }
}

// One workgroup per (sequence, head) when there are enough of them to fill the
// device; otherwise each head's value columns are split over 2 or 4
// workgroups (one workgroup per compute unit fits in LDS).
hipError_t launch_prefill_pipe(const PrefillArgs& a, int32_t* order, hipStream_t stream) {
    const long heads = (long)a.N * a.H_v;
    const long cus = device_compute_units();
    if (heads * 4 <= cus) return launch_pipe<2, 1, 2>(a, order, stream);
    if (heads * 2 <= cus) return launch_pipe<4, 1, 0>(a, order, stream);
    return launch_pipe<4, 2, 0>(a, order, stream);
}

}  // namespace gdn
