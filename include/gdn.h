/*
 * gdn.h -- C ABI of the MI355X (gfx950) Gated DeltaNet library.
 *
 * The operation (paper: appendix "Operator Background and Mathematical
 * Definitions", subsection "Gated Delta Net", the gated delta rule), per
 * sequence and value head, token by token:
 *
 *     S_t = S_{t-1} ( alpha_t (I - beta_t k_t k_t^T) ) + beta_t v_t k_t^T
 *     o_t = scale * S_t q_t,          alpha_t = exp(g_t)
 *
 * in the two execution regimes the same subsection names: decode (one new
 * token per sequence on a prior state) and prefill (whole packed sequences,
 * returning every output and the final state).
 *
 * Conventions shared by every entry point:
 *   - Pointers are DEVICE pointers unless stated otherwise.  Tensors are dense
 *     and row-major (last index contiguous).  bf16 tensors are passed as
 *     untyped pointers to 2-byte IEEE bfloat16 values.
 *   - The state S of one (sequence, value head) is d_v x d_k fp32, stored with
 *     the k index contiguous: state[..., i, j] = S[i][j], i < d_v, j < d_k.
 *   - Value head h reads q/k head floor(h * H_qk / H_v) (H_v must be a multiple
 *     of H_qk; consecutive value heads share a q/k head).
 *   - g is the natural-log gate (alpha = exp(g), normally g <= 0); beta is the
 *     write strength, one fp32 scalar per (token, value head).
 *   - o is written as bf16, rounded to nearest even from fp32.
 *   - Ownership: the caller owns every buffer; the library allocates, frees
 *     and synchronises nothing.  Calls are asynchronous on `stream`
 *     (a hipStream_t; NULL = the null stream).
 *   - Supported shapes: d_k == d_v == D with D in {16, 128}; prefill chunk
 *     C = 16 for D = 16 and C = 64 for D = 128.
 *   - Alignment: q, k, v, o and state pointers must be 16-byte aligned;
 *     g, beta and cu_seqlens 4-byte aligned.
 *   - Errors: every argument check runs on the host before any HIP call.  A
 *     failed check returns a negative gdn_status, records a message for
 *     gdn_last_error() and launches nothing.  A failed launch returns GDN_EHIP.
 *     Faults inside a kernel surface at the caller's next synchronisation.
 *   - Not re-entrant on overlapping outputs: two calls in flight that write the
 *     same state or output memory race.
 */
#ifndef GDN_MI355X_H
#define GDN_MI355X_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define GDN_API __attribute__((visibility("default")))
#else
#define GDN_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gdn_status {
    GDN_OK = 0,
    GDN_EINVAL = -1,       /* null pointer, negative size, bad head ratio, bad cu_seqlens */
    GDN_EUNSUPPORTED = -2, /* head dim or chunk size outside the supported set */
    GDN_EALIGN = -3,       /* pointer not aligned as required */
    GDN_EWORKSPACE = -4,   /* workspace missing or smaller than required */
    GDN_EHIP = -5          /* a HIP runtime call or kernel launch failed */
} gdn_status;

/* Flags of the _ex entry points (bitwise or). */
enum gdn_flags {
    /* q and k are not assumed L2-normalised: each (token, q/k head) row x is
     * replaced by bf16(x * r), r = 1 / sqrt(sum_i x_i^2 + 1e-6), computed in
     * fp32 from the bf16 inputs (sum in index order, correctly rounded square
     * root and division, then round to nearest even), before any other use. */
    GDN_QK_L2NORM = 1,
    /* g and beta hold logits a, b: g = -softplus(a) (so alpha = exp(g) =
     * sigmoid(-a)) and beta = sigmoid(b), computed in fp32 in the kernel. */
    GDN_GATE_LOGITS = 2,
    /* prefill only: the caller promises every sequence has at most 8 tokens
     * (a multi-token decode step, see gdn_decode_multitoken). */
    GDN_SHORT_ONLY = 4
};

/* Message for the most recent non-OK status returned on the calling host
 * thread ("" if none).  The pointer stays valid until the next library call
 * on that thread. */
GDN_API const char* gdn_last_error(void);

/* Library ABI version (major * 100 + minor). */
GDN_API int gdn_abi_version(void);

/*
 * gdn_decode -- one recurrent step for B sequences (the decode regime).
 *
 *   q, k   bf16 [B, H_qk, D]
 *   v      bf16 [B, H_v, D]
 *   g      fp32 [B, H_v]            log gate, alpha = exp(g)
 *   beta   fp32 [B, H_v]
 *   state  fp32 [B, H_v, D, D]      read, then overwritten IN PLACE with S_t
 *   o      bf16 [B, H_v, D]         o = scale * S_t q  (post-update state)
 *
 * Each state is streamed through HBM once.  B = 0 is a no-op returning GDN_OK
 * (pointers are then not checked).  `o` must not overlap any input.
 */
GDN_API int gdn_decode(const void* q, const void* k, const void* v,
               const float* g, const float* beta,
               float* state, void* o,
               int B, int H_qk, int H_v, int D_k, int D_v,
               float scale, void* stream);

/*
 * gdn_decode_indexed -- gdn_decode on states kept in a pool of P slots, as a
 * server keeps one state per request rather than per batch position: batch
 * entry b updates slot state_idx[b].
 *
 *   state_pool  fp32 [P, H_v, D, D]  the slots named in state_idx are read,
 *                                    then overwritten IN PLACE; others untouched
 *   state_idx   int32 [B], device    slot of each batch entry.  Entries outside
 *                                    [0, P) are skipped (their state and o rows
 *                                    are not touched), so -1 marks padding.
 *                                    Slots must be distinct within one call
 *                                    (a repeated slot is a data race).  The
 *                                    library never reads it on the host.
 *   P           number of slots
 *
 * The other arguments are those of gdn_decode.  B = 0 or P = 0 is a no-op
 * returning GDN_OK.  Errors as gdn_decode, plus GDN_EINVAL for P < 0, a NULL
 * state_idx or P * H_v > 2^30, GDN_EALIGN for a state_idx that is not 4-byte
 * aligned.
 */
GDN_API int gdn_decode_indexed(const void* q, const void* k, const void* v,
               const float* g, const float* beta,
               float* state_pool, const int32_t* state_idx, void* o,
               int B, int P, int H_qk, int H_v, int D_k, int D_v,
               float scale, void* stream);

/*
 * Bytes of device workspace gdn_prefill_varlen (and the other prefill-regime
 * entry points) needs for N sequences of T tokens in total with H_v value
 * heads: the longest-first schedule (one int32 per sequence), one int32 count
 * of the sequences run in chunks and one int32 wait-fault word, rounded up to
 * 256 bytes.  T, H_v and the head dims enter only through validation today;
 * they are part of the signature so that the size may depend on them.
 * Returns 0 for invalid arguments (negative N or T, H_v <= 0, d_k != d_v,
 * a head dim outside {16, 128} or a chunk other than the one for that dim).
 */
GDN_API size_t gdn_prefill_workspace_size(int N, int T, int H_v, int D_k, int D_v, int chunk);

/*
 * gdn_prefill_varlen -- packed variable-length prefill (the prefill regime),
 * computed in chunks of `chunk` tokens aligned to each sequence's first token
 * (the last chunk of a sequence may be shorter); the result equals the
 * token-by-token recurrence up to rounding.
 *
 *   q, k           bf16 [T, H_qk, D]
 *   v              bf16 [T, H_v, D]
 *   g, beta        fp32 [T, H_v]
 *   cu_seqlens     int32 [N + 1], device: sequence n is tokens
 *                  [cu_seqlens[n], cu_seqlens[n+1]).  Must hold cu[0] = 0,
 *                  non-decreasing, cu[N] = T.  The library never reads it on
 *                  the host; on the device every kernel clamps each
 *                  sequence's offsets into [0, T] (begin clamp(cu[n], 0, T),
 *                  end clamp(cu[n+1], begin, T)), so a malformed cu_seqlens
 *                  never leads to an access outside the T tokens, and the
 *                  call's first launch checks it and sets bit 2 of the fault
 *                  word (see workspace): the results of such a call are
 *                  meaningless.  Zero-length sequences are allowed: their
 *                  final state is their initial state.
 *   initial_state  fp32 [N, H_v, D, D] or NULL (zero state)
 *   final_state    fp32 [N, H_v, D, D]; may be the same pointer as
 *                  initial_state (in-place), must not partially overlap it.
 *   o              bf16 [T, H_v, D]
 *   workspace      device buffer of at least
 *                  gdn_prefill_workspace_size(...) bytes, 256-byte aligned;
 *                  its contents are scratch (overwritten by each call).  Once
 *                  the call has completed on the stream, int32 word N + 1 of
 *                  it (the fault word) is 0, or has bit 0 set if a wave of
 *                  the chunk kernel gave up one of its bounded waits for
 *                  another wave (a broken synchronisation, never expected),
 *                  or bit 2 if cu_seqlens was malformed: the call's results
 *                  are then invalid.  A diagnostic read, not a status
 *                  the call returns (the call does not wait for its kernels);
 *                  a call that is a no-op (N = 0) leaves the workspace as it
 *                  was.
 *
 * For D = 128, sequences of at most 8 tokens are computed token by token in
 * fp32 (the decode arithmetic), longer ones in chunks; the choice depends
 * only on each sequence's own length, so a sequence's result does not depend
 * on the rest of the batch.  With initial_state == final_state and short
 * sequences this call is a multi-token decode step (n new tokens per
 * sequence, cu_seqlens = [0, n, 2n, ...]); for n <= 8 it equals n calls of
 * gdn_decode bit for bit.
 *
 * N = 0 is a no-op returning GDN_OK.  Size limits (GDN_EINVAL otherwise):
 * T * H_v <= 2^24 and N * H_v <= 2^30.
 */
GDN_API int gdn_prefill_varlen(const void* q, const void* k, const void* v,
                       const float* g, const float* beta,
                       const int32_t* cu_seqlens,
                       const float* initial_state, float* final_state,
                       void* o,
                       int N, int T, int H_qk, int H_v, int D_k, int D_v,
                       int chunk, float scale,
                       void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * gdn_prefill_varlen_noalloc -- gdn_prefill_varlen for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same arguments without the
 * workspace, and the same kernels and results bit for bit.  The workspace is
 * a static device array of the library (one copy per GPU, about 64 KiB, held
 * until the process ends), so N is limited to 16,384 sequences (GDN_EWORKSPACE
 * beyond that, before any HIP call).  The call allocates and frees nothing;
 * its first call on a device looks up the array's address there (no
 * allocation).  Every call on one GPU shares that array and each call's first
 * launch rewrites what it needs, so calls that overlap in time on one GPU
 * (concurrent streams, or host threads) race and must not be issued; calls
 * one after another on a stream are fine.  The wait-fault word of the
 * workspace is not reported by this entry point.  Other errors as
 * gdn_prefill_varlen.
 */
GDN_API int gdn_prefill_varlen_noalloc(const void* q, const void* k, const void* v,
                       const float* g, const float* beta,
                       const int32_t* cu_seqlens,
                       const float* initial_state, float* final_state,
                       void* o,
                       int N, int T, int H_qk, int H_v, int D_k, int D_v,
                       int chunk, float scale, void* stream);

/*
 * gdn_prefill_varlen_indexed -- gdn_prefill_varlen on states kept in a pool
 * of P slots: sequence n starts from slot state_idx[n] and leaves its final
 * state there (in place).  Serving code keeps one state per request; a new
 * request's slot is zeroed by the caller first, and a few new tokens per
 * sequence make this a multi-token decode step on pooled states.
 *
 *   state_pool  fp32 [P, H_v, D, D]  the slots named in state_idx are read,
 *                                    then overwritten IN PLACE; others untouched
 *   state_idx   int32 [N], device    slot of each sequence.  Sequences whose
 *                                    entry is outside [0, P) are skipped: their
 *                                    outputs are not written.  Slots must be
 *                                    distinct within one call.  The library
 *                                    never reads it on the host.
 *   P           number of slots
 *
 * The other arguments are those of gdn_prefill_varlen (same workspace size,
 * same routes).  N = 0 or P = 0 is a no-op returning GDN_OK.  Errors as
 * gdn_prefill_varlen, plus GDN_EINVAL for P < 0, a NULL state_idx or
 * P * H_v > 2^30, GDN_EALIGN for a state_idx that is not 4-byte aligned.
 */
GDN_API int gdn_prefill_varlen_indexed(const void* q, const void* k, const void* v,
                       const float* g, const float* beta,
                       const int32_t* cu_seqlens,
                       float* state_pool, const int32_t* state_idx,
                       void* o,
                       int N, int T, int P, int H_qk, int H_v, int D_k, int D_v,
                       int chunk, float scale,
                       void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * gdn_decode_multitoken -- a decode step of a few new tokens per sequence
 * (the decode regime with n <= 8 updates per state, the state updated in
 * place): the recurrence of gdn_prefill_varlen for sequences the caller
 * promises are at most 8 tokens long.  It runs only the token-by-token
 * kernel, sparing gdn_prefill_varlen's second launch, which that call cannot
 * rule out because it never reads cu_seqlens on the host.  Results equal
 * gdn_prefill_varlen with initial_state == final_state == state bit for bit,
 * and hence n calls of gdn_decode.
 *
 *   q, k, v, g, beta, cu_seqlens, o, scale   as gdn_prefill_varlen (D = 128)
 *   state      fp32 [N, H_v, D, D], read and overwritten IN PLACE
 *   workspace  gdn_prefill_workspace_size(N, T, H_v, 128, 128, 64)
 *              bytes, 256-byte aligned.  After the call has completed, bit 1
 *              of int32 word N + 1 is set if some sequence was longer than 8
 *              tokens: such a sequence is skipped (its state and output rows
 *              are left as they were); the others are computed normally.
 *
 * N = 0 is a no-op returning GDN_OK.  GDN_EUNSUPPORTED unless D_k = D_v =
 * 128; GDN_EINVAL for T > 8 N (some sequence is then necessarily longer),
 * N * H_v > 2^30, a NULL state or cu_seqlens; other errors as
 * gdn_prefill_varlen.
 */
GDN_API int gdn_decode_multitoken(const void* q, const void* k, const void* v,
                       const float* g, const float* beta,
                       const int32_t* cu_seqlens,
                       float* state, void* o,
                       int N, int T, int H_qk, int H_v, int D_k, int D_v,
                       float scale,
                       void* workspace, size_t workspace_bytes,
                       void* stream);

/*
 * gdn_decode_ex -- gdn_decode and gdn_decode_indexed with an input prologue
 * fused into the kernel (paper: "Final Kernel Analysis", GDN prefill, where
 * the gate and beta preprocessing is a helper kernel of its own; here it is
 * part of the one launch).
 *
 *   state_idx  NULL: `state` is fp32 [B, H_v, D, D], one state per batch entry
 *              (gdn_decode; P is ignored).  Otherwise `state` is a pool of P
 *              slots and state_idx int32 [B] names each entry's slot
 *              (gdn_decode_indexed, same rules).
 *   flags      GDN_QK_L2NORM and/or GDN_GATE_LOGITS (see enum gdn_flags);
 *              0 gives gdn_decode / gdn_decode_indexed bit for bit.
 *
 * Other arguments and errors as gdn_decode / gdn_decode_indexed, plus
 * GDN_EINVAL for other flag bits.
 */
GDN_API int gdn_decode_ex(const void* q, const void* k, const void* v,
               const float* g, const float* beta,
               float* state, const int32_t* state_idx, int P, void* o,
               int B, int H_qk, int H_v, int D_k, int D_v,
               float scale, int flags, void* stream);

/*
 * gdn_prefill_varlen_ex -- gdn_prefill_varlen, gdn_prefill_varlen_indexed and
 * gdn_decode_multitoken with the input prologue of gdn_decode_ex fused into
 * the kernels.
 *
 *   state_idx  NULL: initial_state / final_state as gdn_prefill_varlen.
 *              Otherwise final_state is a pool of P slots updated in place
 *              (initial_state must be NULL or equal final_state) and
 *              state_idx int32 [N] names each sequence's slot
 *              (gdn_prefill_varlen_indexed, same rules).
 *   flags      GDN_QK_L2NORM, GDN_GATE_LOGITS, GDN_SHORT_ONLY (the
 *              gdn_decode_multitoken route: D = 128, T <= 8 N, the state
 *              updated in place, so initial_state must be NULL or equal
 *              final_state).  0 gives the plain entry points bit for bit.
 *              GDN_SHORT_ONLY with state_idx is a multi-token decode step on
 *              pooled states in one launch: sequence n (at most 8 tokens)
 *              advances slot state_idx[n]; results equal
 *              gdn_prefill_varlen_indexed bit for bit; a longer sequence is
 *              skipped and sets bit 1 of the fault word.
 *   workspace  gdn_prefill_workspace_size(N, T, H_v, D, D, chunk) bytes, as
 *              gdn_prefill_varlen (same fault word).
 *
 * Other arguments and errors as the corresponding entry point, plus
 * GDN_EINVAL for other flag bits.
 */
GDN_API int gdn_prefill_varlen_ex(const void* q, const void* k, const void* v,
                       const float* g, const float* beta,
                       const int32_t* cu_seqlens,
                       const float* initial_state, float* final_state,
                       const int32_t* state_idx, int P,
                       void* o,
                       int N, int T, int H_qk, int H_v, int D_k, int D_v,
                       int chunk, float scale, int flags,
                       void* workspace, size_t workspace_bytes,
                       void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GDN_MI355X_H */
