"""Plain fp64 CPU oracle for the Gated DeltaNet recurrence.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it, to check and to time against the
HIP kernels.  It shares no code with them.

What it computes (paper: appendix "Operator Background and Mathematical
Definitions", subsection "Gated Delta Net"):

  the gated delta rule, per (sequence, value head), token by token,
      S_t = S_{t-1} ( alpha_t (I - beta_t k_t k_t^T) ) + beta_t v_t k_t^T,
      o_t = S_t q_t,
  with alpha_t = exp(g_t) for the natural-log gate g_t (the same subsection's
  remark on applying the log-domain gate), and the two execution regimes it
  names: decode (a prior state plus one update per sequence, state updated in
  place) and prefill (a whole packed sequence, returning every output and the
  final state).

Readings where the paper is silent:
  * S is d_v x d_k and stored [.., d_v, d_k] with the k index contiguous;
    o_t = S_t q_t uses the state *after* the update.
  * one gate g and one beta per (token, value head); beta is post-sigmoid.
  * value head h_v reads q/k head floor(h_v * H_qk / H_v) (consecutive value
    heads share a q/k head).
  * o is multiplied by ``scale`` (1.0 reproduces the literal equation).
  * q/k/v arrive as bf16 bit patterns (uint16) or fp32 and are upcast exactly;
    g, beta and states are fp32 upcast exactly; all arithmetic is fp64.

Functions:
  step_matrix     the literal matrix form of one update (D x D products).
  step_rank1      the same update regrouped as a rank-1 correction; used for
                  large inputs, and pinned to step_matrix by the tests.
  decode          one step for a batch of states.
  prefill_varlen  packed variable-length prefill, sequential in tokens.
  prefill_units   the same for a chosen subset of (sequence, head) units.
  prefill_chunked the chunked UT / WY form (an exact regrouping of the same
                  recurrence into chunk-local matrix products), in fp64.
  prefill_transfer brute force: final state and outputs as explicit sums of
                  products of per-token transition matrices (tiny inputs only).
  qk_l2norm_bf16  the optional q/k L2 normalisation of the fused prologue.
  gate_from_logits the optional gate/beta prologue: g = -softplus(a),
                  beta = sigmoid(b).
  prologue        both, selected by the same flag bits as the library's.

Readings for the prologue (the paper gives no formula: the gate helper it
profiles is a separate preprocessing kernel of the contest harness; the
workload descriptions fix these forms):
  * q, k rows x -> x / sqrt(sum x^2 + 1e-6), computed in fp32 from the bf16
    values (sum in index order, one rounding per term, correctly rounded
    square root and division) and rounded back to bf16 (nearest even).  The
    rounding decides bf16 codes, so it is taken in the kernel's precision
    (fp32), as the workloads normalise in fp32 and then round; everything
    after it is fp64.
  * g = -softplus(a) = log sigmoid(-a), beta = sigmoid(b), in fp64.
"""
from __future__ import annotations

from typing import Callable, Iterable, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "to_f64",
    "bf16_rne_bits",
    "qk_l2norm_bf16",
    "gate_from_logits",
    "prologue",
    "QK_L2NORM",
    "GATE_LOGITS",
    "head_map",
    "step_matrix",
    "step_rank1",
    "decode",
    "prefill_varlen",
    "prefill_units",
    "prefill_chunked",
    "prefill_transfer",
]


def to_f64(x: Optional[np.ndarray]) -> Optional[np.ndarray]:
    """Exact upcast to fp64.  uint16 arrays are bf16 bit patterns: a bf16 value
    is the fp32 value whose upper 16 bits are the pattern and lower 16 are zero."""
    if x is None:
        return None
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def bf16_rne_bits(x32: np.ndarray) -> np.ndarray:
    """fp32 values -> bf16 bit patterns (uint16), rounded to nearest, ties to
    even: add 0x7FFF plus the lowest kept bit, keep the upper 16 bits."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


QK_L2NORM = 1      # flag bits of the library's _ex entry points
GATE_LOGITS = 2


def qk_l2norm_bf16(x_bits: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """L2-normalise each row (last axis) of bf16 values x: y = bf16(x * r),
    r = 1 / sqrt(sum_i x_i^2 + eps), in fp32 with the sum taken in index order
    (the square of a bf16 value is exact in fp32, so each step rounds once).
    Returns bf16 bit patterns of the same shape."""
    x = (np.asarray(x_bits).astype(np.uint32) << np.uint32(16)).view(np.float32)
    acc = np.zeros(x.shape[:-1], np.float32)
    for i in range(x.shape[-1]):
        xi = x[..., i]
        acc = (acc + xi * xi).astype(np.float32)
    r = (np.float32(1.0) / np.sqrt((acc + np.float32(eps)).astype(np.float32))).astype(np.float32)
    return bf16_rne_bits((x * r[..., None]).astype(np.float32))


def gate_from_logits(a, b):
    """(g, beta) = (-softplus(a), sigmoid(b)) in fp64 from logits a, b."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    g = -(np.maximum(a, 0.0) + np.log1p(np.exp(-np.abs(a))))
    beta = 1.0 / (1.0 + np.exp(-b))
    return g, beta


def prologue(q, k, g, beta, flags: int):
    """The fused input prologue: q, k L2-normalised (bf16 bits out) with
    QK_L2NORM, g and beta from logits (fp64 out) with GATE_LOGITS; inputs are
    returned unchanged otherwise."""
    if flags & QK_L2NORM:
        q, k = qk_l2norm_bf16(q), qk_l2norm_bf16(k)
    if flags & GATE_LOGITS:
        g, beta = gate_from_logits(g, beta)
    return q, k, g, beta


def head_map(H_qk: int, H_v: int) -> np.ndarray:
    """q/k head read by each value head: floor(h_v * H_qk / H_v)."""
    if H_v % H_qk:
        raise ValueError("H_v must be a multiple of H_qk")
    return (np.arange(H_v) * H_qk) // H_v


def step_matrix(S, q, k, v, alpha, beta):
    """One gated-delta update in its literal matrix form.

    S [..., Dv, Dk]; q, k [..., Dk]; v [..., Dv]; alpha, beta [...].
    Returns (S_new, o) with S_new = S (alpha (I - beta k k^T)) + beta v k^T and
    o = S_new q (unscaled)."""
    Dk = k.shape[-1]
    eye = np.eye(Dk)
    kkT = k[..., :, None] * k[..., None, :]
    transition = alpha[..., None, None] * (eye - beta[..., None, None] * kkT)
    write = beta[..., None, None] * (v[..., :, None] * k[..., None, :])
    S_new = S @ transition + write
    o = (S_new @ q[..., :, None])[..., 0]
    return S_new, o


def step_rank1(S, q, k, v, alpha, beta):
    """The same update regrouped: u = beta (v - alpha S k); S_new = alpha S + u k^T.

    (Expand S alpha (I - beta k k^T) + beta v k^T = alpha S + beta (v - alpha S k) k^T.)"""
    Sk = np.einsum("...ij,...j->...i", S, k)
    u = beta[..., None] * (v - alpha[..., None] * Sk)
    S_new = alpha[..., None, None] * S + u[..., :, None] * k[..., None, :]
    o = np.einsum("...ij,...j->...i", S_new, q)
    return S_new, o


Step = Callable[..., Tuple[np.ndarray, np.ndarray]]


def decode(q, k, v, g, beta, state, scale: float = 1.0, step: Step = step_rank1):
    """One decode step for every (b, h_v): q, k [B, H_qk, Dk]; v [B, H_v, Dv];
    g, beta [B, H_v]; state [B, H_v, Dv, Dk].  Returns (o [B, H_v, Dv], new_state),
    both fp64; the caller's arrays are not modified."""
    q, k, v, g, beta, S = map(to_f64, (q, k, v, g, beta, state))
    hq = head_map(q.shape[1], v.shape[1])
    S_new, o = step(S, q[:, hq], k[:, hq], v, np.exp(g), beta)
    return scale * o, S_new


def _check_cu(cu_seqlens, T):
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    if cu[0] != 0 or cu[-1] != T or np.any(np.diff(cu) < 0):
        raise ValueError("cu_seqlens must start at 0, be non-decreasing and end at T")
    return cu


def prefill_varlen(q, k, v, g, beta, cu_seqlens, initial_state=None, scale: float = 1.0,
                   step: Step = step_rank1):
    """Packed varlen prefill, token by token.

    q, k [T, H_qk, Dk]; v [T, H_v, Dv]; g, beta [T, H_v]; cu_seqlens [N+1];
    initial_state [N, H_v, Dv, Dk] or None (zeros).
    Returns (o [T, H_v, Dv], final_state [N, H_v, Dv, Dk]) in fp64.  All heads of
    a sequence advance together (they are independent); sequences run one after
    the other, each from its own initial state."""
    q, k, v, g, beta = map(to_f64, (q, k, v, g, beta))
    T, H_qk, Dk = q.shape
    H_v, Dv = v.shape[1], v.shape[2]
    cu = _check_cu(cu_seqlens, T)
    N = len(cu) - 1
    hq = head_map(H_qk, H_v)
    o = np.zeros((T, H_v, Dv))
    final = np.zeros((N, H_v, Dv, Dk))
    for n in range(N):
        S = np.zeros((H_v, Dv, Dk)) if initial_state is None else to_f64(initial_state[n]).copy()
        for t in range(cu[n], cu[n + 1]):
            S, o_t = step(S, q[t, hq], k[t, hq], v[t], np.exp(g[t]), beta[t])
            o[t] = scale * o_t
        final[n] = S
    return o, final


def prefill_units(q, k, v, g, beta, cu_seqlens, units: Iterable[Tuple[int, int]],
                  initial_state=None, scale: float = 1.0, step: Step = step_rank1):
    """The prefill recurrence for selected (sequence n, value head h) units only.

    Units are independent, so this is exactly prefill_varlen restricted to them.
    Returns {(n, h): (o [len_n, Dv], final [Dv, Dk])} in fp64.  Only the rows
    of the chosen units are upcast, so it works on very large packed inputs."""
    T, H_qk, Dk = q.shape
    H_v, Dv = v.shape[1], v.shape[2]
    cu = _check_cu(cu_seqlens, T)
    hq = head_map(H_qk, H_v)
    out = {}
    by_seq = {}
    for n, h in units:
        by_seq.setdefault(int(n), []).append(int(h))
    for n, heads in by_seq.items():
        hs = np.array(heads)
        s, e = cu[n], cu[n + 1]
        qs, ks = to_f64(q[s:e][:, hq[hs]]), to_f64(k[s:e][:, hq[hs]])
        vs, gs, bs = to_f64(v[s:e][:, hs]), to_f64(g[s:e][:, hs]), to_f64(beta[s:e][:, hs])
        if initial_state is None:
            S = np.zeros((len(hs), Dv, Dk))
        else:
            S = to_f64(initial_state[n][hs]).copy()
        o = np.zeros((e - s, len(hs), Dv))
        for t in range(e - s):
            S, o_t = step(S, qs[t], ks[t], vs[t], np.exp(gs[t]), bs[t])
            o[t] = scale * o_t
        for j, h in enumerate(heads):
            out[(n, h)] = (o[:, j], S[j])
    return out


def prefill_chunked(q, k, v, g, beta, cu_seqlens, initial_state=None, scale: float = 1.0,
                    chunk: int = 64):
    """The chunked form of the same prefill, in fp64.

    Per (sequence, value head), chunks of ``chunk`` tokens start at the
    sequence's first token (the last chunk may be shorter).  With rows
    r = 1..L of one chunk, gamma_r the running sum of g inside the chunk and
    S0 the state entering it:
        A_ri = beta_r exp(gamma_r - gamma_i) (k_r . k_i)  for i < r, else 0
        (I + A) U = diag(beta) (V - diag(exp(gamma)) K S0^T)
        O = scale (diag(exp(gamma)) Q S0^T + (M * Q K^T) U),
            M_ri = exp(gamma_r - gamma_i) for i <= r, else 0
        S_next = exp(gamma_L) S0 + (diag(exp(gamma_L - gamma)) U)^T K.
    Unrolling the recurrence over the chunk gives S_r = exp(gamma_r) S0 +
    sum_{i<=r} exp(gamma_r - gamma_i) u_i k_i^T with u_r = beta_r (v_r -
    alpha_r S_{r-1} k_r); substituting S_{r-1} into u_r gives the triangular
    system above, so this equals the token-by-token form up to rounding.
    The triangular system is solved directly (no explicit inverse)."""
    q, k, v, g, beta = map(to_f64, (q, k, v, g, beta))
    T, H_qk, Dk = q.shape
    H_v, Dv = v.shape[1], v.shape[2]
    cu = _check_cu(cu_seqlens, T)
    N = len(cu) - 1
    hq = head_map(H_qk, H_v)
    o = np.zeros((T, H_v, Dv))
    final = np.zeros((N, H_v, Dv, Dk))
    for n in range(N):
        for h in range(H_v):
            S = np.zeros((Dv, Dk)) if initial_state is None else to_f64(initial_state[n, h]).copy()
            for s in range(cu[n], cu[n + 1], chunk):
                e = min(s + chunk, cu[n + 1])
                L = e - s
                Q, K, V = q[s:e, hq[h]], k[s:e, hq[h]], v[s:e, h]
                b = beta[s:e, h]
                gam = np.cumsum(g[s:e, h])
                diff = gam[:, None] - gam[None, :]
                incl = np.tril(np.ones((L, L), dtype=bool))
                strict = np.tril(np.ones((L, L), dtype=bool), -1)
                M = np.where(incl, np.exp(np.where(incl, diff, 0.0)), 0.0)
                A = np.where(strict, b[:, None] * M * (K @ K.T), 0.0)
                rhs = b[:, None] * (V - np.exp(gam)[:, None] * (K @ S.T))
                U = np.linalg.solve(np.eye(L) + A, rhs)
                o[s:e, h] = scale * (np.exp(gam)[:, None] * (Q @ S.T) + (M * (Q @ K.T)) @ U)
                S = np.exp(gam[-1]) * S + (np.exp(gam[-1] - gam)[:, None] * U).T @ K
            final[n, h] = S
    return o, final


def prefill_transfer(q, k, v, g, beta, cu_seqlens, initial_state=None, scale: float = 1.0):
    """Brute force for tiny inputs: with the per-token transition
    M_t = alpha_t (I - beta_t k_t k_t^T) and write B_t = beta_t v_t k_t^T,
        S_t = S_0 M_1 ... M_t + sum_{j<=t} B_j M_{j+1} ... M_t,
    each product formed explicitly for every t (O(T^2) matrix products)."""
    q, k, v, g, beta = map(to_f64, (q, k, v, g, beta))
    T, H_qk, Dk = q.shape
    H_v, Dv = v.shape[1], v.shape[2]
    cu = _check_cu(cu_seqlens, T)
    N = len(cu) - 1
    hq = head_map(H_qk, H_v)
    eye = np.eye(Dk)
    o = np.zeros((T, H_v, Dv))
    final = np.zeros((N, H_v, Dv, Dk))
    for n in range(N):
        s0, e0 = cu[n], cu[n + 1]
        for h in range(H_v):
            S0 = np.zeros((Dv, Dk)) if initial_state is None else to_f64(initial_state[n, h])
            Ms = [np.exp(g[t, h]) * (eye - beta[t, h] * np.outer(k[t, hq[h]], k[t, hq[h]]))
                  for t in range(s0, e0)]
            Bs = [beta[t, h] * np.outer(v[t, h], k[t, hq[h]]) for t in range(s0, e0)]
            St = S0
            for t in range(e0 - s0):
                prod = eye
                for j in range(t + 1):
                    prod = prod @ Ms[j]
                St = S0 @ prod
                for j in range(t + 1):
                    tail = eye
                    for m in range(j + 1, t + 1):
                        tail = tail @ Ms[m]
                    St = St + Bs[j] @ tail
                o[s0 + t, h] = scale * (St @ q[s0 + t, hq[h]])
            final[n, h] = St
    return o, final
