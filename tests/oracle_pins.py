"""Pins for the fp64 oracle: checks against what the paper's equations and plain
mathematics fix, independent of the oracle's own code paths.

Each ``pin_*`` takes a one-token update ``step(S, q, k, v, alpha, beta) ->
(S_new, o)`` and raises AssertionError when the recurrence built from it
disagrees with a closed form, an invariant, a hand-worked example, brute force
or the chunked form.  The tests run every pin on both oracle step forms and,
in the mutation test, on deliberately wrong steps that every plausible slip
(dropped term, wrong sign, transposed operand, stale state) must trip.

Source of every expected value: the gated delta rule in the paper's appendix
"Operator Background and Mathematical Definitions", subsection "Gated Delta
Net", S_t = S_{t-1}(alpha_t (I - beta_t k_t k_t^T)) + beta_t v_t k_t^T,
o_t = S_t q_t, with alpha_t = exp(g_t).
"""
from __future__ import annotations

import json
import os

import numpy as np

import oracle.gdn_ref as ref

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TOL = 1e-11


def _close(a, b, tol=TOL, what=""):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    scale = max(1.0, float(np.max(np.abs(b))) if b.size else 1.0)
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= tol * scale, f"{what}: max |diff| {err:.3e} > {tol * scale:.3e}"


def rand_case(seed, lengths, H_qk=2, H_v=4, D=8, Dv=None, state=True, unit_keys=True):
    """Small fp64 inputs for the pins (seeded)."""
    rng = np.random.default_rng(seed)
    Dv = D if Dv is None else Dv
    T = int(sum(lengths))
    q = rng.standard_normal((T, H_qk, D))
    k = rng.standard_normal((T, H_qk, D))
    if unit_keys:
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((T, H_v, Dv))
    beta = 1.0 / (1.0 + np.exp(-rng.standard_normal((T, H_v))))
    g = -np.logaddexp(0.0, rng.standard_normal((T, H_v)))
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    S0 = 0.5 * rng.standard_normal((len(lengths), H_v, Dv, D)) if state else None
    return dict(q=q, k=k, v=v, g=g, beta=beta, cu_seqlens=cu, initial_state=S0)


def run(step, case, scale=1.0):
    c = case
    return ref.prefill_varlen(c["q"], c["k"], c["v"], c["g"], c["beta"], c["cu_seqlens"],
                              c["initial_state"], scale=scale, step=step)


# -- invariants and closed forms ------------------------------------------------

def pin_noop(step):
    """alpha = 1 (g = 0) and beta = 0 leave S unchanged, and o = scale S0 q."""
    c = rand_case(11, [5, 3])
    c["g"][:] = 0.0
    c["beta"][:] = 0.0
    o, fin = run(step, c, scale=0.75)
    assert np.array_equal(fin, c["initial_state"]), "state changed under alpha=1, beta=0"
    hq = ref.head_map(2, 4)
    for n, (s, e) in enumerate(zip(c["cu_seqlens"][:-1], c["cu_seqlens"][1:])):
        for t in range(s, e):
            want = 0.75 * np.einsum("hij,hj->hi", c["initial_state"][n], c["q"][t, hq])
            _close(o[t], want, what="noop output")


def pin_beta0_closed_form(step):
    """beta = 0: S_t = exp(gamma_t) S0 with gamma_t the running sum of g, o_t = S_t q_t."""
    c = rand_case(12, [7])
    c["beta"][:] = 0.0
    o, fin = run(step, c)
    gam = np.cumsum(c["g"], axis=0)  # [T, H_v]
    hq = ref.head_map(2, 4)
    S0 = c["initial_state"][0]
    for t in range(7):
        want = np.exp(gam[t])[:, None] * np.einsum("hij,hj->hi", S0, c["q"][t, hq])
        _close(o[t], want, what="beta=0 output")
    _close(fin[0], np.exp(gam[-1])[:, None, None] * S0, what="beta=0 state")


def pin_recall(step):
    """beta = 1 with a unit key: the updated state maps k_t to v_t exactly
    (S_t k_t = alpha S k - alpha S k (k.k) + v (k.k) = v), and with q_t = k_t the
    output is v_t.  Holds for any alpha and any prior state."""
    c = rand_case(13, [6], H_qk=4, H_v=4)
    c["beta"][:] = 1.0
    c["q"] = c["k"].copy()
    o, _ = run(step, c)
    _close(o, c["v"], tol=1e-10, what="recall o_t = v_t")
    # state after every prefix: S_t k_t = v_t
    for t in range(1, 7):
        cc = dict(c)
        for key in ("q", "k", "v", "g", "beta"):
            cc[key] = c[key][:t]
        cc["cu_seqlens"] = np.array([0, t])
        _, fin = run(step, cc)
        Sk = np.einsum("hij,hj->hi", fin[0], c["k"][t - 1])
        _close(Sk, c["v"][t - 1], tol=1e-10, what="recall S_t k_t = v_t")


def pin_orthonormal_keys(step):
    """Keys e_{p(t)} (distinct basis vectors): each step scales every column by
    alpha_t and, in column p(t), keeps (1 - beta_t) of it and adds beta_t v_t."""
    rng = np.random.default_rng(14)
    D, T = 8, 6
    c = rand_case(14, [T], H_qk=1, H_v=1, D=D)
    perm = rng.permutation(D)[:T]
    c["k"] = np.zeros((T, 1, D))
    c["k"][np.arange(T), 0, perm] = 1.0
    _, fin = run(step, c)
    alpha = np.exp(c["g"][:, 0])
    beta = c["beta"][:, 0]
    want = c["initial_state"][0, 0].copy()
    for t in range(T):
        j = perm[t]
        keyed = want[:, j].copy()
        want = alpha[t] * want
        want[:, j] = alpha[t] * (1.0 - beta[t]) * keyed + beta[t] * c["v"][t, 0]
    _close(fin[0, 0], want, what="orthonormal keys")


def pin_scalar_hand(step):
    """D = 1 by hand: S_t = alpha S (1 - beta k^2) + beta v k, o = S q.
    S0 = 2; (alpha, beta, k, v, q) = (1/2, 1/2, 1, 4, 3) gives S1 = 0.5 + 2 = 2.5,
    o1 = 7.5; then (1/4, 1, 2, 1, -1) gives S2 = 0.625 * (-3) + 2 = 0.125, o2 = -0.125."""
    S0 = np.array([[[2.0]]])
    q = np.array([[[3.0]], [[-1.0]]])
    k = np.array([[[1.0]], [[2.0]]])
    v = np.array([[[4.0]], [[1.0]]])
    g = np.log(np.array([[0.5], [0.25]]))
    beta = np.array([[0.5], [1.0]])
    o, fin = ref.prefill_varlen(q, k, v, g, beta, [0, 2], S0[None], step=step)
    _close(o[:, 0, 0], [7.5, -0.125], tol=1e-14, what="scalar outputs")
    _close(fin[0, 0], [[0.125]], tol=1e-14, what="scalar state")


def pin_hand_2x2(step):
    """Hand-worked 2 x 2 example stored in tests/golden/hand_2x2.json."""
    with open(os.path.join(GOLDEN, "hand_2x2.json")) as f:
        ex = json.load(f)
    S = np.array(ex["S0"], dtype=np.float64)[None]
    for st in ex["steps"]:
        S, o = step(S, np.array([st["q"]], np.float64), np.array([st["k"]], np.float64),
                    np.array([st["v"]], np.float64), np.array([st["alpha"]], np.float64),
                    np.array([st["beta"]], np.float64))
        _close(S[0], st["S"], tol=1e-14, what="hand 2x2 state")
        _close(o[0], st["o"], tol=1e-14, what="hand 2x2 output")


# -- independent routes to the same result ------------------------------------

def pin_transfer_brute_force(step):
    """Sequential recurrence = explicit sum of transition-matrix products."""
    c = rand_case(15, [4, 0, 3], H_qk=1, H_v=2, D=4)
    o1, f1 = run(step, c, scale=1.3)
    o2, f2 = ref.prefill_transfer(**c, scale=1.3)
    _close(o1, o2, what="transfer outputs")
    _close(f1, f2, what="transfer states")


def pin_chunked(step):
    """Sequential recurrence = chunked UT form, for several chunk sizes and a
    ragged tail; chunk 1 is the token-by-token limit."""
    c = rand_case(16, [13, 1, 9], H_qk=2, H_v=4, D=8)
    o1, f1 = run(step, c, scale=0.9)
    for C in (1, 2, 4, 5, 16):
        o2, f2 = ref.prefill_chunked(**c, scale=0.9, chunk=C)
        _close(o1, o2, tol=1e-10, what=f"chunk {C} outputs")
        _close(f1, f2, tol=1e-10, what=f"chunk {C} states")


# -- structural properties ----------------------------------------------------

def pin_varlen_independent(step):
    """A packed batch equals each sequence run alone (zero-length ones included)."""
    lengths = [3, 0, 5, 1]
    c = rand_case(17, lengths)
    o, fin = run(step, c)
    cu = c["cu_seqlens"]
    for n, L in enumerate(lengths):
        s, e = cu[n], cu[n + 1]
        single = dict(q=c["q"][s:e], k=c["k"][s:e], v=c["v"][s:e], g=c["g"][s:e],
                      beta=c["beta"][s:e], cu_seqlens=np.array([0, L]),
                      initial_state=c["initial_state"][n:n + 1])
        o1, f1 = run(step, single)
        _close(o[s:e], o1, what="varlen outputs")
        _close(fin[n], f1[0], what="varlen states")
    _close(fin[1], c["initial_state"][1], what="zero-length sequence keeps its state")


def pin_gva(step):
    """Value heads 2j and 2j+1 read q/k head j: repeating each q/k head twice and
    running with H_qk = H_v gives the same result."""
    c = rand_case(18, [6, 4], H_qk=2, H_v=4)
    o1, f1 = run(step, c)
    c2 = dict(c)
    c2["q"] = np.repeat(c["q"], 2, axis=1)
    c2["k"] = np.repeat(c["k"], 2, axis=1)
    o2, f2 = run(step, c2)
    _close(o1, o2, what="GVA outputs")
    _close(f1, f2, what="GVA states")


def pin_decode_prefill(step):
    """T decode steps equal a T-token prefill; a prefill continued from its own
    final state equals one prefill of the whole sequence."""
    c = rand_case(19, [7], H_qk=2, H_v=4)
    o, fin = run(step, c, scale=0.5)
    S = c["initial_state"].copy()
    for t in range(7):
        od, S = ref.decode(c["q"][t:t + 1], c["k"][t:t + 1], c["v"][t:t + 1], c["g"][t:t + 1],
                           c["beta"][t:t + 1], S, scale=0.5, step=step)
        _close(od[0], o[t], what="decode vs prefill output")
    _close(S, fin, what="decode vs prefill state")
    a = 3
    first = {key: c[key][:a] for key in ("q", "k", "v", "g", "beta")}
    rest = {key: c[key][a:] for key in ("q", "k", "v", "g", "beta")}
    oa, fa = run(step, dict(first, cu_seqlens=np.array([0, a]), initial_state=c["initial_state"]), 0.5)
    ob, fb = run(step, dict(rest, cu_seqlens=np.array([0, 7 - a]), initial_state=fa), 0.5)
    _close(np.concatenate([oa, ob]), o, what="continuation outputs")
    _close(fb, fin, what="continuation state")


def pin_value_permutation(step):
    """Permuting the value dimensions permutes o and the rows of S the same way."""
    c = rand_case(20, [6], H_qk=1, H_v=1, D=6)
    o, fin = run(step, c)
    p = np.random.default_rng(20).permutation(6)
    c2 = dict(c)
    c2["v"] = c["v"][:, :, p]
    c2["initial_state"] = c["initial_state"][:, :, p, :]
    o2, f2 = run(step, c2)
    _close(o2, o[:, :, p], what="permuted outputs")
    _close(f2, fin[:, :, p, :], what="permuted states")


def pin_linear_in_v(step):
    """From a zero state, outputs and final state are linear in V."""
    c = rand_case(21, [5, 4], state=False)
    v1 = c["v"]
    v2 = np.random.default_rng(21).standard_normal(v1.shape)
    oa, fa = run(step, dict(c, v=v1))
    ob, fb = run(step, dict(c, v=v2))
    oc, fc = run(step, dict(c, v=2.0 * v1 - 3.0 * v2))
    _close(oc, 2.0 * oa - 3.0 * ob, tol=1e-10, what="linear outputs")
    _close(fc, 2.0 * fa - 3.0 * fb, tol=1e-10, what="linear states")


def pin_scale(step):
    """scale multiplies o only."""
    c = rand_case(22, [4])
    o1, f1 = run(step, c, scale=1.0)
    o2, f2 = run(step, c, scale=0.125)
    _close(o2, 0.125 * o1, what="scaled outputs")
    assert np.array_equal(f1, f2), "scale changed the state"


PINS = [
    pin_noop,
    pin_beta0_closed_form,
    pin_recall,
    pin_orthonormal_keys,
    pin_scalar_hand,
    pin_hand_2x2,
    pin_transfer_brute_force,
    pin_chunked,
    pin_varlen_independent,
    pin_gva,
    pin_decode_prefill,
    pin_value_permutation,
    pin_linear_in_v,
    pin_scale,
]
