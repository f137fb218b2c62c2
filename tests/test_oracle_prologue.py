"""Pins of the oracle's input prologue (the fused q/k L2 normalisation and the
gate/beta logits), each against something other than the formula itself:
exact invariances, closed forms and an independent computation."""
import math

import numpy as np
import pytest

import oracle.gdn_ref as ref
from paper_2607_17979_amd import workloads as wl


def _f64(bits):
    return ref.to_f64(bits)


def _raw_rows(seed, n=64, d=128, std=3.0):
    rng = np.random.default_rng(seed)
    return wl.bf16_bits((std * rng.standard_normal((n, d))).astype(np.float32))


def test_bf16_rounding_matches_an_independent_rounding():
    """The oracle's bf16 rounding against rounding done with fp64 arithmetic:
    the nearest bf16 value, ties to the even code."""
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(5000).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, 2 ** -130], np.float32)])
    got = _f64(ref.bf16_rne_bits(x))
    for xv, gv in zip(x.astype(np.float64), got):
        if xv == 0.0:
            assert gv == 0.0
            continue
        e = math.floor(math.log2(abs(xv)))
        ulp = 2.0 ** (max(e, -126) - 7)
        lo = math.floor(xv / ulp) * ulp
        cands = [lo, lo + ulp]
        best = min(cands, key=lambda c: (abs(c - xv), (round(c / ulp) % 2)))
        assert gv == best, (xv, gv, best)


def test_l2norm_is_exactly_scale_invariant():
    """Scaling a bf16 row by a power of two is exact and scales the fp32 sum of
    squares exactly, so the normalised codes must not change at all."""
    x = _raw_rows(1)
    y = ref.qk_l2norm_bf16(x)
    for j in (-3, 1, 4):
        xs = wl.bf16_bits((_f64(x) * 2.0 ** j).astype(np.float32))
        assert np.array_equal(_f64(xs), _f64(x) * 2.0 ** j)
        # the eps term breaks exact invariance only below |x|^2 ~ 1e-6, far from these rows
        assert np.array_equal(ref.qk_l2norm_bf16(xs), y), j


def test_l2norm_rows_have_unit_norm_within_bf16_rounding():
    y = _f64(ref.qk_l2norm_bf16(_raw_rows(2)))
    norms = np.linalg.norm(y, axis=-1)
    assert np.all(np.abs(norms - 1.0) <= 2.0 ** -8)


def test_l2norm_is_idempotent_to_one_code():
    """Normalising normalised rows changes each code by at most one unit in the
    last place (their norm is 1 up to the bf16 rounding)."""
    y = ref.qk_l2norm_bf16(_raw_rows(3))
    yy = ref.qk_l2norm_bf16(y)
    assert np.max(np.abs(yy.astype(np.int64) - y.astype(np.int64))) <= 1


def test_l2norm_closed_forms():
    """A row with one nonzero value c becomes sign(c) exactly (|c| >= 1/64);
    the zero row stays zero; a row of n equal values c becomes 1/sqrt(n)."""
    x = np.zeros((3, 128), np.float32)
    x[0, 17] = -5.25
    x[2, :] = 0.75
    y = _f64(ref.qk_l2norm_bf16(wl.bf16_bits(x)))
    assert y[0, 17] == -1.0 and np.count_nonzero(y[0]) == 1
    assert np.all(y[1] == 0.0)
    want = _f64(wl.bf16_bits(np.full(128, 1 / math.sqrt(128), np.float32)))
    assert np.array_equal(y[2], want)


def test_l2norm_against_an_fp64_normalisation():
    """Against the normalisation done in fp64 and rounded once: codes agree
    except where the fp64 value lies within fp32 rounding of a bf16 rounding
    boundary, and then differ by one code."""
    x = _raw_rows(4, n=256)
    y = ref.qk_l2norm_bf16(x)
    xf = _f64(x)
    z = xf / np.sqrt(np.sum(xf * xf, axis=-1, keepdims=True) + 1e-6)
    y64 = wl.bf16_bits(z.astype(np.float32))
    diff = np.abs(y.astype(np.int64) - y64.astype(np.int64))
    assert diff.max() <= 1
    assert np.count_nonzero(diff) <= 0.001 * diff.size


def test_gate_from_logits_closed_forms():
    a = np.array([0.0, 30.0, -30.0, 1.5, -1.5])
    g, beta = ref.gate_from_logits(a, a)
    assert g[0] == -math.log(2.0)
    assert abs(g[1] - (-30.0 - math.exp(-30.0))) < 1e-15
    assert abs(g[2] + math.exp(-30.0)) < 1e-20
    # alpha = exp(g) = sigmoid(-a), and sigmoid(b) + sigmoid(-b) = 1
    assert np.allclose(np.exp(g), 1.0 / (1.0 + np.exp(a)), rtol=1e-14, atol=0)
    assert beta[0] == 0.5
    assert abs(beta[3] + beta[4] - 1.0) < 1e-15
    assert np.all(g <= 0.0) and np.all((beta > 0) & (beta < 1))


def test_prologue_selects_by_flags_and_feeds_the_recurrence():
    """flags 0 leaves inputs unchanged; with both flags the recurrence on raw
    inputs equals the recurrence on the transformed inputs given directly."""
    inp = wl.prefill_inputs(5, [9, 4], 2, 4, 16, raw=2.0, state_std=0.1)
    same = ref.prologue(inp.q, inp.k, inp.g, inp.beta, 0)
    assert same[0] is inp.q and same[2] is inp.g
    q, k, g, b = ref.prologue(inp.q, inp.k, inp.g, inp.beta, ref.QK_L2NORM | ref.GATE_LOGITS)
    o1, s1 = ref.prefill_varlen(q, k, inp.v, g, b, inp.cu_seqlens, inp.initial_state)
    o2, s2 = ref.prefill_chunked(q, k, inp.v, g, b, inp.cu_seqlens, inp.initial_state, chunk=4)
    assert np.max(np.abs(o1 - o2)) < 1e-10 and np.max(np.abs(s1 - s2)) < 1e-10
    assert np.all(np.abs(np.linalg.norm(_f64(k), axis=-1) - 1.0) <= 2.0 ** -8)


@pytest.mark.parametrize("mutant", ["no_eps_sqrt", "wrong_axis", "softplus_sign", "beta_as_g"])
def test_prologue_mutants_fail_a_pin(mutant):
    """Plausible mistakes in the prologue each fail one of the pins above."""
    x = _raw_rows(6)
    a = np.array([0.0, 1.5, -1.5])
    if mutant == "no_eps_sqrt":       # normalise by the sum of squares, not its root
        xf = _f64(x)
        y = wl.bf16_bits((xf / (np.sum(xf * xf, -1, keepdims=True) + 1e-6)).astype(np.float32))
        assert not np.all(np.abs(np.linalg.norm(_f64(y), axis=-1) - 1.0) <= 2.0 ** -8)
    elif mutant == "wrong_axis":      # normalise columns instead of rows
        xf = _f64(x)
        y = wl.bf16_bits((xf / np.linalg.norm(xf, axis=0, keepdims=True)).astype(np.float32))
        assert not np.all(np.abs(np.linalg.norm(_f64(y), axis=-1) - 1.0) <= 2.0 ** -8)
    elif mutant == "softplus_sign":   # g = +softplus(a)
        g = np.maximum(a, 0.0) + np.log1p(np.exp(-np.abs(a)))
        assert not np.allclose(np.exp(g), 1.0 / (1.0 + np.exp(a)))
    else:                             # beta computed like g
        beta = -(np.maximum(a, 0.0) + np.log1p(np.exp(-np.abs(a))))
        assert beta[0] != 0.5
