"""Mutation check of the pins: each planted mistake in the one-token update
(on the CPU, in a copy of the oracle's step) must make at least one pin fail,
so a slip of that kind in the oracle itself could not go unnoticed."""
import numpy as np
import pytest

import oracle.gdn_ref as ref
from oracle_pins import PINS


def _outer(a, b):
    return a[..., :, None] * b[..., None, :]


def _eye_like(k):
    return np.eye(k.shape[-1])


def m_drop_beta_in_erase(S, q, k, v, alpha, beta):
    S_new = S @ (alpha[..., None, None] * (_eye_like(k) - _outer(k, k))) + beta[..., None, None] * _outer(v, k)
    return S_new, (S_new @ q[..., None])[..., 0]


def m_drop_alpha(S, q, k, v, alpha, beta):
    return ref.step_matrix(S, q, k, v, np.ones_like(alpha), beta)


def m_alpha_on_write(S, q, k, v, alpha, beta):
    S_new = alpha[..., None, None] * (S @ (_eye_like(k) - beta[..., None, None] * _outer(k, k))
                                      + beta[..., None, None] * _outer(v, k))
    return S_new, (S_new @ q[..., None])[..., 0]


def m_left_multiply(S, q, k, v, alpha, beta):
    M = alpha[..., None, None] * (_eye_like(k) - beta[..., None, None] * _outer(k, k))
    S_new = M @ S + beta[..., None, None] * _outer(v, k)
    return S_new, (S_new @ q[..., None])[..., 0]


def m_output_from_old_state(S, q, k, v, alpha, beta):
    S_new, _ = ref.step_matrix(S, q, k, v, alpha, beta)
    return S_new, (S @ q[..., None])[..., 0]


def m_erase_sign(S, q, k, v, alpha, beta):
    M = alpha[..., None, None] * (_eye_like(k) + beta[..., None, None] * _outer(k, k))
    S_new = S @ M + beta[..., None, None] * _outer(v, k)
    return S_new, (S_new @ q[..., None])[..., 0]


def m_write_transposed(S, q, k, v, alpha, beta):
    M = alpha[..., None, None] * (_eye_like(k) - beta[..., None, None] * _outer(k, k))
    S_new = S @ M + beta[..., None, None] * _outer(k, v)
    return S_new, (S_new @ q[..., None])[..., 0]


def m_gate_inverted(S, q, k, v, alpha, beta):
    return ref.step_rank1(S, q, k, v, 1.0 / alpha, beta)


def m_query_in_erase(S, q, k, v, alpha, beta):
    Sq = np.einsum("...ij,...j->...i", S, q)
    u = beta[..., None] * (v - alpha[..., None] * Sq)
    S_new = alpha[..., None, None] * S + u[..., :, None] * k[..., None, :]
    return S_new, np.einsum("...ij,...j->...i", S_new, q)


def m_output_transposed_state(S, q, k, v, alpha, beta):
    S_new, _ = ref.step_rank1(S, q, k, v, alpha, beta)
    return S_new, np.einsum("...ji,...j->...i", S_new, q)


def m_beta_squared_write(S, q, k, v, alpha, beta):
    return ref.step_rank1(S, q, k, v * beta[..., None], alpha, beta)


MUTANTS = [m_drop_beta_in_erase, m_drop_alpha, m_alpha_on_write, m_left_multiply,
           m_output_from_old_state, m_erase_sign, m_write_transposed, m_gate_inverted,
           m_query_in_erase, m_output_transposed_state, m_beta_squared_write]


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m.__name__ for m in MUTANTS])
def test_some_pin_catches(mutant):
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mutant)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches {mutant.__name__}"


def test_gva_mapping_mistake_is_caught(monkeypatch):
    """A modulo head map (h_v % H_qk) instead of floor(h_v * H_qk / H_v)."""
    from oracle_pins import pin_gva
    monkeypatch.setattr(ref, "head_map", lambda H_qk, H_v: np.arange(H_v) % H_qk)
    with pytest.raises(AssertionError):
        pin_gva(ref.step_rank1)


def test_chunk_decay_sign_mistake_is_caught(monkeypatch):
    """The chunked form with the within-chunk decay taken as exp(gamma_i - gamma_r)."""
    from oracle_pins import pin_chunked
    real_exp = np.exp
    orig = ref.prefill_chunked

    def bad(*a, **kw):
        monkeypatch.setattr(ref.np, "exp", lambda x: real_exp(-x) if np.ndim(x) == 2 else real_exp(x))
        try:
            return orig(*a, **kw)
        finally:
            monkeypatch.setattr(ref.np, "exp", real_exp)

    monkeypatch.setattr(ref, "prefill_chunked", bad)
    with pytest.raises(AssertionError):
        pin_chunked(ref.step_rank1)
