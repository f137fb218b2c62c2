"""The fp64 oracle against its pins (CPU only)."""
import numpy as np
import pytest

import oracle.gdn_ref as ref
from oracle_pins import PINS, rand_case, _close
from paper_2607_17979_amd import workloads


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
@pytest.mark.parametrize("step", [ref.step_matrix, ref.step_rank1], ids=["matrix", "rank1"])
def test_pin(pin, step):
    pin(step)


def test_matrix_and_rank1_forms_agree():
    c = rand_case(31, [9, 4], H_qk=2, H_v=4, D=16, Dv=8)
    o1, f1 = ref.prefill_varlen(**c, scale=0.7, step=ref.step_matrix)
    o2, f2 = ref.prefill_varlen(**c, scale=0.7, step=ref.step_rank1)
    _close(o1, o2, tol=1e-12, what="outputs")
    _close(f1, f2, tol=1e-12, what="states")


def test_chunked_matches_sequential_at_head_dim_128():
    """The chunk-64 form at the production head size, two ragged sequences."""
    inp = workloads.prefill_inputs(41, [150, 70], H_qk=1, H_v=2, D=128, state_std=0.02)
    args = (inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens, inp.initial_state)
    o1, f1 = ref.prefill_varlen(*args)
    o2, f2 = ref.prefill_chunked(*args, chunk=64)
    _close(o1, o2, tol=1e-10, what="outputs")
    _close(f1, f2, tol=1e-10, what="states")


def test_tiny_workload_fp32_sequential_vs_chunk16():
    """The tiny workload on its fp32 draws: sequential decode calls, sequential
    prefill and chunk-16 prefill agree to 1e-12."""
    w = workloads.WORKLOADS["tiny"]
    inp = workloads.prefill_inputs(w["seed"], [w["T"]], w["H_qk"], w["H_v"], w["D"], qkv_dtype="f32")
    args = (inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens, None)
    o_seq, f_seq = ref.prefill_varlen(*args)
    o_chk, f_chk = ref.prefill_chunked(*args, chunk=16)
    _close(o_seq, o_chk, tol=1e-12, what="chunk-16 outputs")
    _close(f_seq, f_chk, tol=1e-12, what="chunk-16 states")
    S = np.zeros((1, w["H_v"], w["D"], w["D"]))
    for t in range(w["T"]):
        o_t, S = ref.decode(inp.q[t:t + 1], inp.k[t:t + 1], inp.v[t:t + 1], inp.g[t:t + 1],
                            inp.beta[t:t + 1], S)
        _close(o_t[0], o_seq[t], tol=1e-12, what="decode outputs")
    _close(S[0], f_seq[0], tol=1e-12, what="decode state")


def test_prefill_units_matches_full():
    inp = workloads.prefill_inputs(42, [20, 0, 33], H_qk=2, H_v=4, D=16, state_std=0.02)
    args = (inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens)
    o, fin = ref.prefill_varlen(*args, inp.initial_state, scale=0.5)
    units = [(0, 3), (2, 0), (2, 1), (1, 2)]
    got = ref.prefill_units(*args, units, inp.initial_state, scale=0.5)
    cu = inp.cu_seqlens
    for (n, h) in units:
        ou, fu = got[(n, h)]
        np.testing.assert_array_equal(ou, o[cu[n]:cu[n + 1], h])
        np.testing.assert_array_equal(fu, fin[n, h])


def test_bf16_upcast_is_exact():
    x = np.array([1.0, -2.5, 3.140625, 1e-30, 65504.0, -0.0], np.float32)
    bits = workloads.bf16_bits(x)
    back = ref.to_f64(bits)
    # every value above is exactly representable in bf16 except pi's tail
    np.testing.assert_array_equal(back[[0, 1, 2, 5]], x[[0, 1, 2, 5]].astype(np.float64))
    # round to nearest even: 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7
    assert ref.to_f64(workloads.bf16_bits(np.array([1.0 + 2.0 ** -8], np.float32)))[0] == 1.0
    assert ref.to_f64(workloads.bf16_bits(np.array([1.0 + 3 * 2.0 ** -8], np.float32)))[0] == 1.0 + 2.0 ** -6


def test_head_map():
    np.testing.assert_array_equal(ref.head_map(16, 32), np.repeat(np.arange(16), 2))
    np.testing.assert_array_equal(ref.head_map(2, 2), [0, 1])
    with pytest.raises(ValueError):
        ref.head_map(3, 4)


def test_bad_cu_seqlens_rejected():
    c = rand_case(43, [3, 2])
    with pytest.raises(ValueError):
        ref.prefill_varlen(**dict(c, cu_seqlens=np.array([0, 4, 3])))
    with pytest.raises(ValueError):
        ref.prefill_varlen(**dict(c, cu_seqlens=np.array([0, 3, 6])))
