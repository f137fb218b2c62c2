"""The fused input prologue on the GPU (gdn_decode_ex, gdn_prefill_varlen_ex):
q/k L2 normalisation and gate/beta logits computed in the kernels, against
the oracle's prologue followed by the recurrence.  With the normalisation
alone the kernels' normalised codes are the oracle's bit for bit (both take
the rounding in fp32 with the same summation order), so the fused call must
equal the plain entry point on the oracle-normalised inputs bit for bit."""
import numpy as np
import pytest

import oracle.gdn_ref as ref
from gpu_helpers import bf16_np, check_outputs, check_states, device, note, to_dev
from paper_2607_17979_amd import gdn
from paper_2607_17979_amd import workloads as wl

pytestmark = pytest.mark.gpu

NORM, LOGITS, SHORT = gdn.GDN_QK_L2NORM, gdn.GDN_GATE_LOGITS, gdn.GDN_SHORT_ONLY


def _dec_dev(inp, dev):
    return [to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v)] + [to_dev(inp.g, dev), to_dev(inp.beta, dev)]


@pytest.mark.parametrize("flags", [NORM, LOGITS, NORM | LOGITS])
@pytest.mark.parametrize("seed", [60, 61, 62])
def test_decode_prologue_matches_oracle(flags, seed):
    import torch

    dev = device()
    inp = wl.decode_inputs(seed, 64, 16, 32, 128, raw=3.0)
    if not flags & LOGITS:  # post-transform gates, raw q/k
        inp.g = -np.log1p(np.exp(inp.g)).astype(np.float32)
        inp.beta = (1 / (1 + np.exp(-inp.beta))).astype(np.float32)
    if not flags & NORM:
        inp.q, inp.k = ref.qk_l2norm_bf16(inp.q), ref.qk_l2norm_bf16(inp.k)
    note(f"decode prologue flags={flags} seed={seed}")
    q, k, v, g, b = _dec_dev(inp, dev)
    state = to_dev(inp.state, dev)
    o = torch.empty(v.shape, dtype=torch.bfloat16, device=dev)
    gdn.gdn_decode_ex(q, k, v, g, b, state, o, flags=flags)
    torch.cuda.synchronize()
    pq, pk, pg, pb = ref.prologue(inp.q, inp.k, inp.g, inp.beta, flags)
    o_ref, s_ref = ref.decode(pq, pk, inp.v, pg, pb, inp.state)
    check_outputs(bf16_np(o), o_ref, f"decode prologue {flags}")
    check_states(state.cpu().numpy(), s_ref, f"decode prologue {flags}")


def test_decode_norm_equals_plain_on_normalised_inputs_bitwise():
    import torch

    dev = device()
    inp = wl.decode_inputs(63, 16, 4, 8, 128, raw=5.0)
    inp.g = -np.log1p(np.exp(inp.g)).astype(np.float32)
    inp.beta = (1 / (1 + np.exp(-inp.beta))).astype(np.float32)
    q, k, v, g, b = _dec_dev(inp, dev)
    s1, s2 = to_dev(inp.state, dev), to_dev(inp.state, dev)
    o1, o2 = (torch.empty(v.shape, dtype=torch.bfloat16, device=dev) for _ in range(2))
    gdn.gdn_decode_ex(q, k, v, g, b, s1, o1, flags=NORM)
    qn, kn = (to_dev(ref.qk_l2norm_bf16(x), dev, bf16=True) for x in (inp.q, inp.k))
    gdn.gdn_decode(qn, kn, v, g, b, s2, o2)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(s1, s2)


def test_ex_without_flags_equals_plain_entry_points_bitwise():
    import torch

    dev = device()
    inp = wl.decode_inputs(64, 8, 2, 4, 128)
    q, k, v, g, b = _dec_dev(inp, dev)
    s1, s2 = to_dev(inp.state, dev), to_dev(inp.state, dev)
    o1, o2 = (torch.empty(v.shape, dtype=torch.bfloat16, device=dev) for _ in range(2))
    gdn.gdn_decode_ex(q, k, v, g, b, s1, o1)
    gdn.gdn_decode(q, k, v, g, b, s2, o2)
    p = wl.prefill_inputs(65, [70, 3, 0, 130], 2, 4, 128, state_std=0.02)
    pq, pk, pv = (to_dev(x, dev, bf16=True) for x in (p.q, p.k, p.v))
    pg, pb, cu, init = to_dev(p.g, dev), to_dev(p.beta, dev), to_dev(p.cu_seqlens, dev), to_dev(p.initial_state, dev)
    f1, f2 = torch.empty_like(init), torch.empty_like(init)
    po1, po2 = (torch.empty((p.q.shape[0], 4, 128), dtype=torch.bfloat16, device=dev) for _ in range(2))
    gdn.gdn_prefill_varlen_ex(pq, pk, pv, pg, pb, cu, init, f1, po1)
    gdn.gdn_prefill_varlen(pq, pk, pv, pg, pb, cu, init, f2, po2)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(s1, s2)
    assert torch.equal(po1.view(torch.int16), po2.view(torch.int16)) and torch.equal(f1, f2)


def _prefill_case(inp, dev, flags, idx=None, pool=None, in_place=False):
    import torch

    N, T, H_qk, H_v, D = inp.shape
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    o = torch.full((T, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)
    if idx is not None:
        st = to_dev(pool, dev)
        ws = gdn.gdn_prefill_varlen_ex(q, k, v, g, b, cu, None, st, o, state_idx=to_dev(idx, dev), flags=flags,
                                       scale=inp.scale)
        fin = st
    else:
        init = to_dev(inp.initial_state, dev)
        fin = init if in_place else torch.full((N, H_v, D, D), float("nan"), dtype=torch.float32, device=dev)
        ws = gdn.gdn_prefill_varlen_ex(q, k, v, g, b, cu, init, fin, o, flags=flags, scale=inp.scale)
    assert gdn.workspace_fault(ws, N) == 0
    return o, fin


def _oracle(inp, flags, init=None):
    pq, pk, pg, pb = ref.prologue(inp.q, inp.k, inp.g, inp.beta, flags)
    return ref.prefill_varlen(pq, pk, inp.v, pg, pb, inp.cu_seqlens,
                              inp.initial_state if init is None else init, scale=inp.scale)


@pytest.mark.parametrize("D", [128, 16])
@pytest.mark.parametrize("flags", [NORM, LOGITS, NORM | LOGITS])
def test_prefill_prologue_matches_oracle(D, flags):
    """Both routes (short sequences token by token, longer ones in chunks) and
    both head dims, raw q/k of norm about 3 sqrt(D) and gate/beta logits."""
    dev = device()
    C = 64 if D == 128 else 16
    lengths = [0, 1, 5, C - 1, C + 1, 3 * C + 7, 8, 200]
    note(f"prefill prologue D={D} flags={flags} lengths={lengths}")
    inp = wl.prefill_inputs(66 + flags, lengths, 2, 4, D, state_std=0.02, scale=D ** -0.5, raw=3.0)
    if not flags & LOGITS:
        inp.g = -np.log1p(np.exp(inp.g)).astype(np.float32)
        inp.beta = (1 / (1 + np.exp(-inp.beta))).astype(np.float32)
    if not flags & NORM:
        inp.q, inp.k = ref.qk_l2norm_bf16(inp.q), ref.qk_l2norm_bf16(inp.k)
    o, fin = _prefill_case(inp, dev, flags)
    o_ref, s_ref = _oracle(inp, flags)
    check_outputs(bf16_np(o), o_ref, f"prefill prologue D={D} flags={flags}")
    check_states(fin.cpu().numpy(), s_ref, f"prefill prologue D={D} flags={flags}")


# (sequences, value heads) for each launch shape of the chunk kernel on 256 CUs
SHAPES = [(9, 32), (3, 32), (2, 32)]


@pytest.mark.parametrize("shape", SHAPES, ids=["one workgroup per head", "two per head", "four per head"])
def test_prefill_norm_equals_plain_on_normalised_inputs_bitwise(shape):
    """Each chunk-kernel launch shape with the fused normalisation equals the
    plain call on the oracle-normalised inputs bit for bit (the producers'
    operand fragments, the staged rows and the first chunk's staging all use
    the same normalised codes)."""
    import torch

    N, H_v = shape
    dev = device()
    lengths = list(np.random.default_rng(N).integers(70, 400, size=N))
    inp = wl.prefill_inputs(70 + N, lengths, H_v // 2, H_v, 128, state_std=0.02, raw=4.0)
    inp.g = -np.log1p(np.exp(inp.g)).astype(np.float32)
    inp.beta = (1 / (1 + np.exp(-inp.beta))).astype(np.float32)
    o1, f1 = _prefill_case(inp, dev, NORM)
    nrm = wl.PrefillInputs(ref.qk_l2norm_bf16(inp.q), ref.qk_l2norm_bf16(inp.k), inp.v, inp.g, inp.beta,
                           inp.cu_seqlens, inp.initial_state, inp.scale)
    o2, f2 = _prefill_case(nrm, dev, 0)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(f1.view(torch.int32), f2.view(torch.int32))


def test_multitoken_and_pool_with_prologue():
    """The multi-token decode route (GDN_SHORT_ONLY, in place) and a pool of
    slots, each with both prologue flags, against the oracle."""
    dev = device()
    flags = NORM | LOGITS
    lengths = [4, 0, 8, 2, 7]
    inp = wl.prefill_inputs(80, lengths, 16, 32, 128, state_std=0.02, raw=2.0)
    o, fin = _prefill_case(inp, dev, flags | SHORT, in_place=True)
    o_ref, s_ref = _oracle(inp, flags)
    check_outputs(bf16_np(o), o_ref, "multi-token prologue")
    check_states(fin.cpu().numpy(), s_ref, "multi-token prologue")
    # pool: sequences take slots 5, 0, -1 (skipped), 2, 7 of 8
    idx = np.array([5, 0, -1, 2, 7], np.int32)
    pool = (0.02 * np.random.default_rng(81).standard_normal((8, 32, 128, 128))).astype(np.float32)
    inp2 = wl.prefill_inputs(82, [9, 70, 3, 130, 1], 16, 32, 128, raw=2.0)
    o2, pool_out = _prefill_case(inp2, dev, flags, idx=idx, pool=pool)
    init = np.stack([pool[s] if s >= 0 else np.zeros_like(pool[0]) for s in idx])
    o_ref2, s_ref2 = _oracle(inp2, flags, init=init)
    ok = idx >= 0
    cu = inp2.cu_seqlens
    keep = np.concatenate([np.arange(cu[n], cu[n + 1]) for n in range(len(idx)) if ok[n]])
    check_outputs(bf16_np(o2)[keep], o_ref2[keep], "pool prologue")
    check_states(pool_out.cpu().numpy()[idx[ok]], s_ref2[ok], "pool prologue")


def test_multitoken_on_a_pool():
    """A multi-token decode step on pooled states in one call:
    gdn_prefill_varlen_ex with GDN_SHORT_ONLY and state_idx (the token-by-token
    launch alone).  Slots and outputs equal gdn_prefill_varlen_indexed on the
    same pool bit for bit (for at most 8 tokens both take the token-by-token
    route) and match the oracle; slots not named and the output rows of
    skipped entries (-1, past the pool) stay untouched.  A second call with a
    9-token sequence skips it, leaves its slot and rows untouched and sets
    bit 1 of the fault word."""
    import torch

    dev = device()
    P, H_qk, H_v, D = 12, 16, 32, 128
    lengths = [4, 0, 8, 2, 7, 3]
    idx = np.array([5, 0, -1, 2, 11, 13], np.int32)
    note(f"multi-token decode on a pool: lengths {lengths}, slots {idx.tolist()} of {P}")
    inp = wl.prefill_inputs(85, lengths, H_qk, H_v, D, scale=D ** -0.5)
    pool = (0.02 * np.random.default_rng(86).standard_normal((P, H_v, D, D))).astype(np.float32)
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    sidx = to_dev(idx, dev)
    T = int(inp.cu_seqlens[-1])

    def out():
        return torch.full((T, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)

    pool_a, o_a = to_dev(pool, dev), out()
    ws = gdn.gdn_prefill_varlen_ex(q, k, v, g, b, cu, None, pool_a, o_a, state_idx=sidx, flags=SHORT,
                                   scale=inp.scale)
    assert gdn.workspace_fault(ws, len(lengths)) == 0
    pool_b, o_b = to_dev(pool, dev), out()
    ws = gdn.gdn_prefill_varlen_indexed(q, k, v, g, b, cu, pool_b, sidx, o_b, scale=inp.scale)
    assert gdn.workspace_fault(ws, len(lengths)) == 0
    torch.cuda.synchronize()
    assert torch.equal(pool_a.view(torch.int32), pool_b.view(torch.int32))
    assert torch.equal(o_a.view(torch.int16), o_b.view(torch.int16))
    ok = (idx >= 0) & (idx < P)
    untouched = sorted(set(range(P)) - set(idx[ok].tolist()))
    assert np.array_equal(pool_a.cpu().numpy()[untouched], pool[untouched])
    cu_h = inp.cu_seqlens
    skipped = np.concatenate([np.arange(cu_h[n], cu_h[n + 1]) for n in range(len(idx)) if not ok[n]])
    assert bool(torch.isnan(o_a.float()[skipped]).all())
    init = np.stack([pool[s] if ok[n] else np.zeros_like(pool[0]) for n, s in enumerate(idx)])
    o_ref, s_ref = ref.prefill_varlen(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens, init,
                                      scale=inp.scale)
    keep = np.concatenate([np.arange(cu_h[n], cu_h[n + 1]) for n in range(len(idx)) if ok[n]])
    check_outputs(bf16_np(o_a)[keep], o_ref[keep], "multi-token pool")
    check_states(pool_a.cpu().numpy()[idx[ok]], s_ref[ok], "multi-token pool")
    # a sequence longer than 8 tokens is skipped and flagged
    inp9 = wl.prefill_inputs(87, [3, 9, 1], H_qk, H_v, D, scale=D ** -0.5)
    idx9 = to_dev(np.array([1, 4, 7], np.int32), dev)
    q9, k9, v9 = (to_dev(x, dev, bf16=True) for x in (inp9.q, inp9.k, inp9.v))
    g9, b9, cu9 = to_dev(inp9.g, dev), to_dev(inp9.beta, dev), to_dev(inp9.cu_seqlens, dev)
    pool_c = to_dev(pool, dev)
    o_c = torch.full((13, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)
    ws = gdn.gdn_prefill_varlen_ex(q9, k9, v9, g9, b9, cu9, None, pool_c, o_c, state_idx=idx9, flags=SHORT,
                                   scale=inp9.scale)
    assert gdn.workspace_fault(ws, 3) == 2
    pc = pool_c.cpu().numpy()
    assert np.array_equal(pc[4], pool[4]) and not np.array_equal(pc[1], pool[1])
    assert bool(torch.isnan(o_c.float()[3:12]).all()) and not bool(torch.isnan(o_c.float()[:3]).any())
