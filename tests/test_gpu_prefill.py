"""gdn_prefill_varlen on the GPU (through the C ABI) against the fp64 oracle."""
import numpy as np
import pytest

import oracle.gdn_ref as ref
from gpu_helpers import (bf16_np, check_outputs, check_states, device, note, record, rel_frob_units, to_dev)
from paper_2607_17979_amd import gdn
from paper_2607_17979_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _workspace(N, T, H_qk, H_v, D, dev):
    """A prefill workspace filled with 0xFF bytes, so that the wait-fault word
    reads 0 afterwards only if the call cleared it."""
    import torch

    need = gdn.gdn_prefill_workspace_size(N, T, H_v, D, D, gdn.default_chunk(D))
    return torch.full((max(need, 256),), 255, dtype=torch.uint8, device=dev)


def _assert_no_wait_fault(ws, N):
    """Word N + 1 of the workspace is set if a wave of the chunk kernel gave up
    one of its bounded waits (its results would then be invalid)."""
    import torch

    if N == 0:
        return  # a no-op call leaves the workspace alone
    torch.cuda.synchronize()
    assert int(ws.view(torch.int32)[N + 1].item()) == 0, "a chunk-kernel wait ran out of its bound"


def _prefill_gpu(inp, dev, scale=None, in_place=False, workspace=None):
    import torch

    N, T, H_qk, H_v, D = inp.shape
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b = to_dev(inp.g, dev), to_dev(inp.beta, dev)
    cu = to_dev(inp.cu_seqlens, dev)
    init = to_dev(inp.initial_state, dev)
    if in_place:
        assert init is not None
        fin = init
    else:
        fin = torch.full((N, H_v, D, D), float("nan"), dtype=torch.float32, device=dev)
    o = torch.full((T, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)
    if workspace is None:
        workspace = _workspace(N, T, H_qk, H_v, D, dev)
    gdn.gdn_prefill_varlen(q, k, v, g, b, cu, init, fin, o,
                           scale=inp.scale if scale is None else scale, workspace=workspace)
    _assert_no_wait_fault(workspace, N)
    return o, fin


def _full_oracle_check(inp, o, fin, what):
    o_ref, s_ref = ref.prefill_varlen(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens,
                                      inp.initial_state, scale=inp.scale)
    check_outputs(bf16_np(o), o_ref, what)
    check_states(fin.cpu().numpy(), s_ref, what)


def test_prefill_tiny_chunk16():
    """The tiny workload: one 64-token sequence, two heads, d = 16, chunk 16."""
    dev = device()
    w = wl.WORKLOADS["tiny"]
    note("prefill tiny d=16 chunk=16")
    inp = wl.prefill_inputs(w["seed"], [w["T"]], w["H_qk"], w["H_v"], w["D"])
    o, fin = _prefill_gpu(inp, dev)
    _full_oracle_check(inp, o, fin, "tiny")


@pytest.mark.parametrize("D", [16, 128])
@pytest.mark.parametrize("with_state", [False, True])
@pytest.mark.parametrize("seed", [30, 31, 32])
def test_prefill_ragged_small(D, with_state, seed):
    """Ragged lengths around the chunk size (empty, 1, C-1, C, C+1, several
    chunks) in one packed batch, GVA 2:1."""
    dev = device()
    C = 16 if D == 16 else 64
    lengths = [0, 1, C - 1, C, C + 1, 2 * C + 2, 3 * C + 7]
    note(f"prefill ragged D={D} state={with_state} seed={seed} lengths={lengths}")
    inp = wl.prefill_inputs(seed, lengths, 2, 4, D, state_std=0.02 if with_state else None,
                            scale=D ** -0.5)
    o, fin = _prefill_gpu(inp, dev)
    _full_oracle_check(inp, o, fin, f"ragged D={D}")


def _sampled_check(inp, o, fin, units, what):
    cu = inp.cu_seqlens
    got = ref.prefill_units(inp.q, inp.k, inp.v, inp.g, inp.beta, cu, units, inp.initial_state,
                            scale=inp.scale)
    o_bits = bf16_np(o)
    fin_np = fin.cpu().numpy()
    worst_o, worst_s = 0.0, 0.0
    for (n, h), (o_ref, s_ref) in got.items():
        out = ref.to_f64(o_bits[cu[n]:cu[n + 1], h])
        worst_o = max(worst_o, float(np.max(np.abs(out - o_ref))) if out.size else 0.0)
        worst_s = max(worst_s, float(rel_frob_units(fin_np[n, h], s_ref)))
    note(f"  {what}: {len(units)} units, outputs max-abs {worst_o:.3e}, "
         f"states worst rel-Frobenius {worst_s:.3e}")
    record("outputs max-abs", what, worst_o)
    record("states rel-F worst unit", what, worst_s)
    assert worst_o <= 2e-2
    assert worst_s <= 1e-3


@pytest.mark.parametrize("seed", [4, 14, 24])
def test_prefill_varlen16_parity(seed):
    """16 packed sequences, lengths uniform in [128, 2048], 32 value / 16 q/k
    heads, d = 128, chunk 64, zero initial state.  The oracle follows every
    head of four sequences and two heads of every other sequence."""
    dev = device()
    w = wl.WORKLOADS["prefill_varlen16"]
    lengths = wl.varlen_lengths(seed, w["N"], w["len_lo"], w["len_hi"])
    note(f"prefill varlen16 seed {seed} T={lengths.sum()}")
    inp = wl.prefill_inputs(seed, lengths, w["H_qk"], w["H_v"], w["D"])
    o, fin = _prefill_gpu(inp, dev)
    units = [(n, h) for n in range(4) for h in range(w["H_v"])]
    units += [(n, (7 * n + 3) % w["H_v"]) for n in range(4, w["N"])]
    units += [(n, (11 * n + 20) % w["H_v"]) for n in range(4, w["N"])]
    _sampled_check(inp, o, fin, units, "varlen16")


def test_prefill_long_2x64k():
    """Two 65,536-token sequences from a nonzero initial state; the oracle
    follows two value heads (one q/k pair and one unpaired) per sequence over
    all 65,536 tokens."""
    dev = device()
    w = wl.WORKLOADS["prefill_long2x64k"]
    note("prefill long 2 x 65536")
    inp = wl.prefill_inputs(w["seed"], [w["len"]] * w["N"], w["H_qk"], w["H_v"], w["D"],
                            state_std=w["state_std"])
    o, fin = _prefill_gpu(inp, dev)
    units = [(0, 0), (0, 1), (1, 17), (1, 30)]
    _sampled_check(inp, o, fin, units, "long 2x64k")


def test_prefill_maximum_size():
    """T * H_v = 2^24, the largest problem the entry point accepts (v and o are
    then 4 GiB, so byte offsets near their end need 32 bits): 8 sequences x
    65,536 tokens x 32 value heads, inputs drawn on the device by torch's
    seeded generator.  The oracle follows the first and the last (sequence,
    head) unit, the one at the highest addresses, over all their tokens; the
    fault word is clear."""
    import torch

    dev = device()
    N, L, H_qk, H_v, D = 8, 65536, 16, 32, 128
    T = N * L
    assert T * H_v == 1 << 24
    note(f"prefill maximum size: N={N} x {L} tokens, H_v={H_v} (T * H_v = 2^24)")
    x = wl.prefill_inputs_device(62, N, L, H_qk, H_v, D, 0.02, dev)
    fin = torch.empty_like(x["init"])
    o = torch.empty((T, H_v, D), dtype=torch.bfloat16, device=dev)
    ws = _workspace(N, T, H_qk, H_v, D, dev)
    gdn.gdn_prefill_varlen(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["init"], fin, o,
                           workspace=ws)
    _assert_no_wait_fault(ws, N)

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    for n, h in ((0, 0), (N - 1, H_v - 1)):
        rows = slice(n * L, (n + 1) * L)
        hq = h * H_qk // H_v
        note(f"  oracle on unit (sequence {n}, head {h}), {L} tokens")
        o_ref, s_ref = ref.prefill_varlen(
            bits(x["q"][rows, hq:hq + 1]), bits(x["k"][rows, hq:hq + 1]), bits(x["v"][rows, h:h + 1]),
            x["g"][rows, h:h + 1].cpu().numpy(), x["beta"][rows, h:h + 1].cpu().numpy(),
            np.array([0, L], np.int32), x["init"][n:n + 1, h:h + 1].cpu().numpy())
        check_outputs(bits(o[rows, h:h + 1]), o_ref, f"maximum size, unit ({n}, {h})")
        check_states(fin[n:n + 1, h:h + 1].cpu().numpy(), s_ref, f"maximum size, unit ({n}, {h})")


@pytest.mark.parametrize("L", [10, 4])
def test_prefill_states_beyond_4gib(L):
    """4,096 sequences x 32 value heads: 8 GiB of fp32 state in and out, so
    byte offsets into the states need more than 32 bits past the first half.
    L = 10: every sequence in the chunk kernel (separate final states); L = 4:
    every sequence token by token, states in place.  Inputs drawn on the
    device; the oracle checks the first unit and the one at the highest
    addresses; the fault word is clear."""
    import torch

    dev = device()
    N, H_qk, H_v, D = 4096, 16, 32, 128
    T = N * L
    note(f"prefill states beyond 4 GiB: N={N} x {L} tokens, H_v={H_v}")
    x = wl.prefill_inputs_device(72 + L, N, L, H_qk, H_v, D, 0.02, dev)
    units = ((0, 0), (N - 1, H_v - 1))
    before = {u: x["init"][u[0], u[1]].cpu().numpy() for u in units}
    in_place = L <= 8
    fin = x["init"] if in_place else torch.empty_like(x["init"])
    o = torch.empty((T, H_v, D), dtype=torch.bfloat16, device=dev)
    ws = _workspace(N, T, H_qk, H_v, D, dev)
    gdn.gdn_prefill_varlen(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["init"], fin, o,
                           workspace=ws)
    _assert_no_wait_fault(ws, N)

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    for n, h in units:
        rows = slice(n * L, (n + 1) * L)
        hq = h * H_qk // H_v
        o_ref, s_ref = ref.prefill_varlen(
            bits(x["q"][rows, hq:hq + 1]), bits(x["k"][rows, hq:hq + 1]), bits(x["v"][rows, h:h + 1]),
            x["g"][rows, h:h + 1].cpu().numpy(), x["beta"][rows, h:h + 1].cpu().numpy(),
            np.array([0, L], np.int32), before[(n, h)][None, None])
        check_outputs(bits(o[rows, h:h + 1]), o_ref, f"8 GiB states L={L}, unit ({n}, {h})")
        check_states(fin[n:n + 1, h:h + 1].cpu().numpy(), s_ref, f"8 GiB states L={L}, unit ({n}, {h})")


def test_prefill_identity_gate_bitwise_and_zero_length():
    """g = 0, beta = 0 leaves every state bit for bit; a zero-length sequence
    returns its initial state bit for bit."""
    dev = device()
    inp = wl.prefill_inputs(40, [70, 0, 5], 2, 4, 128, state_std=0.3)
    inp.g[:] = 0.0
    inp.beta[:] = 0.0
    o, fin = _prefill_gpu(inp, dev)
    assert np.array_equal(fin.cpu().numpy(), inp.initial_state)
    _full_oracle_check(inp, o, fin, "identity gate")


def test_prefill_in_place_and_deterministic():
    dev = device()
    inp = wl.prefill_inputs(41, [200, 64, 1], 2, 4, 128, state_std=0.02)
    o1, f1 = _prefill_gpu(inp, dev)
    o2, f2 = _prefill_gpu(inp, dev, in_place=True)
    import torch

    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(f1, f2)
    _full_oracle_check(inp, o1, f1, "in place")


def test_prefill_gva_equals_repeated_heads_bitwise():
    import torch

    dev = device()
    inp = wl.prefill_inputs(42, [150, 90], 2, 4, 128, state_std=0.02)
    o1, f1 = _prefill_gpu(inp, dev)
    rep = wl.PrefillInputs(np.repeat(inp.q, 2, axis=1), np.repeat(inp.k, 2, axis=1), inp.v, inp.g,
                           inp.beta, inp.cu_seqlens, inp.initial_state, inp.scale)
    o2, f2 = _prefill_gpu(rep, dev)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(f1, f2)


def test_prefill_schedule_is_longest_first():
    """The workspace holds the sequence order, longest first, ties by index,
    then the count of sequences run in chunks, then the cleared wait-fault
    word (integer work: compared exactly)."""
    import torch

    dev = device()
    lengths = [5, 130, 0, 130, 64, 1, 300, 5]
    inp = wl.prefill_inputs(43, lengths, 1, 2, 128)
    ws = torch.full((256,), 255, dtype=torch.uint8, device=dev)
    _prefill_gpu(inp, dev, workspace=ws)
    torch.cuda.synchronize()
    N = len(lengths)
    words = ws.view(torch.int32)[:N + 2].cpu().numpy()
    expect = sorted(range(N), key=lambda i: (-lengths[i], i))
    assert words[:N].tolist() == expect
    # then the number of sequences run in chunks (longer than 8 tokens)
    assert words[N] == sum(n > 8 for n in lengths)
    assert words[N + 1] == 0


def test_prefill_then_decode_continues_the_sequence():
    """Prefill of the first 100 tokens, then 5 decode steps on its final state,
    equals the oracle over all 105 tokens."""
    import torch

    dev = device()
    full = wl.prefill_inputs(44, [105], 2, 4, 128, state_std=0.02)
    head = wl.PrefillInputs(full.q[:100], full.k[:100], full.v[:100], full.g[:100],
                            full.beta[:100], np.array([0, 100], np.int32), full.initial_state)
    o_pre, fin = _prefill_gpu(head, dev)
    outs = [bf16_np(o_pre)]
    for t in range(100, 105):
        q, k, v = (to_dev(x[t:t + 1], dev, bf16=True) for x in (full.q, full.k, full.v))
        o = torch.empty(v.shape, dtype=torch.bfloat16, device=dev)
        gdn.gdn_decode(q, k, v, to_dev(full.g[t:t + 1], dev), to_dev(full.beta[t:t + 1], dev), fin, o)
        outs.append(bf16_np(o))
    torch.cuda.synchronize()
    o_ref, s_ref = ref.prefill_varlen(full.q, full.k, full.v, full.g, full.beta, full.cu_seqlens,
                                      full.initial_state)
    check_outputs(np.concatenate(outs), o_ref, "prefill+decode")
    check_states(fin.cpu().numpy(), s_ref, "prefill+decode")


def test_prefill_value_split_is_bitwise_batch_independent():
    """With few (sequence, head) items the kernel splits each head's value
    columns over 2 or 4 workgroups (1 x 32 heads: 4-way; 3 x 32: 2-way on
    256 compute units; 8 x 32: none).  Every value column evolves on its own,
    so one sequence gives bitwise the same outputs and final state in all
    three batches; the single-sequence run is also checked against the oracle."""
    import torch

    dev = device()
    L, H_qk, H_v, D = 200, 16, 32, 128
    base = wl.prefill_inputs(41, [L], H_qk, H_v, D, state_std=0.02, scale=D ** -0.5)
    o1, f1 = _prefill_gpu(base, dev)
    _full_oracle_check(base, o1, f1, "value split, 1 sequence")
    for copies in (3, 8):
        note(f"prefill value split: {copies} copies of one {L}-token sequence")
        rep = wl.PrefillInputs(
            q=np.concatenate([base.q] * copies), k=np.concatenate([base.k] * copies),
            v=np.concatenate([base.v] * copies), g=np.concatenate([base.g] * copies),
            beta=np.concatenate([base.beta] * copies),
            cu_seqlens=np.arange(copies + 1, dtype=np.int32) * L,
            initial_state=np.concatenate([base.initial_state] * copies), scale=base.scale)
        o, f = _prefill_gpu(rep, dev)
        for c in range(copies):
            assert torch.equal(o[c * L:(c + 1) * L].view(torch.int16), o1.view(torch.int16)), (copies, c)
            assert torch.equal(f[c].view(torch.int32), f1[0].view(torch.int32)), (copies, c)


def test_prefill_several_items_per_workgroup():
    """48 sequences x 32 value heads = 1,536 work items, more than the
    workgroups launched (one per compute unit), so each workgroup walks several
    items as one chunk stream: lengths from 0 to 260 (zero-length ones, single
    tokens, chunk boundaries 63/64/65) from a nonzero initial state.  The
    oracle follows two heads of every sequence; zero-length sequences keep
    their initial state bit for bit; three sequences run alone give bitwise
    the same outputs and states as inside the large batch."""
    import torch

    dev = device()
    rng = np.random.default_rng(77)
    lengths = rng.integers(0, 261, size=48)
    lengths[[3, 17, 30, 41]] = 0
    lengths[[5, 6, 7, 8]] = [1, 63, 64, 65]
    H_qk, H_v, D = 16, 32, 128
    note(f"prefill several items per workgroup: N=48, T={lengths.sum()}")
    inp = wl.prefill_inputs(78, lengths, H_qk, H_v, D, state_std=0.02, scale=D ** -0.5)
    o, fin = _prefill_gpu(inp, dev)
    units = [(n, h) for n in range(48) for h in ((7 * n) % H_v, (7 * n + 13) % H_v)]
    _sampled_check(inp, o, fin, units, "several items per workgroup")
    fin_np = fin.cpu().numpy()
    for n in np.nonzero(lengths == 0)[0]:
        assert np.array_equal(fin_np[n], inp.initial_state[n]), n
    cu = inp.cu_seqlens
    for n in (0, 7, int(np.argmax(lengths))):
        a, b = cu[n], cu[n + 1]
        one = wl.PrefillInputs(q=inp.q[a:b], k=inp.k[a:b], v=inp.v[a:b], g=inp.g[a:b], beta=inp.beta[a:b],
                               cu_seqlens=np.array([0, b - a], dtype=np.int32),
                               initial_state=inp.initial_state[n:n + 1], scale=inp.scale)
        o1, f1 = _prefill_gpu(one, dev)
        assert torch.equal(o[a:b].view(torch.int16), o1.view(torch.int16)), n
        assert torch.equal(fin[n].view(torch.int32), f1[0].view(torch.int32)), n


def test_prefill_short_sequences_token_by_token():
    """Sequences of at most 8 tokens run token by token (the chunk kernel skips
    them): lengths on both sides of that threshold, zero included, against the
    oracle; a zero-length sequence keeps its initial state bit for bit."""
    dev = device()
    lengths = [0, 1, 2, 7, 8, 9, 15, 16, 31, 64, 65, 8, 3]
    note(f"prefill short sequences {lengths}")
    inp = wl.prefill_inputs(45, lengths, 2, 4, 128, state_std=0.02)
    inp.scale = 128 ** -0.5
    o, fin = _prefill_gpu(inp, dev)
    _full_oracle_check(inp, o, fin, "short sequences")
    assert np.array_equal(fin.cpu().numpy()[0], inp.initial_state[0])


def test_prefill_short_route_zero_initial_state():
    """Only short sequences (T <= 8: the chunk kernel is not launched), no
    initial state."""
    dev = device()
    inp = wl.prefill_inputs(46, [3, 0, 5], 2, 4, 128)
    note("prefill short route, T = 8, zero initial state")
    o, fin = _prefill_gpu(inp, dev)
    _full_oracle_check(inp, o, fin, "short route, zero state")


@pytest.mark.parametrize("H_qk,H_v", [(4, 4), (2, 8)])
def test_short_route_head_ratios(H_qk, H_v):
    """The token-by-token walk groups the units that share a q/k head (the row
    blocks of H_v / H_qk value heads) on one XCD; with 1 and 4 value heads per
    q/k head (groups of 4 and 16 units, full and partial blocks of slots) every
    unit still runs once: outputs and states against the oracle, and bit for
    bit equal to the same call with q and k repeated per value head."""
    import torch

    dev = device()
    rng = np.random.default_rng(49 + H_v)
    lengths = [int(x) for x in rng.integers(0, 9, size=13)]
    note(f"short route H_qk={H_qk} H_v={H_v} lengths={lengths}")
    inp = wl.prefill_inputs(49 + H_v, lengths, H_qk, H_v, 128, state_std=0.02, scale=128 ** -0.5)
    o, fin = _prefill_gpu(inp, dev)
    _full_oracle_check(inp, o, fin, f"short route {H_qk}/{H_v}")
    r = H_v // H_qk
    rep = wl.PrefillInputs(np.repeat(inp.q, r, axis=1), np.repeat(inp.k, r, axis=1), inp.v, inp.g,
                           inp.beta, inp.cu_seqlens, inp.initial_state, inp.scale)
    o2, f2 = _prefill_gpu(rep, dev)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(fin, f2)


def test_multi_token_decode_equals_decode_steps_bitwise():
    """B sequences with Tn new tokens each and states updated in place (a
    multi-token decode step) equal Tn gdn_decode calls bit for bit: the
    token-by-token route applies the decode arithmetic per token.  Checked
    against the oracle as well."""
    import torch

    dev = device()
    B, Tn = 8, 4
    note(f"multi-token decode B={B} Tn={Tn}")
    inp = wl.prefill_inputs(47, [Tn] * B, 16, 32, 128, state_std=0.02)
    o1, f1 = _prefill_gpu(inp, dev, in_place=True)
    st = to_dev(inp.initial_state, dev)
    outs = []
    for t in range(Tn):
        idx = np.arange(B) * Tn + t
        q, k, v = (to_dev(x[idx], dev, bf16=True) for x in (inp.q, inp.k, inp.v))
        o = torch.empty(v.shape, dtype=torch.bfloat16, device=dev)
        gdn.gdn_decode(q, k, v, to_dev(inp.g[idx], dev), to_dev(inp.beta[idx], dev), st, o)
        outs.append(o)
    torch.cuda.synchronize()
    o_dec = torch.stack(outs, dim=1).reshape(B * Tn, 32, 128)
    assert torch.equal(o1.view(torch.int16), o_dec.view(torch.int16))
    assert torch.equal(f1, st)
    _full_oracle_check(inp, o1, f1, "multi-token decode")


def test_decode_multitoken_entry_point():
    """gdn_decode_multitoken (only the token-by-token launch) equals
    gdn_prefill_varlen in place bit for bit on 0..8-token sequences, with the
    fault word clear.  A batch that also holds a 9-token sequence: that
    sequence is skipped (its state and output rows untouched) and bit 1 of the
    fault word is set; every other sequence is computed as before."""
    import torch

    dev = device()
    lengths = [4, 0, 8, 1, 3, 8, 2, 5]
    H_qk, H_v, D = 16, 32, 128
    N, T = len(lengths), sum(lengths)
    note(f"multi-token entry point, lengths {lengths}")
    inp = wl.prefill_inputs(55, lengths, H_qk, H_v, D, state_std=0.02)
    o_ref, f_ref = _prefill_gpu(inp, dev, in_place=True)
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    st = to_dev(inp.initial_state, dev)
    o = torch.full((T, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)
    ws = _workspace(N, T, H_qk, H_v, D, dev)
    gdn.gdn_decode_multitoken(q, k, v, g, b, cu, st, o, workspace=ws)
    _assert_no_wait_fault(ws, N)
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(st.view(torch.int32), f_ref.view(torch.int32))

    # one sequence of 9 tokens: skipped and flagged
    lengths2 = [3, 9, 2, 6]
    N2, T2 = len(lengths2), sum(lengths2)
    inp2 = wl.prefill_inputs(56, lengths2, H_qk, H_v, D, state_std=0.02)
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp2.q, inp2.k, inp2.v))
    g, b, cu = to_dev(inp2.g, dev), to_dev(inp2.beta, dev), to_dev(inp2.cu_seqlens, dev)
    st = to_dev(inp2.initial_state, dev)
    o = torch.full((T2, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)
    ws = _workspace(N2, T2, H_qk, H_v, D, dev)
    gdn.gdn_decode_multitoken(q, k, v, g, b, cu, st, o, workspace=ws)
    torch.cuda.synchronize()
    assert int(ws.view(torch.int32)[N2 + 1].item()) == 2
    long_rows = slice(3, 12)
    assert torch.isnan(o[long_rows].float()).all()
    assert np.array_equal(st[1].cpu().numpy(), inp2.initial_state[1])
    o_ref2, s_ref2 = ref.prefill_varlen(inp2.q, inp2.k, inp2.v, inp2.g, inp2.beta, inp2.cu_seqlens,
                                        inp2.initial_state, scale=inp2.scale)
    keep = np.r_[0:3, 12:T2]
    check_outputs(bf16_np(o)[keep], o_ref2[keep], "multi-token entry, short sequences")
    check_states(st.cpu().numpy()[[0, 2, 3]], s_ref2[[0, 2, 3]], "multi-token entry, short sequences")


def test_prefill_many_short_sequences():
    """The short-sequence regime at the bench's head layout: 64 sequences of
    8 tokens, 32 value / 16 q/k heads, nonzero states (sampled units)."""
    dev = device()
    note("prefill 64 x 8 tokens")
    inp = wl.prefill_inputs(48, [8] * 64, 16, 32, 128, state_std=0.02)
    o, fin = _prefill_gpu(inp, dev)
    units = [(n, (5 * n + 1) % 32) for n in range(64)] + [(3, h) for h in range(32)]
    _sampled_check(inp, o, fin, units, "64 x 8")


def test_decode_multitoken_workload_parity():
    """The bench's multi-token decode step: 64 sequences x 4 new tokens, 32
    value / 16 q/k heads, states updated in place (sampled units)."""
    dev = device()
    w = wl.WORKLOADS["decode_multitoken"]
    note("multi-token decode workload 64 x 4, in place")
    inp = wl.prefill_inputs(w["seed"], [w["len"]] * w["N"], w["H_qk"], w["H_v"], w["D"],
                            state_std=w["state_std"])
    o, fin = _prefill_gpu(inp, dev, in_place=True)
    units = [(n, (3 * n + 5) % w["H_v"]) for n in range(w["N"])] + [(0, h) for h in range(w["H_v"])]
    _sampled_check(inp, o, fin, units, "multi-token decode 64 x 4")



@pytest.mark.parametrize("D", [16, 128])
def test_prefill_indexed_pool(D):
    """Sequences start from, and leave their final state in, the pool slots
    state_idx names: slots and outputs equal gdn_prefill_varlen on the gathered
    states bit for bit (both routes), and the oracle; other slots, and the
    outputs of a sequence whose index is -1, are untouched."""
    import torch

    dev = device()
    lengths = [0, 3, 8, 9, 70, 130] if D == 128 else [5, 0, 20, 33]
    slots = np.array([7, -1, 2, 9, 0, 4] if D == 128 else [1, 3, -1, 0], np.int32)
    P = 10 if D == 128 else 4
    note(f"prefill indexed D={D} lengths {lengths} slots {slots.tolist()}")
    inp = wl.prefill_inputs(49 + D, lengths, 2, 4, D)
    rng = np.random.default_rng(50 + D)
    pool_host = (0.02 * rng.standard_normal((P, 4, D, D))).astype(np.float32)
    valid = (slots >= 0) & (slots < P)
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    pool = to_dev(pool_host, dev)
    o = torch.full((inp.q.shape[0], 4, D), float("nan"), dtype=torch.bfloat16, device=dev)
    ws = _workspace(len(lengths), int(sum(lengths)), 2, 4, D, dev)
    gdn.gdn_prefill_varlen_indexed(q, k, v, g, b, cu, pool, to_dev(slots, dev), o, workspace=ws)
    _assert_no_wait_fault(ws, len(lengths))
    # the same sequences with gdn_prefill_varlen on the gathered states
    init_host = np.stack([pool_host[s] if ok else np.zeros_like(pool_host[0]) for s, ok in zip(slots, valid)])
    init = to_dev(init_host, dev)
    fin = torch.empty_like(init)
    o2 = torch.empty_like(o)
    gdn.gdn_prefill_varlen(q, k, v, g, b, cu, init, fin, o2)
    torch.cuda.synchronize()
    cu_h = inp.cu_seqlens
    pool_np, fin_np = pool.cpu().numpy(), fin.cpu().numpy()
    for n, (s, ok) in enumerate(zip(slots, valid)):
        rows = slice(cu_h[n], cu_h[n + 1])
        if ok:
            assert np.array_equal(pool_np[s], fin_np[n]), n
            assert torch.equal(o[rows].view(torch.int16), o2[rows].view(torch.int16)), n
        else:
            assert torch.isnan(o[rows].float()).all(), n
    untouched = np.setdiff1d(np.arange(P), slots[valid])
    assert np.array_equal(pool_np[untouched], pool_host[untouched])
    o_ref, s_ref = ref.prefill_varlen(inp.q, inp.k, inp.v, inp.g, inp.beta, cu_h, init_host,
                                      scale=inp.scale)
    keep = np.concatenate([np.arange(cu_h[n], cu_h[n + 1]) for n in range(len(lengths)) if valid[n]])
    check_outputs(bf16_np(o)[keep], o_ref[keep], f"indexed D={D}")
    check_states(pool_np[slots[valid]], s_ref[valid], f"indexed D={D}")


def test_prefill_indexed_pool_many_short_sequences():
    """800 sequences of 0..8 tokens on a 1,000-slot pool (shuffled slots, some
    -1): every token-by-token workgroup walks several units, prefetching the
    next unit's state.  Slots and outputs equal gdn_prefill_varlen on the
    gathered states bit for bit; skipped sequences' rows and unnamed slots are
    untouched; the oracle on every sequence."""
    import torch

    dev = device()
    rng = np.random.default_rng(52)
    N, P, D = 800, 1000, 128
    lengths = rng.integers(0, 9, size=N).tolist()
    slots = rng.permutation(P)[:N].astype(np.int32)
    slots[rng.choice(N, size=40, replace=False)] = -1
    valid = slots >= 0
    note(f"prefill indexed, {N} short sequences, T={sum(lengths)}")
    inp = wl.prefill_inputs(53, lengths, 2, 4, D)
    pool_host = (0.02 * rng.standard_normal((P, 4, D, D))).astype(np.float32)
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    pool = to_dev(pool_host, dev)
    o = torch.full((inp.q.shape[0], 4, D), float("nan"), dtype=torch.bfloat16, device=dev)
    ws = _workspace(N, int(sum(lengths)), 2, 4, D, dev)
    gdn.gdn_prefill_varlen_indexed(q, k, v, g, b, cu, pool, to_dev(slots, dev), o, workspace=ws)
    _assert_no_wait_fault(ws, N)
    init_host = np.where(valid[:, None, None, None], pool_host[np.maximum(slots, 0)], 0.0).astype(np.float32)
    init = to_dev(init_host, dev)
    fin = torch.empty_like(init)
    o2 = torch.empty_like(o)
    gdn.gdn_prefill_varlen(q, k, v, g, b, cu, init, fin, o2)
    torch.cuda.synchronize()
    pool_np, fin_np = pool.cpu().numpy(), fin.cpu().numpy()
    assert np.array_equal(pool_np[slots[valid]], fin_np[valid])
    cu_h = inp.cu_seqlens
    keep = np.concatenate([np.arange(cu_h[n], cu_h[n + 1]) for n in range(N) if valid[n]])
    skip = np.concatenate([np.arange(cu_h[n], cu_h[n + 1]) for n in range(N) if not valid[n]])
    assert torch.equal(o[keep].view(torch.int16), o2[keep].view(torch.int16))
    assert torch.isnan(o[skip].float()).all()
    untouched = np.setdiff1d(np.arange(P), slots[valid])
    assert np.array_equal(pool_np[untouched], pool_host[untouched])
    o_ref, s_ref = ref.prefill_varlen(inp.q, inp.k, inp.v, inp.g, inp.beta, cu_h, init_host, scale=inp.scale)
    check_outputs(bf16_np(o)[keep], o_ref[keep], "indexed, many short")
    check_states(pool_np[slots[valid]], s_ref[valid], "indexed, many short")
