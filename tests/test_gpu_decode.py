"""gdn_decode on the GPU (through the C ABI) against the fp64 oracle."""
import numpy as np
import pytest

import oracle.gdn_ref as ref
from gpu_helpers import (bf16_np, check_outputs, check_states, device, note, record, to_dev)
from paper_2607_17979_amd import gdn
from paper_2607_17979_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _decode_gpu(step, state_t, dev, scale=1.0):
    import torch

    q, k, v = (to_dev(x, dev, bf16=True) for x in (step.q, step.k, step.v))
    g, b = to_dev(step.g, dev), to_dev(step.beta, dev)
    o = torch.empty(v.shape, dtype=torch.bfloat16, device=dev)
    gdn.gdn_decode(q, k, v, g, b, state_t, o, scale=scale)
    return o


def test_library_is_the_native_one():
    import torch

    dev = device()
    lib = gdn.load_library()
    assert lib.gdn_abi_version() == 210
    maps = open("/proc/self/maps").read()
    assert "libgdn_mi355x.so" in maps
    assert torch.cuda.get_device_properties(dev).gcnArchName.startswith("gfx950")


def test_decode_tiny_sequence_matches_prefill_oracle():
    """The tiny workload (d = 16, two heads): 64 consecutive decode calls."""
    import torch

    dev = device()
    w = wl.WORKLOADS["tiny"]
    inp = wl.prefill_inputs(w["seed"], [w["T"]], w["H_qk"], w["H_v"], w["D"])
    note(f"decode tiny: T={w['T']} H={w['H_v']} D={w['D']}")
    o_ref, s_ref = ref.prefill_varlen(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens, None)
    state = torch.zeros((1, w["H_v"], w["D"], w["D"]), dtype=torch.float32, device=dev)
    outs = []
    for t in range(w["T"]):
        st = wl.DecodeInputs(inp.q[t:t + 1], inp.k[t:t + 1], inp.v[t:t + 1], inp.g[t:t + 1],
                             inp.beta[t:t + 1], None)
        outs.append(bf16_np(_decode_gpu(st, state, dev)))
    torch.cuda.synchronize()
    check_outputs(np.concatenate(outs), o_ref, "tiny decode")
    check_states(state.cpu().numpy(), s_ref, "tiny decode")


@pytest.mark.parametrize("seed", [2, 12, 22])
def test_decode_b64_parity(seed):
    """Batch 64, 32 value heads on 16 q/k heads, d = 128, state ~ 0.02 N(0,1)."""
    import torch

    dev = device()
    w = wl.WORKLOADS["decode_b64"]
    note(f"decode b64 seed {seed}")
    inp = wl.decode_inputs(seed, w["B"], w["H_qk"], w["H_v"], w["D"], state_std=w["state_std"])
    state = to_dev(inp.state, dev)
    o = _decode_gpu(inp, state, dev)
    torch.cuda.synchronize()
    o_ref, s_ref = ref.decode(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.state)
    check_outputs(bf16_np(o), o_ref, "b64")
    check_states(state.cpu().numpy(), s_ref, "b64")


def _sample_units(rng, B, H_v, n):
    if B * H_v <= n:
        bb, hh = np.meshgrid(np.arange(B), np.arange(H_v), indexing="ij")
        return bb.ravel(), hh.ravel()
    flat = rng.choice(B * H_v, size=n, replace=False)
    return flat // H_v, flat % H_v


@pytest.mark.parametrize("seed_off", [0, 1000, 2000])
@pytest.mark.parametrize("B", [1, 8, 256, 1024])
def test_decode_sweep_100_steps(B, seed_off):
    """100 consecutive in-place steps with fresh inputs, three seeds per batch
    size; the oracle follows a seeded sample of (b, h) units (units are
    independent, so this is exact)."""
    import torch

    dev = device()
    w = wl.WORKLOADS["decode_sweep"]
    H_qk, H_v, D, steps = w["H_qk"], w["H_v"], w["D"], w["steps"]
    seed = w["seed"] + B + seed_off
    note(f"decode sweep B={B} x {steps} steps, seed {seed}")
    state0 = wl.decode_state(seed, B, H_v, D, w["state_std"])
    state = to_dev(state0, dev)
    bs, hs = _sample_units(np.random.default_rng(B + seed_off), B, H_v, 32)
    hq = ref.head_map(H_qk, H_v)
    S = ref.to_f64(state0[bs, hs])[:, None]
    worst_o = 0.0
    for s in range(steps):
        st = wl.decode_step_inputs(seed, s, B, H_qk, H_v, D)
        o = _decode_gpu(st, state, dev)
        o_ref, S = ref.decode(st.q[bs, hq[hs]][:, None], st.k[bs, hq[hs]][:, None],
                              st.v[bs, hs][:, None], st.g[bs, hs][:, None], st.beta[bs, hs][:, None], S)
        got = ref.to_f64(bf16_np(o)[bs, hs])
        worst_o = max(worst_o, float(np.max(np.abs(got - o_ref[:, 0]))))
    torch.cuda.synchronize()
    note(f"  sweep B={B}: outputs max-abs over {steps} steps {worst_o:.3e}")
    record("outputs max-abs", f"sweep B={B}", worst_o)
    assert worst_o <= 2e-2
    got_s = state[torch.as_tensor(bs, device=dev), torch.as_tensor(hs, device=dev)].cpu().numpy()
    check_states(got_s, S[:, 0], f"sweep B={B}")


def test_decode_identity_gate_leaves_state_bitwise():
    """alpha = 1 (g = 0), beta = 0: the state is unchanged bit for bit and
    o = scale S q."""
    import torch

    dev = device()
    inp = wl.decode_inputs(7, 4, 2, 4, 128, state_std=0.5)
    inp.g[:] = 0.0
    inp.beta[:] = 0.0
    state = to_dev(inp.state, dev)
    o = _decode_gpu(inp, state, dev, scale=0.5)
    torch.cuda.synchronize()
    assert np.array_equal(state.cpu().numpy(), inp.state)
    o_ref, _ = ref.decode(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.state, scale=0.5)
    check_outputs(bf16_np(o), o_ref, "identity gate")


def test_decode_recall_unit_key():
    """beta = 1, k = q = e_j: column j of the new state and the output are v."""
    import torch

    dev = device()
    B, H, D = 3, 2, 128
    inp = wl.decode_inputs(8, B, H, H, D, state_std=0.1)
    j = np.array([5, 77, 127])
    e = np.zeros((B, H, D), np.float32)
    e[np.arange(B), :, j] = 1.0
    inp.q = wl.bf16_bits(e)
    inp.k = wl.bf16_bits(e)
    inp.beta[:] = 1.0
    state = to_dev(inp.state, dev)
    o = _decode_gpu(inp, state, dev)
    torch.cuda.synchronize()
    v = ref.to_f64(inp.v)
    got_o = ref.to_f64(bf16_np(o))
    assert np.max(np.abs(got_o - v)) <= 1e-2
    S = state.cpu().numpy()
    for b in range(B):
        assert np.max(np.abs(S[b, :, :, j[b]] - v[b])) <= 1e-5


def test_decode_scale_and_determinism():
    import torch

    dev = device()
    inp = wl.decode_inputs(9, 16, 4, 8, 128)
    s1, s2 = to_dev(inp.state, dev), to_dev(inp.state, dev)
    scale = 128 ** -0.5
    o1 = _decode_gpu(inp, s1, dev, scale=scale)
    o2 = _decode_gpu(inp, s2, dev, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(s1, s2)
    o_ref, s_ref = ref.decode(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.state, scale=scale)
    check_outputs(bf16_np(o1), o_ref, "scaled")
    check_states(s1.cpu().numpy(), s_ref, "scaled")


def test_decode_gva_equals_repeated_heads_bitwise():
    """Value heads 2j, 2j+1 read q/k head j: the same call with q/k repeated to
    H_v heads gives identical bits."""
    import torch

    dev = device()
    inp = wl.decode_inputs(10, 8, 4, 8, 128)
    s1, s2 = to_dev(inp.state, dev), to_dev(inp.state, dev)
    o1 = _decode_gpu(inp, s1, dev)
    rep = wl.DecodeInputs(np.repeat(inp.q, 2, axis=1), np.repeat(inp.k, 2, axis=1), inp.v, inp.g,
                          inp.beta, None)
    o2 = _decode_gpu(rep, s2, dev)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(s1, s2)


def test_decode_zero_batch():
    import torch

    dev = device()
    z = torch.empty((0, 2, 128), dtype=torch.bfloat16, device=dev)
    zv = torch.empty((0, 4, 128), dtype=torch.bfloat16, device=dev)
    zf = torch.empty((0, 4), dtype=torch.float32, device=dev)
    zs = torch.empty((0, 4, 128, 128), dtype=torch.float32, device=dev)
    gdn.gdn_decode(z, z, zv, zf, zf, zs, zv.clone())
    torch.cuda.synchronize()


def test_decode_graph_replay_matches_eager():
    """Decode steps captured once in a HIP graph and replayed three times, with
    eager steps and synchronisations between the replays, leave bitwise the
    states and outputs of the same steps run eagerly (the benchmark's decode
    sweep times such replays)."""
    import torch

    dev = device()
    B, H_qk, H_v, D, n, seed = 8, 16, 32, 128, 6, 31
    note(f"decode graph replay: B={B}, {n} steps per replay, 3 replays")
    xs = []
    for s in range(n):
        st = wl.decode_step_inputs(seed, s, B, H_qk, H_v, D)
        xs.append(dict(q=to_dev(st.q, dev, bf16=True), k=to_dev(st.k, dev, bf16=True),
                       v=to_dev(st.v, dev, bf16=True), g=to_dev(st.g, dev), b=to_dev(st.beta, dev)))
    state0 = wl.decode_state(seed, B, H_v, D, 0.02)

    def outs():
        return [torch.empty((B, H_v, D), dtype=torch.bfloat16, device=dev) for _ in range(n)]

    def run(state, os_):
        for x, o in zip(xs, os_):
            gdn.gdn_decode(x["q"], x["k"], x["v"], x["g"], x["b"], state, o)

    s_graph, o_graph = to_dev(state0, dev), outs()
    s_eager, o_eager = to_dev(state0, dev), outs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(to_dev(state0, dev), outs())          # warm-up before capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run(s_graph, o_graph)
    torch.cuda.synchronize()
    assert torch.equal(s_graph, to_dev(state0, dev)), "capture must not execute the steps"
    for r in range(3):
        graph.replay()
        torch.cuda.synchronize()
        run(s_eager, o_eager)
        torch.cuda.synchronize()
        assert torch.equal(s_graph, s_eager), f"state after replay {r}"
        for i, (a, b) in enumerate(zip(o_graph, o_eager)):
            assert torch.equal(a, b), f"output of step {i} after replay {r}"


def test_decode_indexed_pool():
    """Batch entries update the pool slots state_idx names: those slots and the
    outputs equal gdn_decode on the gathered states bit for bit, and the
    oracle; slots not named, and the output rows of entries whose index is
    -1 or past the pool, are left untouched."""
    import torch

    dev = device()
    B, P, H_qk, H_v, D = 64, 96, 16, 32, 128
    note(f"decode indexed B={B} P={P}")
    inp = wl.decode_inputs(60, B, H_qk, H_v, D, state_std=0.0)
    rng = np.random.default_rng(61)
    pool_host = (0.02 * rng.standard_normal((P, H_v, D, D))).astype(np.float32)
    slots = rng.permutation(P)[:B].astype(np.int32)
    slots[[3, 10]] = -1
    slots[20] = P
    valid = (slots >= 0) & (slots < P)
    pool = to_dev(pool_host, dev)
    q, k, v = (to_dev(x, dev, bf16=True) for x in (inp.q, inp.k, inp.v))
    g, b = to_dev(inp.g, dev), to_dev(inp.beta, dev)
    o = torch.full(v.shape, float("nan"), dtype=torch.bfloat16, device=dev)
    gdn.gdn_decode_indexed(q, k, v, g, b, pool, to_dev(slots, dev), o)
    # the same step with gdn_decode on the gathered states of the valid entries
    vi = torch.as_tensor(np.nonzero(valid)[0], device=dev)
    st = to_dev(pool_host[slots[valid]], dev)
    o2 = torch.empty((int(valid.sum()), H_v, D), dtype=torch.bfloat16, device=dev)
    gdn.gdn_decode(q[vi].contiguous(), k[vi].contiguous(), v[vi].contiguous(), g[vi].contiguous(),
                   b[vi].contiguous(), st, o2)
    torch.cuda.synchronize()
    pool_np = pool.cpu().numpy()
    assert np.array_equal(pool_np[slots[valid]], st.cpu().numpy())
    assert torch.equal(o[vi].view(torch.int16), o2.view(torch.int16))
    assert torch.isnan(o[torch.as_tensor(np.nonzero(~valid)[0], device=dev)].float()).all()
    untouched = np.setdiff1d(np.arange(P), slots[valid])
    assert np.array_equal(pool_np[untouched], pool_host[untouched])
    o_ref, s_ref = ref.decode(inp.q[valid], inp.k[valid], inp.v[valid], inp.g[valid], inp.beta[valid],
                              pool_host[slots[valid]])
    check_outputs(bf16_np(o[vi]), o_ref, "indexed")
    check_states(pool_np[slots[valid]], s_ref, "indexed")


def test_decode_state_beyond_4gib():
    """Batch 4,096 x 32 value heads: 8 GiB of fp32 state, so byte offsets into
    it need more than 32 bits past the first half.  Inputs drawn on the device
    by torch's seeded generator; the oracle checks the first (batch, head)
    unit and the one at the highest addresses."""
    import torch

    dev = device()
    B, H_qk, H_v, D = 4096, 16, 32, 128
    note(f"decode state beyond 4 GiB: B={B}, H_v={H_v} ({B * H_v * D * D * 4 / 2**30:.0f} GiB)")
    x = wl.decode_inputs_device(71, B, H_qk, H_v, D, 0.02, dev)
    units = ((0, 0), (B - 1, H_v - 1))
    before = {u: x["state"][u[0], u[1]].cpu().numpy() for u in units}
    o = torch.empty((B, H_v, D), dtype=torch.bfloat16, device=dev)
    gdn.gdn_decode(x["q"], x["k"], x["v"], x["g"], x["beta"], x["state"], o)
    torch.cuda.synchronize()

    def bits(t):
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

    for b, h in units:
        hq = h * H_qk // H_v
        o_ref, s_ref = ref.decode(bits(x["q"][b:b + 1, hq:hq + 1]), bits(x["k"][b:b + 1, hq:hq + 1]),
                                  bits(x["v"][b:b + 1, h:h + 1]), x["g"][b:b + 1, h:h + 1].cpu().numpy(),
                                  x["beta"][b:b + 1, h:h + 1].cpu().numpy(), before[(b, h)][None, None])
        check_outputs(bits(o[b:b + 1, h:h + 1]), o_ref, f"decode 8 GiB, unit ({b}, {h})")
        check_states(x["state"][b:b + 1, h:h + 1].cpu().numpy(), s_ref, f"decode 8 GiB, unit ({b}, {h})")
