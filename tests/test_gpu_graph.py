"""Prefill-regime calls captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed, for serving loops that replay a captured step: the no-allocation
entry point (its workspace is the library's static scratch) and
gdn_prefill_varlen with a workspace allocated before the capture.  The calls
run in place (initial_state == final_state), so every replay advances the
states by one call; after each of three replays, with eager calls of the same
step and synchronisations in between, the graph's states and outputs must
equal the eager ones bit for bit.  The batches mix sequences of at most 8
tokens (token-by-token launch), longer ones (chunk kernel) and an empty one;
both head dims.  Also: calls issued on a side stream (the binding's stream
argument) match those on the current stream bit for bit."""
import pytest

from gpu_helpers import device, note, to_dev
from paper_2607_17979_amd import gdn
from paper_2607_17979_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("entry", ["noalloc", "workspace"])
@pytest.mark.parametrize("D", [128, 16])
def test_prefill_graph_replay_matches_eager(D, entry):
    import torch

    dev = device()
    C = gdn.default_chunk(D)
    lengths = [3 * C + 5, 0, 7, 2 * C + 2, 1, C + 6] if D == 128 else [2 * C + 3, 0, 5, C, 1]
    inp = wl.prefill_inputs(901 + D, lengths, 2, 4, D, state_std=0.02, scale=D ** -0.5)
    N, T, H_qk, H_v, _ = inp.shape
    note(f"prefill graph replay: D={D}, {entry}, lengths {lengths}, 3 replays")
    q, k, v = (to_dev(a, dev, bf16=True) for a in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    state0 = to_dev(inp.initial_state, dev)
    ws = torch.empty(gdn.gdn_prefill_workspace_size(N, T, H_v, D, D, C), dtype=torch.uint8, device=dev)

    def call(state, o):
        if entry == "noalloc":
            gdn.gdn_prefill_varlen_noalloc(q, k, v, g, b, cu, state, state, o, scale=inp.scale)
        else:
            gdn.gdn_prefill_varlen(q, k, v, g, b, cu, state, state, o, scale=inp.scale, workspace=ws)

    def out():
        return torch.full((T, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)

    s_graph, o_graph = state0.clone(), out()
    s_eager, o_eager = state0.clone(), out()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(state0.clone(), out())               # warm-up before the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(s_graph, o_graph)
    torch.cuda.synchronize()
    assert torch.equal(s_graph, state0), "the capture must not run the call"
    for r in range(3):
        graph.replay()
        torch.cuda.synchronize()
        call(s_eager, o_eager)
        torch.cuda.synchronize()
        assert torch.equal(s_graph.view(torch.int32), s_eager.view(torch.int32)), f"states after replay {r}"
        assert torch.equal(o_graph.view(torch.int16), o_eager.view(torch.int16)), f"outputs after replay {r}"
        if entry == "workspace":
            assert gdn.workspace_fault(ws, N) == 0
    assert not torch.equal(s_graph, state0), "the replays must advance the states"


def test_calls_on_a_side_stream_match_the_current_stream():
    """The binding's stream argument: a decode step and a prefill call (with
    the workspace the binding allocates on the launch stream) issued on a side
    stream while the current stream is kept busy give bit for bit the results
    of the same calls on the current stream."""
    import torch

    dev = device()
    note("decode and prefill on a side stream")
    d = wl.decode_inputs(911, 16, 16, 32, 128)
    dq, dk, dv = (to_dev(a, dev, bf16=True) for a in (d.q, d.k, d.v))
    dg, db = to_dev(d.g, dev), to_dev(d.beta, dev)
    p = wl.prefill_inputs(912, [150, 3, 0, 64, 9], 2, 4, 128, state_std=0.02)
    N, T, _, H_v, D = p.shape
    pq, pk, pv = (to_dev(a, dev, bf16=True) for a in (p.q, p.k, p.v))
    pg, pb, cu = to_dev(p.g, dev), to_dev(p.beta, dev), to_dev(p.cu_seqlens, dev)
    init = to_dev(p.initial_state, dev)

    def buffers():
        return (to_dev(d.state, dev), torch.empty((16, 32, 128), dtype=torch.bfloat16, device=dev),
                torch.empty((N, H_v, D, D), dtype=torch.float32, device=dev),
                torch.empty((T, H_v, D), dtype=torch.bfloat16, device=dev))

    def run(bufs, stream):
        st, od, fin, op = bufs
        gdn.gdn_decode(dq, dk, dv, dg, db, st, od, stream=stream)
        ws = gdn.gdn_prefill_varlen(pq, pk, pv, pg, pb, cu, init, fin, op, stream=stream)
        return (st, od, fin, op, ws)

    ref = run(buffers(), None)
    side_bufs = buffers()
    busy = torch.randn((4096, 4096), device=dev)
    torch.cuda.synchronize()
    for _ in range(8):
        busy = torch.mm(busy, busy) * 1e-3    # keeps the current stream busy meanwhile
    side = torch.cuda.Stream()
    got = run(side_bufs, side)
    torch.cuda.synchronize()
    assert gdn.workspace_fault(got[4], N) == 0
    for a, b in zip(ref[:4], got[:4]):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32))
