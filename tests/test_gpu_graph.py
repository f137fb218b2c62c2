"""Prefill-regime calls captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed, for serving loops that replay a captured step: the no-allocation
entry point (its workspace is the library's static scratch) and
gdn_prefill_varlen with a workspace allocated before the capture.  The calls
run in place (initial_state == final_state), so every replay advances the
states by one call; after each of three replays, with eager calls of the same
step and synchronisations in between, the graph's states and outputs must
equal the eager ones bit for bit.  The batches mix sequences of at most 8
tokens (token-by-token launch), longer ones (chunk kernel) and an empty one;
both head dims."""
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
