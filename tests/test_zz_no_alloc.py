"""gdn_prefill_varlen_noalloc on the GPU: the entry point for callers that
cannot allocate, whose workspace is the library's static per-GPU scratch.
Through the C ABI it must give bit for bit the outputs and final states of
gdn_prefill_varlen with a caller workspace, on two calls in a row (the second
with a smaller batch, so the scratch holds the first call's schedule when the
second starts), for both head dims, and match the oracle."""
import numpy as np
import pytest

import oracle.gdn_ref as ref
from gpu_helpers import bf16_np, check_outputs, check_states, device, note, to_dev
from paper_2607_17979_amd import gdn
from paper_2607_17979_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _run(inp, dev, noalloc):
    import torch

    N, T, H_qk, H_v, D = inp.shape
    q, k, v = (to_dev(a, dev, bf16=True) for a in (inp.q, inp.k, inp.v))
    g, b, cu = to_dev(inp.g, dev), to_dev(inp.beta, dev), to_dev(inp.cu_seqlens, dev)
    init = to_dev(inp.initial_state, dev)
    fin = torch.full((N, H_v, D, D), float("nan"), dtype=torch.float32, device=dev)
    o = torch.full((T, H_v, D), float("nan"), dtype=torch.bfloat16, device=dev)
    if noalloc:
        gdn.gdn_prefill_varlen_noalloc(q, k, v, g, b, cu, init, fin, o, scale=inp.scale)
    else:
        ws = gdn.gdn_prefill_varlen(q, k, v, g, b, cu, init, fin, o, scale=inp.scale)
        assert gdn.workspace_fault(ws, N) == 0
    torch.cuda.synchronize()
    return o, fin


@pytest.mark.parametrize("D", [128, 16])
def test_noalloc_equals_workspace_entry_point(D):
    import torch

    dev = device()
    C = 64 if D == 128 else 16
    batches = [
        wl.prefill_inputs(801, [3 * C + 5, 0, 7, 2 * C, C + 1, 300, 5, 1], 2, 4, D, state_std=0.02,
                          scale=D ** -0.5),
        wl.prefill_inputs(802, [C - 1, 2 * C + 9, 4], 2, 4, D, state_std=0.02, scale=D ** -0.5),
    ]
    for i, inp in enumerate(batches):
        note(f"no-allocation entry point D={D}, call {i + 1}: lengths {np.diff(inp.cu_seqlens).tolist()}")
        o_ws, f_ws = _run(inp, dev, noalloc=False)
        o_na, f_na = _run(inp, dev, noalloc=True)
        assert torch.equal(o_na.view(torch.int16), o_ws.view(torch.int16)), i
        assert torch.equal(f_na.view(torch.int32), f_ws.view(torch.int32)), i
        o_ref, s_ref = ref.prefill_varlen(inp.q, inp.k, inp.v, inp.g, inp.beta, inp.cu_seqlens,
                                          inp.initial_state, scale=inp.scale)
        check_outputs(bf16_np(o_na), o_ref, f"no-allocation D={D} call {i + 1}")
        check_states(f_na.cpu().numpy(), s_ref, f"no-allocation D={D} call {i + 1}")


def test_noalloc_rejects_too_many_sequences():
    import torch

    dev = device()
    N = 16385
    z = torch.zeros((N, 1, 128), dtype=torch.bfloat16, device=dev)
    zv = torch.zeros((N, 2, 128), dtype=torch.bfloat16, device=dev)
    zf = torch.zeros((N, 2), dtype=torch.float32, device=dev)
    cu = torch.arange(N + 1, dtype=torch.int32, device=dev)
    fin = torch.empty((N, 2, 128, 128), dtype=torch.float32, device=dev)
    with pytest.raises(gdn.GdnError, match="16384"):
        gdn.gdn_prefill_varlen_noalloc(z, z, zv, zf, zf, cu, None, fin, zv.clone())
