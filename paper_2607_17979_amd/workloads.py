"""Seeded synthetic inputs for the Gated DeltaNet decode and varlen-prefill paths.

This module only draws numbers; it holds none of the recurrence's arithmetic.
Both the CPU oracle (through the tests) and the HIP path (through the binding,
the tests and the benchmark) take their inputs from here, so the two sides see
bit-identical operands.

Distributions follow the workload descriptions used throughout the build:
  q, k : N(0, 1) in fp32, L2-normalised over the head dimension, then rounded
         to bf16 (round-to-nearest-even).  The kernels do not normalise.
  v    : N(0, 1) rounded to bf16.
  beta : sigmoid(N(0, 1)) in fp32, i.e. post-sigmoid write strength in (0, 1).
  g    : -softplus(N(0, 1)) in fp32, the natural-log gate; alpha = exp(g).
  state: 0.02 * N(0, 1) in fp32 (std 0.02), or zeros where a workload says so.

bf16 tensors are returned as numpy ``uint16`` arrays holding the raw bit
patterns; :func:`to_torch` turns them into ``torch.bfloat16`` tensors without
changing a bit.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "bf16_bits",
    "DecodeInputs",
    "PrefillInputs",
    "decode_inputs",
    "decode_state",
    "decode_step_inputs",
    "prefill_inputs",
    "varlen_lengths",
    "WORKLOADS",
    "to_torch",
]


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return the uint16 bit patterns.

    NaN is not produced by the generators and is not handled specially.
    """
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


_BLOCK = 1 << 21  # elements per independently seeded block


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _normal(entropy: Tuple[int, ...], shape, unit_last: bool = False, std: float = 1.0,
            bf16: bool = False) -> np.ndarray:
    """N(0, 1) draws of ``shape`` in fixed blocks of rows; block i is drawn from
    PCG64(SeedSequence(entropy + (i,))), so the values do not depend on the
    number of worker threads.  ``unit_last`` L2-normalises over the last axis;
    ``std`` scales; ``bf16`` returns bf16 bit patterns (uint16)."""
    shape = tuple(int(x) for x in shape)
    n = int(np.prod(shape)) if shape else 1
    row = shape[-1] if (unit_last and shape) else 1
    block = max(row, (_BLOCK // row) * row)
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    nblocks = (n + block - 1) // block

    def work(i):
        s, e = i * block, min(n, (i + 1) * block)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(tuple(entropy) + (i,))))
        x = rng.standard_normal(e - s, dtype=np.float32)
        if unit_last:
            x2 = x.reshape(-1, row)
            x2 /= np.sqrt(np.einsum("ij,ij->i", x2, x2))[:, None]
        if std != 1.0:
            x *= np.float32(std)
        out[s:e] = bf16_bits(x) if bf16 else x

    if nblocks <= 1:
        for i in range(nblocks):
            work(i)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(nblocks)))
    return out.reshape(shape)


def _softplus(x: np.ndarray) -> np.ndarray:
    return np.logaddexp(np.float32(0.0), x).astype(np.float32)


def _sigmoid(x: np.ndarray) -> np.ndarray:
    return (1.0 / (1.0 + np.exp(-x))).astype(np.float32)


# tensor tags mixed into the seeds
_Q, _K, _V, _BETA, _G, _STATE, _LEN = 1, 2, 3, 4, 5, 6, 7


@dataclasses.dataclass
class DecodeInputs:
    """One decode step: q, k [B, H_qk, D] bf16 bits; v [B, H_v, D] bf16 bits;
    g, beta [B, H_v] fp32; state [B, H_v, D_v, D_k] fp32 (k index contiguous)."""

    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: np.ndarray
    state: np.ndarray
    scale: float = 1.0

    @property
    def shape(self):
        B, H_qk, D = self.q.shape
        return B, H_qk, self.v.shape[1], D


@dataclasses.dataclass
class PrefillInputs:
    """Packed varlen prefill: q, k [T, H_qk, D] bf16 bits; v [T, H_v, D] bf16 bits;
    g, beta [T, H_v] fp32; cu_seqlens int32 [N + 1]; initial_state fp32
    [N, H_v, D_v, D_k] or None (zero state)."""

    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    g: np.ndarray
    beta: np.ndarray
    cu_seqlens: np.ndarray
    initial_state: Optional[np.ndarray]
    scale: float = 1.0

    @property
    def shape(self):
        T, H_qk, D = self.q.shape
        return len(self.cu_seqlens) - 1, T, H_qk, self.v.shape[1], D


def decode_inputs(seed: int, B: int, H_qk: int, H_v: int, D: int,
                  state_std: float = 0.02, scale: float = 1.0,
                  qkv_dtype: str = "bf16", raw: Optional[float] = None) -> DecodeInputs:
    """Draw one decode step and its prior state.  ``qkv_dtype="f32"`` keeps
    q/k/v as fp32 (oracle-only use); ``raw`` as decode_step_inputs."""
    step = decode_step_inputs(seed, 0, B, H_qk, H_v, D, qkv_dtype=qkv_dtype, raw=raw)
    step.state = decode_state(seed, B, H_v, D, state_std)
    step.scale = scale
    return step


def decode_state(seed: int, B: int, H_v: int, D: int, state_std: float = 0.02) -> np.ndarray:
    """Prior decode state [B, H_v, D, D] fp32: std * N(0, 1), or zeros if std is 0."""
    if state_std == 0.0:
        return np.zeros((B, H_v, D, D), np.float32)
    return _normal((seed, _STATE), (B, H_v, D, D), std=state_std)


def decode_step_inputs(seed: int, step: int, B: int, H_qk: int, H_v: int, D: int,
                       qkv_dtype: str = "bf16", raw: Optional[float] = None) -> DecodeInputs:
    """Fresh q, k, v, g, beta for decode step ``step`` (state left as None).
    ``raw`` (a scale) draws the inputs of the fused prologue instead: q, k
    N(0, raw^2) per element, not normalised; g and beta the N(0, 1) logits
    themselves (g = -softplus and beta = sigmoid of them are then the
    kernel's work)."""
    bf = qkv_dtype == "bf16"
    unit = raw is None
    std = 1.0 if raw is None else raw
    q = _normal((seed, step, _Q), (B, H_qk, D), unit_last=unit, std=std, bf16=bf)
    k = _normal((seed, step, _K), (B, H_qk, D), unit_last=unit, std=std, bf16=bf)
    v = _normal((seed, step, _V), (B, H_v, D), bf16=bf)
    xb = _normal((seed, step, _BETA), (B, H_v))
    xg = _normal((seed, step, _G), (B, H_v))
    if raw is not None:
        return DecodeInputs(q, k, v, xg, xb, None)
    return DecodeInputs(q, k, v, -_softplus(xg), _sigmoid(xb), None)


def varlen_lengths(seed: int, N: int, lo: int, hi: int) -> np.ndarray:
    """N sequence lengths drawn uniformly from the integers in [lo, hi]."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence((seed, _LEN))))
    return rng.integers(lo, hi + 1, size=N).astype(np.int64)


def prefill_inputs(seed: int, lengths: Sequence[int], H_qk: int, H_v: int, D: int,
                   state_std: Optional[float] = None, scale: float = 1.0,
                   qkv_dtype: str = "bf16", raw: Optional[float] = None) -> PrefillInputs:
    """Draw a packed varlen batch.  ``state_std=None`` means a zero initial state
    (passed to the library as NULL).  ``raw`` (a scale) draws the inputs of the
    fused prologue instead: q, k N(0, raw^2) per element, not normalised; g and
    beta the N(0, 1) logits themselves."""
    lengths = np.asarray(lengths, dtype=np.int64)
    N = len(lengths)
    cu = np.zeros(N + 1, np.int64)
    np.cumsum(lengths, out=cu[1:])
    T = int(cu[-1])
    bf = qkv_dtype == "bf16"
    unit = raw is None
    std = 1.0 if raw is None else raw
    q = _normal((seed, _Q), (T, H_qk, D), unit_last=unit, std=std, bf16=bf)
    k = _normal((seed, _K), (T, H_qk, D), unit_last=unit, std=std, bf16=bf)
    v = _normal((seed, _V), (T, H_v, D), bf16=bf)
    xb = _normal((seed, _BETA), (T, H_v))
    xg = _normal((seed, _G), (T, H_v))
    beta, g = (xb, xg) if raw is not None else (_sigmoid(xb), -_softplus(xg))
    init = None
    if state_std is not None:
        init = _normal((seed, _STATE), (N, H_v, D, D), std=state_std)
    return PrefillInputs(q, k, v, g, beta, cu.astype(np.int32), init, scale)


def prefill_inputs_device(seed: int, N: int, L: int, H_qk: int, H_v: int, D: int,
                          state_std: float, device, g_scale: float = 1.0,
                          beta_range: Optional[Tuple[float, float]] = None):
    """An equal-length packed batch (N sequences of L tokens) drawn on the GPU
    with torch's seeded generator, for sizes whose host draw would take
    minutes; the same distributions as prefill_inputs: q, k N(0, 1)
    L2-normalised per head in fp32, then rounded to bf16; v N(0, 1) in bf16;
    beta = sigmoid(N(0, 1)); g = -softplus(N(0, 1)); initial state
    N(0, state_std^2).  ``g_scale`` multiplies g (0 gives g = 0 exactly, slow
    decay regimes lie between); ``beta_range`` = (lo, hi) draws beta uniformly
    in [lo, hi) instead.  Returns a dict of device tensors (q, k, v, g, beta,
    init, cu)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    T = N * L

    def normal(shape):
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)

    q = torch.empty((T, H_qk, D), dtype=torch.bfloat16, device=device)
    k = torch.empty_like(q)
    v = torch.empty((T, H_v, D), dtype=torch.bfloat16, device=device)
    for t0 in range(0, T, L):  # one sequence at a time: the fp32 draws stay small
        for dst, H, unit in ((q, H_qk, True), (k, H_qk, True), (v, H_v, False)):
            x = normal((L, H, D))
            if unit:
                x = x / x.norm(dim=-1, keepdim=True)
            dst[t0:t0 + L] = x.to(torch.bfloat16)
    beta = torch.sigmoid(normal((T, H_v)))
    if beta_range is not None:
        u = torch.rand((T, H_v), generator=gen, device=device, dtype=torch.float32)
        beta = beta_range[0] + (beta_range[1] - beta_range[0]) * u
    g = -torch.nn.functional.softplus(normal((T, H_v)))
    g = g * g_scale if g_scale != 0.0 else torch.zeros_like(g)
    init = torch.empty((N, H_v, D, D), dtype=torch.float32, device=device)
    for n0 in range(0, N, 256):  # in slices: no second full-size temporary
        init[n0:n0 + 256] = state_std * normal((min(256, N - n0), H_v, D, D))
    cu = torch.arange(N + 1, dtype=torch.int32, device=device) * L
    return dict(q=q, k=k, v=v, g=g, beta=beta, init=init, cu=cu)


def decode_inputs_device(seed: int, B: int, H_qk: int, H_v: int, D: int, state_std: float,
                         device):
    """One decode step's inputs drawn on the GPU with torch's seeded generator
    (for states of many GiB), with the distributions of decode_inputs.
    Returns a dict of device tensors (q, k, v, g, beta, state)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)

    def normal(shape):
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)

    q = normal((B, H_qk, D))
    k = normal((B, H_qk, D))
    q = (q / q.norm(dim=-1, keepdim=True)).to(torch.bfloat16)
    k = (k / k.norm(dim=-1, keepdim=True)).to(torch.bfloat16)
    v = normal((B, H_v, D)).to(torch.bfloat16)
    beta = torch.sigmoid(normal((B, H_v)))
    g = -torch.nn.functional.softplus(normal((B, H_v)))
    state = torch.empty((B, H_v, D, D), dtype=torch.float32, device=device)
    for b0 in range(0, B, 256):  # in slices: no second full-size temporary
        state[b0:b0 + 256] = state_std * normal((min(256, B - b0), H_v, D, D))
    return dict(q=q, k=k, v=v, g=g, beta=beta, state=state)


# The five synthetic workloads (sizes and distributions as described in the
# module docstring).  Values are plain dicts so both sides can read them.
WORKLOADS = {
    "tiny": dict(kind="both", N=1, T=64, H_qk=2, H_v=2, D=16, chunk=16, state_std=None, seed=1),
    "decode_b64": dict(kind="decode", B=64, H_qk=16, H_v=32, D=128, state_std=0.02, seed=2),
    "decode_sweep": dict(kind="decode", batches=(1, 8, 256, 1024), steps=100, H_qk=16, H_v=32,
                         D=128, state_std=0.02, seed=3),
    "prefill_varlen16": dict(kind="prefill", N=16, len_lo=128, len_hi=2048, H_qk=16, H_v=32,
                             D=128, chunk=64, state_std=None, seed=4),
    "prefill_long2x64k": dict(kind="prefill", N=2, len=65536, H_qk=16, H_v=32, D=128, chunk=64,
                              state_std=0.02, seed=5),
    # a multi-token decode step: 64 sequences with 4 new tokens each, states in place
    "decode_multitoken": dict(kind="prefill", N=64, len=4, H_qk=16, H_v=32, D=128, chunk=64,
                              state_std=0.02, seed=6),
}


def to_torch(x: Optional[np.ndarray], device=None, bf16: bool = False):
    """numpy -> torch on ``device``; uint16 bf16 bit patterns become torch.bfloat16."""
    import torch

    if x is None:
        return None
    if bf16:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(device) if device is not None else t
