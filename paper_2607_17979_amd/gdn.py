"""Thin ctypes binding of the C ABI in ``include/gdn.h``.

The functions carry the C names and only marshal arguments: they check dtype,
shape, contiguity and device of the torch tensors, pass raw device pointers and
the current HIP stream, and turn a non-zero status into an exception.  Every
step of the computation runs in the HIP kernels of ``libgdn_mi355x.so``; there
is no fallback of any kind: if the library is missing, calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

from .build import LIB_PATH

__all__ = [
    "GdnError",
    "load_library",
    "gdn_last_error",
    "gdn_abi_version",
    "gdn_decode",
    "gdn_decode_indexed",
    "gdn_prefill_workspace_size",
    "gdn_prefill_varlen",
    "gdn_prefill_varlen_indexed",
    "gdn_decode_multitoken",
    "gdn_prefill_varlen_noalloc",
    "gdn_decode_ex",
    "gdn_prefill_varlen_ex",
    "GDN_QK_L2NORM",
    "GDN_GATE_LOGITS",
    "GDN_SHORT_ONLY",
    "workspace_fault",
    "EXPORTED_SYMBOLS",
]

EXPORTED_SYMBOLS = ("gdn_last_error", "gdn_abi_version", "gdn_decode", "gdn_decode_indexed",
                    "gdn_prefill_workspace_size", "gdn_prefill_varlen", "gdn_prefill_varlen_indexed",
                    "gdn_decode_multitoken", "gdn_prefill_varlen_noalloc", "gdn_decode_ex",
                    "gdn_prefill_varlen_ex")

# flag bits of the _ex entry points (enum gdn_flags in include/gdn.h)
GDN_QK_L2NORM = 1
GDN_GATE_LOGITS = 2
GDN_SHORT_ONLY = 4

_STATUS = {0: "GDN_OK", -1: "GDN_EINVAL", -2: "GDN_EUNSUPPORTED", -3: "GDN_EALIGN",
           -4: "GDN_EWORKSPACE", -5: "GDN_EHIP"}


class GdnError(RuntimeError):
    """A non-zero status from the library; ``status`` holds the code."""

    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load (once) and return the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"HIP library {p} is missing; build it with "
                           "`python -m paper_2607_17979_amd.build`")
    lib = ctypes.CDLL(p)
    vp, ci, cf, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.gdn_last_error.restype = ctypes.c_char_p
    lib.gdn_last_error.argtypes = []
    lib.gdn_abi_version.restype = ci
    lib.gdn_abi_version.argtypes = []
    lib.gdn_decode.restype = ci
    lib.gdn_decode.argtypes = [vp, vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, cf, vp]
    lib.gdn_decode_indexed.restype = ci
    lib.gdn_decode_indexed.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, cf, vp]
    lib.gdn_prefill_workspace_size.restype = sz
    lib.gdn_prefill_workspace_size.argtypes = [ci, ci, ci, ci, ci, ci]
    lib.gdn_prefill_varlen.restype = ci
    lib.gdn_prefill_varlen.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                       ci, ci, ci, ci, ci, ci, ci, cf, vp, sz, vp]
    lib.gdn_prefill_varlen_indexed.restype = ci
    lib.gdn_prefill_varlen_indexed.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                               ci, ci, ci, ci, ci, ci, ci, ci, cf, vp, sz, vp]
    lib.gdn_prefill_varlen_noalloc.restype = ci
    lib.gdn_prefill_varlen_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                               ci, ci, ci, ci, ci, ci, ci, cf, vp]
    lib.gdn_decode_ex.restype = ci
    lib.gdn_decode_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp, ci, vp, ci, ci, ci, ci, ci, cf, ci, vp]
    lib.gdn_prefill_varlen_ex.restype = ci
    lib.gdn_prefill_varlen_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, ci, vp,
                                          ci, ci, ci, ci, ci, ci, ci, cf, ci, vp, sz, vp]
    lib.gdn_decode_multitoken.restype = ci
    lib.gdn_decode_multitoken.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp,
                                          ci, ci, ci, ci, ci, ci, cf, vp, sz, vp]
    if path is None:
        _lib = lib
    return lib


def gdn_last_error() -> str:
    return load_library().gdn_last_error().decode()


def gdn_abi_version() -> int:
    return load_library().gdn_abi_version()


def _check(status: int) -> None:
    if status != 0:
        raise GdnError(status, gdn_last_error())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(t, stream) -> Optional[int]:
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(t.device)
    return getattr(stream, "cuda_stream", stream)


def _torch_stream(t, stream):
    """The launch stream as a torch stream object (a raw hipStream_t handle is
    wrapped, not adopted)."""
    import torch

    if stream is None:
        return torch.cuda.current_stream(t.device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=t.device)


def _workspace_for(t, need, workspace, stream):
    """The caller's workspace, or a new one allocated on the launch stream, so
    that torch's caching allocator does not hand its memory to other work
    while the kernels of this call may still use it."""
    import torch

    if workspace is not None:
        return workspace
    with torch.cuda.stream(_torch_stream(t, stream)):
        return torch.empty(max(need, 256), dtype=torch.uint8, device=t.device)


def workspace_fault(workspace, N: int) -> int:
    """The wait-fault word of a prefill workspace after the call that used it
    has completed (synchronises the device): 0, or bit 0 set if a wave of the
    chunk kernel gave up a bounded wait (results invalid), bit 1 set if
    gdn_decode_multitoken met a sequence longer than 8 tokens, bit 2 set if
    cu_seqlens was malformed (results meaningless; no access went outside the
    T tokens)."""
    import torch

    torch.cuda.synchronize(workspace.device)
    return int(workspace.view(torch.int32)[N + 1].item())


def _need(t, name, dtype, shape, device):
    import torch

    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")


def gdn_decode(q, k, v, g, beta, state, o, scale: float = 1.0, stream=None) -> None:
    """One decode step (see include/gdn.h).  q, k: bf16 [B, H_qk, D]; v: bf16
    [B, H_v, D]; g, beta: fp32 [B, H_v]; state: fp32 [B, H_v, D, D], updated in
    place; o: bf16 [B, H_v, D], written.  Asynchronous on ``stream`` (default:
    torch's current stream of the tensors' device)."""
    import torch

    B, H_qk, D = q.shape
    H_v = v.shape[1]
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (B, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (B, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (B, H_v, D), dev)
    _need(g, "g", torch.float32, (B, H_v), dev)
    _need(beta, "beta", torch.float32, (B, H_v), dev)
    _need(state, "state", torch.float32, (B, H_v, D, D), dev)
    _need(o, "o", torch.bfloat16, (B, H_v, D), dev)
    lib = load_library()
    _check(lib.gdn_decode(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(state), _ptr(o),
                          B, H_qk, H_v, D, D, float(scale), _stream(q, stream)))


def gdn_decode_indexed(q, k, v, g, beta, state_pool, state_idx, o, scale: float = 1.0,
                       stream=None) -> None:
    """One decode step on pooled states (see include/gdn.h).  As gdn_decode,
    with state_pool: fp32 [P, H_v, D, D] and state_idx: int32 [B] on the
    device (slot of each batch entry; entries outside [0, P) are skipped)."""
    import torch

    B, H_qk, D = q.shape
    H_v = v.shape[1]
    P = state_pool.shape[0]
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (B, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (B, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (B, H_v, D), dev)
    _need(g, "g", torch.float32, (B, H_v), dev)
    _need(beta, "beta", torch.float32, (B, H_v), dev)
    _need(state_pool, "state_pool", torch.float32, (P, H_v, D, D), dev)
    _need(state_idx, "state_idx", torch.int32, (B,), dev)
    _need(o, "o", torch.bfloat16, (B, H_v, D), dev)
    lib = load_library()
    _check(lib.gdn_decode_indexed(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(state_pool),
                                  _ptr(state_idx), _ptr(o), B, P, H_qk, H_v, D, D, float(scale),
                                  _stream(q, stream)))


def gdn_prefill_workspace_size(N: int, T: int, H_v: int, D_k: int, D_v: int, chunk: int) -> int:
    return int(load_library().gdn_prefill_workspace_size(N, T, H_v, D_k, D_v, chunk))


def default_chunk(D: int) -> int:
    return 16 if D == 16 else 64


def gdn_prefill_varlen(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o,
                       scale: float = 1.0, chunk: Optional[int] = None, workspace=None,
                       stream=None):
    """Packed varlen prefill (see include/gdn.h).  q, k: bf16 [T, H_qk, D]; v:
    bf16 [T, H_v, D]; g, beta: fp32 [T, H_v]; cu_seqlens: int32 [N + 1] on the
    device; initial_state: fp32 [N, H_v, D, D] or None; final_state: fp32
    [N, H_v, D, D] (may be initial_state); o: bf16 [T, H_v, D].  ``workspace``
    (uint8, at least gdn_prefill_workspace_size bytes) is allocated with torch
    when omitted, on the launch stream.  Returns the workspace (its int32 word
    N + 1 is the wait-fault word, see ``workspace_fault``)."""
    import torch

    T, H_qk, D = q.shape
    H_v = v.shape[1]
    N = cu_seqlens.shape[0] - 1
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (T, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (T, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (T, H_v, D), dev)
    _need(g, "g", torch.float32, (T, H_v), dev)
    _need(beta, "beta", torch.float32, (T, H_v), dev)
    _need(cu_seqlens, "cu_seqlens", torch.int32, (N + 1,), dev)
    if initial_state is not None:
        _need(initial_state, "initial_state", torch.float32, (N, H_v, D, D), dev)
    _need(final_state, "final_state", torch.float32, (N, H_v, D, D), dev)
    _need(o, "o", torch.bfloat16, (T, H_v, D), dev)
    chunk = default_chunk(D) if chunk is None else chunk
    need = gdn_prefill_workspace_size(N, T, H_v, D, D, chunk)
    workspace = _workspace_for(q, need, workspace, stream)
    lib = load_library()
    _check(lib.gdn_prefill_varlen(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                  _ptr(cu_seqlens), _ptr(initial_state), _ptr(final_state),
                                  _ptr(o), N, T, H_qk, H_v, D, D, chunk, float(scale),
                                  _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(q, stream)))
    return workspace


def gdn_prefill_varlen_indexed(q, k, v, g, beta, cu_seqlens, state_pool, state_idx, o,
                               scale: float = 1.0, chunk: Optional[int] = None, workspace=None,
                               stream=None):
    """Packed varlen prefill on pooled states (see include/gdn.h).  As
    gdn_prefill_varlen, with state_pool: fp32 [P, H_v, D, D] (sequence n starts
    from slot state_idx[n] and leaves its final state there) and state_idx:
    int32 [N] on the device (entries outside [0, P) skip the sequence)."""
    import torch

    T, H_qk, D = q.shape
    H_v = v.shape[1]
    N = cu_seqlens.shape[0] - 1
    P = state_pool.shape[0]
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (T, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (T, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (T, H_v, D), dev)
    _need(g, "g", torch.float32, (T, H_v), dev)
    _need(beta, "beta", torch.float32, (T, H_v), dev)
    _need(cu_seqlens, "cu_seqlens", torch.int32, (N + 1,), dev)
    _need(state_pool, "state_pool", torch.float32, (P, H_v, D, D), dev)
    _need(state_idx, "state_idx", torch.int32, (N,), dev)
    _need(o, "o", torch.bfloat16, (T, H_v, D), dev)
    chunk = default_chunk(D) if chunk is None else chunk
    need = gdn_prefill_workspace_size(N, T, H_v, D, D, chunk)
    workspace = _workspace_for(q, need, workspace, stream)
    lib = load_library()
    _check(lib.gdn_prefill_varlen_indexed(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                          _ptr(cu_seqlens), _ptr(state_pool), _ptr(state_idx),
                                          _ptr(o), N, T, P, H_qk, H_v, D, D, chunk, float(scale),
                                          _ptr(workspace), workspace.numel() * workspace.element_size(),
                                          _stream(q, stream)))
    return workspace


def gdn_decode_multitoken(q, k, v, g, beta, cu_seqlens, state, o, scale: float = 1.0,
                          workspace=None, stream=None):
    """Decode step of at most 8 new tokens per sequence, state in place (see
    include/gdn.h).  q, k: bf16 [T, H_qk, 128]; v: bf16 [T, H_v, 128]; g, beta:
    fp32 [T, H_v]; cu_seqlens: int32 [N + 1] on the device; state: fp32
    [N, H_v, 128, 128]; o: bf16 [T, H_v, 128].  ``workspace`` (uint8, at least
    gdn_prefill_workspace_size bytes) is allocated with torch on the launch
    stream when omitted.  Returns the workspace."""
    import torch

    T, H_qk, D = q.shape
    H_v = v.shape[1]
    N = cu_seqlens.shape[0] - 1
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (T, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (T, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (T, H_v, D), dev)
    _need(g, "g", torch.float32, (T, H_v), dev)
    _need(beta, "beta", torch.float32, (T, H_v), dev)
    _need(cu_seqlens, "cu_seqlens", torch.int32, (N + 1,), dev)
    _need(state, "state", torch.float32, (N, H_v, D, D), dev)
    _need(o, "o", torch.bfloat16, (T, H_v, D), dev)
    need = gdn_prefill_workspace_size(N, T, H_v, D, D, default_chunk(D))
    workspace = _workspace_for(q, need, workspace, stream)
    lib = load_library()
    _check(lib.gdn_decode_multitoken(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(cu_seqlens),
                                     _ptr(state), _ptr(o), N, T, H_qk, H_v, D, D, float(scale),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(q, stream)))
    return workspace


def gdn_prefill_varlen_noalloc(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o,
                               scale: float = 1.0, chunk: Optional[int] = None, stream=None) -> None:
    """gdn_prefill_varlen without a workspace argument (see include/gdn.h): the
    library's static per-GPU scratch serves instead, nothing is allocated, N
    is at most 16,384; calls must not overlap in time on one GPU."""
    import torch

    T, H_qk, D = q.shape
    H_v = v.shape[1]
    N = cu_seqlens.shape[0] - 1
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (T, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (T, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (T, H_v, D), dev)
    _need(g, "g", torch.float32, (T, H_v), dev)
    _need(beta, "beta", torch.float32, (T, H_v), dev)
    _need(cu_seqlens, "cu_seqlens", torch.int32, (N + 1,), dev)
    if initial_state is not None:
        _need(initial_state, "initial_state", torch.float32, (N, H_v, D, D), dev)
    _need(final_state, "final_state", torch.float32, (N, H_v, D, D), dev)
    _need(o, "o", torch.bfloat16, (T, H_v, D), dev)
    chunk = default_chunk(D) if chunk is None else chunk
    lib = load_library()
    _check(lib.gdn_prefill_varlen_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                          _ptr(cu_seqlens), _ptr(initial_state), _ptr(final_state),
                                          _ptr(o), N, T, H_qk, H_v, D, D, chunk, float(scale),
                                          _stream(q, stream)))


def gdn_decode_ex(q, k, v, g, beta, state, o, state_idx=None, flags: int = 0, scale: float = 1.0,
                  stream=None) -> None:
    """gdn_decode / gdn_decode_indexed with the fused input prologue (see
    include/gdn.h): ``flags`` GDN_QK_L2NORM (q, k normalised in the kernel)
    and/or GDN_GATE_LOGITS (g, beta hold logits).  ``state_idx`` (int32 [B])
    makes ``state`` a pool of slots."""
    import torch

    B, H_qk, D = q.shape
    H_v = v.shape[1]
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (B, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (B, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (B, H_v, D), dev)
    _need(g, "g", torch.float32, (B, H_v), dev)
    _need(beta, "beta", torch.float32, (B, H_v), dev)
    P = 0
    if state_idx is None:
        _need(state, "state", torch.float32, (B, H_v, D, D), dev)
    else:
        P = state.shape[0]
        _need(state, "state", torch.float32, (P, H_v, D, D), dev)
        _need(state_idx, "state_idx", torch.int32, (B,), dev)
    _need(o, "o", torch.bfloat16, (B, H_v, D), dev)
    lib = load_library()
    _check(lib.gdn_decode_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(state), _ptr(state_idx),
                             P, _ptr(o), B, H_qk, H_v, D, D, float(scale), int(flags), _stream(q, stream)))


def gdn_prefill_varlen_ex(q, k, v, g, beta, cu_seqlens, initial_state, final_state, o, state_idx=None,
                          flags: int = 0, scale: float = 1.0, chunk: Optional[int] = None, workspace=None,
                          stream=None):
    """gdn_prefill_varlen / gdn_prefill_varlen_indexed / gdn_decode_multitoken
    with the fused input prologue (see include/gdn.h).  ``state_idx`` (int32
    [N]) makes ``final_state`` a pool of slots updated in place;
    GDN_SHORT_ONLY in ``flags`` takes the multi-token decode route.  Returns
    the workspace."""
    import torch

    T, H_qk, D = q.shape
    H_v = v.shape[1]
    N = cu_seqlens.shape[0] - 1
    dev = q.device
    if dev.type != "cuda":
        raise ValueError("tensors must be on a GPU device")
    _need(q, "q", torch.bfloat16, (T, H_qk, D), dev)
    _need(k, "k", torch.bfloat16, (T, H_qk, D), dev)
    _need(v, "v", torch.bfloat16, (T, H_v, D), dev)
    _need(g, "g", torch.float32, (T, H_v), dev)
    _need(beta, "beta", torch.float32, (T, H_v), dev)
    _need(cu_seqlens, "cu_seqlens", torch.int32, (N + 1,), dev)
    P = 0
    if state_idx is None:
        if initial_state is not None:
            _need(initial_state, "initial_state", torch.float32, (N, H_v, D, D), dev)
        _need(final_state, "final_state", torch.float32, (N, H_v, D, D), dev)
    else:
        P = final_state.shape[0]
        _need(final_state, "final_state", torch.float32, (P, H_v, D, D), dev)
        _need(state_idx, "state_idx", torch.int32, (N,), dev)
    _need(o, "o", torch.bfloat16, (T, H_v, D), dev)
    chunk = default_chunk(D) if chunk is None else chunk
    need = gdn_prefill_workspace_size(N, T, H_v, D, D, chunk)
    workspace = _workspace_for(q, need, workspace, stream)
    lib = load_library()
    _check(lib.gdn_prefill_varlen_ex(_ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), _ptr(cu_seqlens),
                                     _ptr(initial_state), _ptr(final_state), _ptr(state_idx), P, _ptr(o),
                                     N, T, H_qk, H_v, D, D, chunk, float(scale), int(flags),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(q, stream)))
    return workspace
