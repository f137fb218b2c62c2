"""The C ABI on a machine without a GPU: the library loads, exports every
symbol include/gdn.h declares, and every argument check fails with its own
status and message before any HIP call (so nothing is launched)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2607_17979_amd import gdn
from paper_2607_17979_amd.build import LIB_PATH

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdn.h")

OK, EINVAL, EUNSUP, EALIGN, EWS, EHIP = 0, -1, -2, -3, -4, -5
P = 0x10000  # a fake, 256-byte aligned "device" address: never dereferenced


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"GDN_API\s+[\w\s\*]+?\b(gdn_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return gdn.load_library()


def test_header_declares_the_bound_symbols():
    assert declared_symbols() == sorted(gdn.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    gdn_exported = {s for s in exported if s.startswith("gdn_")}
    assert gdn_exported == set(declared_symbols())


def test_abi_version(lib):
    assert lib.gdn_abi_version() == 210


def decode(lib, q=P, k=P, v=P, g=P, beta=P, state=P, o=P, B=2, H_qk=1, H_v=2, Dk=128, Dv=128,
           scale=1.0):
    return lib.gdn_decode(q, k, v, g, beta, state, o, B, H_qk, H_v, Dk, Dv, scale, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(B=-1), EINVAL, "B must be"),
    (dict(H_qk=0), EINVAL, "head counts"),
    (dict(H_qk=3, H_v=4), EINVAL, "multiple"),
    (dict(Dk=64, Dv=64), EUNSUP, "head dim"),
    (dict(Dk=128, Dv=16), EUNSUP, "must equal"),
    (dict(q=None), EINVAL, "q is NULL"),
    (dict(state=None), EINVAL, "state is NULL"),
    (dict(o=P + 8), EALIGN, "o is not 16-byte"),
    (dict(state=P + 4), EALIGN, "state is not 16-byte"),
    (dict(g=P + 2), EALIGN, "g is not 4-byte"),
])
def test_decode_rejects(lib, kw, status, msg):
    assert decode(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def test_decode_zero_batch_is_noop(lib):
    assert decode(lib, q=None, k=None, v=None, g=None, beta=None, state=None, o=None, B=0) == OK
    assert gdn.gdn_last_error() == ""


def ws_size(lib, N=3, T=10, H_v=2, D=128, chunk=64, Dv=None):
    return lib.gdn_prefill_workspace_size(N, T, H_v, D, D if Dv is None else Dv, chunk)


def test_workspace_size(lib):
    """The signature is (N, T, H_v, D_k, D_v, chunk): the schedule, the
    chunk-kernel count and the fault word, rounded up to 256 bytes."""
    assert ws_size(lib) == 256
    assert ws_size(lib, N=100) == 512
    assert ws_size(lib, N=0) == 0
    assert ws_size(lib, D=16, chunk=16) == 256
    assert ws_size(lib, chunk=16) == 0
    assert ws_size(lib, H_v=0) == 0
    assert ws_size(lib, D=128, Dv=16) == 0
    assert ws_size(lib, N=-1) == 0
    assert ws_size(lib, T=-1) == 0


def decode_indexed(lib, q=P, k=P, v=P, g=P, beta=P, pool=P, idx=P, o=P, B=2, Pn=4, H_qk=1, H_v=2,
                   Dk=128, Dv=128, scale=1.0):
    return lib.gdn_decode_indexed(q, k, v, g, beta, pool, idx, o, B, Pn, H_qk, H_v, Dk, Dv, scale, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(B=-1), EINVAL, "B must be"),
    (dict(Pn=-1), EINVAL, "P must be"),
    (dict(H_qk=3, H_v=4), EINVAL, "multiple"),
    (dict(Dk=64, Dv=64), EUNSUP, "head dim"),
    (dict(idx=None), EINVAL, "state_idx is NULL"),
    (dict(idx=P + 2), EALIGN, "state_idx"),
    (dict(pool=None), EINVAL, "state_pool is NULL"),
    (dict(pool=P + 4), EALIGN, "state_pool"),
    (dict(Pn=1 << 30), EINVAL, "P * H_v"),
    (dict(o=None), EINVAL, "o is NULL"),
])
def test_decode_indexed_rejects(lib, kw, status, msg):
    assert decode_indexed(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def test_decode_indexed_empty_is_noop(lib):
    assert decode_indexed(lib, q=None, k=None, v=None, g=None, beta=None, pool=None, idx=None, o=None,
                          B=0) == OK
    assert decode_indexed(lib, pool=None, idx=None, Pn=0) == OK


def prefill(lib, q=P, k=P, v=P, g=P, beta=P, cu=P, init=None, fin=P, o=P, N=3, T=10, H_qk=1,
            H_v=2, Dk=128, Dv=128, chunk=64, ws=P, ws_bytes=256):
    return lib.gdn_prefill_varlen(q, k, v, g, beta, cu, init, fin, o, N, T, H_qk, H_v, Dk, Dv,
                                  chunk, 1.0, ws, ws_bytes, None)


STATE_BYTES = 3 * 2 * 128 * 128 * 4


@pytest.mark.parametrize("kw,status,msg", [
    (dict(N=-1), EINVAL, "must be >= 0"),
    (dict(T=-5), EINVAL, "must be >= 0"),
    (dict(H_qk=2, H_v=3), EINVAL, "multiple"),
    (dict(Dk=32, Dv=32), EUNSUP, "head dim"),
    (dict(chunk=32), EUNSUP, "chunk 32"),
    (dict(Dk=16, Dv=16, chunk=64), EUNSUP, "chunk 64"),
    (dict(cu=None), EINVAL, "cu_seqlens is NULL"),
    (dict(cu=P + 2), EALIGN, "cu_seqlens"),
    (dict(fin=None), EINVAL, "final_state is NULL"),
    (dict(init=P + 4, fin=P + 0x100000), EALIGN, "initial_state"),
    (dict(init=P, fin=P + 1024), EINVAL, "overlap"),
    (dict(init=P + 2 * STATE_BYTES, fin=P + STATE_BYTES // 2 // 16 * 16 + 2 * STATE_BYTES), EINVAL, "overlap"),
    (dict(q=None), EINVAL, "q is NULL"),
    (dict(v=P + 8), EALIGN, "v is not"),
    (dict(beta=None), EINVAL, "beta is NULL"),
    (dict(ws=None), EWS, "workspace"),
    (dict(ws_bytes=100), EWS, "256 bytes needed"),
    (dict(ws=P + 16), EALIGN, "workspace"),
    (dict(T=1 << 20, H_qk=16, H_v=32), EINVAL, "problem too large"),
])
def test_prefill_rejects(lib, kw, status, msg):
    assert prefill(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def test_prefill_zero_sequences_is_noop(lib):
    assert prefill(lib, q=None, k=None, v=None, g=None, beta=None, cu=None, fin=None, o=None,
                   N=0, T=0, ws=None, ws_bytes=0) == OK


def test_error_message_is_per_call(lib):
    assert decode(lib, B=-1) == EINVAL
    assert gdn.gdn_last_error() != ""
    assert decode(lib, q=None, k=None, v=None, g=None, beta=None, state=None, o=None, B=0) == OK
    assert gdn.gdn_last_error() == ""


def test_binding_raises_on_missing_library(tmp_path):
    with pytest.raises(RuntimeError, match="missing"):
        gdn.load_library(str(tmp_path / "nope.so"))


def prefill_indexed(lib, q=P, k=P, v=P, g=P, beta=P, cu=P, pool=P, idx=P, o=P, N=3, T=10, Pn=4,
                    H_qk=1, H_v=2, Dk=128, Dv=128, chunk=64, ws=P, ws_bytes=256):
    return lib.gdn_prefill_varlen_indexed(q, k, v, g, beta, cu, pool, idx, o, N, T, Pn, H_qk, H_v, Dk,
                                          Dv, chunk, 1.0, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(N=-1), EINVAL, "must be >= 0"),
    (dict(Pn=-1), EINVAL, "P must be"),
    (dict(H_qk=2, H_v=3), EINVAL, "multiple"),
    (dict(chunk=32), EUNSUP, "chunk 32"),
    (dict(cu=None), EINVAL, "cu_seqlens is NULL"),
    (dict(pool=None), EINVAL, "state_pool is NULL"),
    (dict(pool=P + 8), EALIGN, "state_pool"),
    (dict(idx=None), EINVAL, "state_idx is NULL"),
    (dict(idx=P + 1), EALIGN, "state_idx"),
    (dict(Pn=1 << 30), EINVAL, "P * H_v"),
    (dict(q=None), EINVAL, "q is NULL"),
    (dict(ws=None), EWS, "workspace"),
])
def test_prefill_indexed_rejects(lib, kw, status, msg):
    assert prefill_indexed(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def test_prefill_indexed_empty_is_noop(lib):
    assert prefill_indexed(lib, q=None, k=None, v=None, g=None, beta=None, cu=None, pool=None, idx=None,
                           o=None, N=0, T=0, ws=None, ws_bytes=0) == OK
    assert prefill_indexed(lib, pool=None, idx=None, Pn=0) == OK


def multitoken(lib, q=P, k=P, v=P, g=P, beta=P, cu=P, state=P, o=P, N=3, T=10, H_qk=1, H_v=2,
               Dk=128, Dv=128, ws=P, ws_bytes=256):
    return lib.gdn_decode_multitoken(q, k, v, g, beta, cu, state, o, N, T, H_qk, H_v, Dk, Dv, 1.0,
                                     ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(N=-1), EINVAL, "must be >= 0"),
    (dict(H_qk=2, H_v=3), EINVAL, "multiple"),
    (dict(Dk=16, Dv=16), EUNSUP, "head dim 128"),
    (dict(T=25), EINVAL, "more than 8 tokens"),
    (dict(cu=None), EINVAL, "cu_seqlens is NULL"),
    (dict(state=None), EINVAL, "state is NULL"),
    (dict(state=P + 8), EALIGN, "state"),
    (dict(q=None), EINVAL, "q is NULL"),
    (dict(ws=None), EWS, "workspace"),
    (dict(ws=P + 16), EALIGN, "workspace"),
])
def test_decode_multitoken_rejects(lib, kw, status, msg):
    assert multitoken(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def test_decode_multitoken_empty_is_noop(lib):
    assert multitoken(lib, q=None, k=None, v=None, g=None, beta=None, cu=None, state=None, o=None,
                      N=0, T=0, ws=None, ws_bytes=0) == OK


def noalloc(lib, q=P, k=P, v=P, g=P, beta=P, cu=P, init=None, fin=P, o=P, N=3, T=10, H_qk=1, H_v=2,
            Dk=128, Dv=128, chunk=64):
    return lib.gdn_prefill_varlen_noalloc(q, k, v, g, beta, cu, init, fin, o, N, T, H_qk, H_v, Dk, Dv,
                                          chunk, 1.0, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(N=-1), EINVAL, "must be >= 0"),
    (dict(H_qk=3, H_v=4), EINVAL, "multiple"),
    (dict(chunk=32), EUNSUP, "chunk 32"),
    (dict(cu=None), EINVAL, "cu_seqlens is NULL"),
    (dict(fin=None), EINVAL, "final_state is NULL"),
    (dict(init=P, fin=P + 1024), EINVAL, "overlap"),
    (dict(q=None), EINVAL, "q is NULL"),
    (dict(N=16385, T=16385), EWS, "16384"),
])
def test_prefill_noalloc_rejects(lib, kw, status, msg):
    """The no-allocation entry point checks its arguments as gdn_prefill_varlen
    does, and rejects more sequences than its static scratch holds, all on the
    host before any HIP call."""
    assert noalloc(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def test_prefill_noalloc_zero_sequences_is_noop(lib):
    assert noalloc(lib, q=None, k=None, v=None, g=None, beta=None, cu=None, fin=None, o=None, N=0, T=0) == OK


def decode_ex(lib, q=P, k=P, v=P, g=P, beta=P, state=P, idx=None, Pn=0, o=P, B=2, H_qk=1, H_v=2, Dk=128,
              Dv=128, scale=1.0, flags=0):
    return lib.gdn_decode_ex(q, k, v, g, beta, state, idx, Pn, o, B, H_qk, H_v, Dk, Dv, scale, flags, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(flags=4), EINVAL, "flags 0x4"),
    (dict(flags=8), EINVAL, "flags 0x8"),
    (dict(B=-1, flags=3), EINVAL, "B must be"),
    (dict(state=None, flags=1), EINVAL, "state is NULL"),
    (dict(idx=P, Pn=-1, flags=2), EINVAL, "P must be"),
    (dict(idx=P + 2, Pn=4), EALIGN, "state_idx"),
])
def test_decode_ex_rejects(lib, kw, status, msg):
    assert decode_ex(lib, **kw) == status
    assert msg in gdn.gdn_last_error()


def prefill_ex(lib, q=P, k=P, v=P, g=P, beta=P, cu=P, init=None, fin=P, idx=None, Pn=0, o=P, N=3, T=10,
               H_qk=1, H_v=2, Dk=128, Dv=128, chunk=64, flags=0, ws=P, ws_bytes=256):
    return lib.gdn_prefill_varlen_ex(q, k, v, g, beta, cu, init, fin, idx, Pn, o, N, T, H_qk, H_v, Dk, Dv, chunk,
                                     1.0, flags, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(flags=8), EINVAL, "flags 0x8"),
    (dict(idx=P, Pn=4, init=P + 0x100000), EINVAL, "in place"),
    (dict(flags=4, init=P + 0x100000), EINVAL, "in place"),
    (dict(flags=4, Dk=16, Dv=16, chunk=16), EUNSUP, "head dim 128"),
    (dict(flags=4, chunk=16), EUNSUP, "use 64"),
    (dict(flags=4, T=25), EINVAL, "more than 8 tokens"),
    (dict(flags=3, chunk=32), EUNSUP, "chunk 32"),
    (dict(idx=P + 1, Pn=4, flags=1), EALIGN, "state_idx"),
    (dict(flags=1, ws=None), EWS, "workspace"),
])
def test_prefill_ex_rejects(lib, kw, status, msg):
    assert prefill_ex(lib, **kw) == status
    assert msg in gdn.gdn_last_error()
