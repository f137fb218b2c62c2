"""Host logic under the address and undefined-behaviour sanitizers (CPU only).

1. The C ABI layer (csrc/gdn_api.cpp) built for the host with the sanitizers,
   its launchers replaced by stubs: every argument-check case of
   test_abi_host.py runs through it and must give the same status and message,
   calls that pass the checks must reach a launch stub, rejected ones must not.
2. The kernels' work-walk index arithmetic (csrc/gdn_index.h: the
   token-by-token unit walk, the longest-first schedule, the chunk kernel's
   item walk, logical_item) built for the host with the sanitizers and
   enumerated over random batches, compared with an independent enumeration
   written here, including a reconstruction of an earlier form of the unit
   walk (one function that scanned for the next unit and returned all of its
   fields), which must agree as well.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import test_abi_host as abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_17979_amd", "csrc")
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _build(out, *srcs):
    # sanitizer flags for the host compiler only (the device pass is not instrumented)
    cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, *srcs, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return str(out)


@pytest.fixture(scope="module")
def bins(tmp_path_factory):
    if not os.path.exists(HIPCC) or shutil.which("nm") is None:
        pytest.skip("hipcc not available")
    d = tmp_path_factory.mktemp("san")
    return dict(
        abi=_build(d / "abi_driver", os.path.join(SAN, "abi_driver.cpp"), os.path.join(SAN, "launch_stub.cpp"),
                   os.path.join(CSRC, "gdn_api.cpp")),
        walk=_build(d / "walk_check", os.path.join(SAN, "walk_check.cpp")))


def _run(exe, text):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], input=text, capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, f"sanitizer run failed ({r.returncode}):\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    return r.stdout


class _Recorder:
    """Stands in for the ctypes library: records the call the test helper makes."""

    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        def call(*args):
            self.calls.append((name, args))
            return 0
        return call


def _line(name, args):
    out = [name]
    for a in args:
        out.append("0" if a is None else (repr(float(a)) if isinstance(a, float) else str(int(a))))
    return " ".join(out)


def _cases():
    """(call line, expected status, expected message fragment) for every case
    of test_abi_host.py, plus calls that pass the checks."""
    tables = [(abi.decode, abi.test_decode_rejects), (abi.decode_indexed, abi.test_decode_indexed_rejects),
              (abi.prefill, abi.test_prefill_rejects), (abi.prefill_indexed, abi.test_prefill_indexed_rejects),
              (abi.multitoken, abi.test_decode_multitoken_rejects), (abi.decode_ex, abi.test_decode_ex_rejects),
              (abi.prefill_ex, abi.test_prefill_ex_rejects)]
    cases = []
    for helper, test in tables:
        params = [m for m in test.pytestmark if m.name == "parametrize"][0].args[1]
        for kw, status, msg in params:
            rec = _Recorder()
            helper(rec, **kw)
            cases.append((_line(*rec.calls[0]), status, msg, False))
        rec = _Recorder()
        helper(rec)  # defaults pass every check
        cases.append((_line(*rec.calls[0]), abi.OK, "", True))
    # the no-allocation entry point: its checks only (its launch needs a GPU)
    params = [m for m in abi.test_prefill_noalloc_rejects.pytestmark if m.name == "parametrize"][0].args[1]
    for kw, status, msg in params:
        rec = _Recorder()
        abi.noalloc(rec, **kw)
        cases.append((_line(*rec.calls[0]), status, msg, False))
    for kw in (dict(q=None, k=None, v=None, g=None, beta=None, state=None, o=None, B=0),):
        rec = _Recorder()
        abi.decode(rec, **kw)
        cases.append((_line(*rec.calls[0]), abi.OK, "", False))
    return cases


def test_abi_checks_under_sanitizers(bins):
    cases = _cases()
    out = _run(bins["abi"], "\n".join(c[0] for c in cases) + "\n").splitlines()
    assert len(out) == len(cases)
    for (line, status, msg, launches), got in zip(cases, out):
        st, nl, err = got.split("\t", 2)
        assert int(st) == status, (line, got)
        assert msg in err, (line, got)
        assert int(nl) == (1 if launches else 0), (line, got)


def test_workspace_size_under_sanitizers(bins):
    lines = ["gdn_prefill_workspace_size 3 10 2 128 128 64", "gdn_prefill_workspace_size 100 10 2 128 128 64",
             "gdn_prefill_workspace_size -1 10 2 128 128 64", "gdn_prefill_workspace_size 3 10 0 128 128 64",
             "gdn_prefill_workspace_size 3 10 2 16 16 16", "gdn_prefill_workspace_size 2147483000 1 1 128 128 64"]
    got = [int(x.split("\t")[0]) for x in _run(bins["abi"], "\n".join(lines) + "\n").splitlines()]
    assert got[:5] == [256, 512, 0, 0, 256]
    assert got[5] == ((2147483000 + 2) * 4 + 255) // 256 * 256


def _slot_unit(s, units, grp):
    """Slot -> unit of the token-by-token walk: in each full block of 8 grp
    slots, slots c, c + 8, c + 16, ... (one XCD) hold the grp units of one q/k
    head; a last partial block is the identity."""
    blk, r = divmod(s, 8 * grp)
    if (blk + 1) * 8 * grp > units:
        return s
    return blk * 8 * grp + grp * (r % 8) + r // 8


def _expected_recur(N, H_qk, H_v, P, grid, lengths, idx):
    """The unit walk of the token-by-token kernel, enumerated directly:
    workgroup b >= 1 visits slots b - 1, b - 1 + (grid - 1), ..., slot s holds
    unit u = _slot_unit(s), and units are (sequence n, head h, row block blk) =
    u // (4 H_v), (u // 4) % H_v, u % 4; only units whose sequence has at most
    8 tokens and whose slot is in the pool run."""
    cu = np.concatenate([[0], np.cumsum(lengths)])
    units, stride, r = N * H_v * 4, grid - 1, H_v // H_qk
    out = []
    for b in range(1, grid):
        for s in range(b - 1, units, stride):
            u = _slot_unit(s, units, r * 4)
            n, h, blk = u // (4 * H_v), (u // 4) % H_v, u % 4
            if lengths[n] > 8:
                continue
            if idx is not None and not (0 <= idx[n] < P):
                continue
            shead = (idx[n] if idx is not None else n) * H_v + h
            out.append((b, u, h, h // r, blk, shead, int(cu[n]), int(lengths[n])))
    return out


@pytest.mark.parametrize("seed", range(12))
def test_work_walks_under_sanitizers(bins, seed):
    rng = np.random.default_rng(1000 + seed)
    N = int(rng.integers(1, 40)) if seed < 10 else 4100 + seed
    H_qk = int(rng.choice([1, 2, 4]))
    H_v = H_qk * int(rng.choice([1, 2, 4]))
    P = N + int(rng.integers(0, 20))
    use_idx = bool(seed % 2)
    lengths = rng.integers(0, 150, size=N) * (rng.random(N) < 0.7) + rng.integers(0, 9, size=N)
    idx = None
    if use_idx:
        idx = rng.permutation(P)[:N].astype(np.int64)
        idx[rng.random(N) < 0.15] = -1
        idx[rng.random(N) < 0.05] = P + 3
    grid_recur = 1 + int(rng.integers(1, 50))
    vsplit = int(rng.choice([1, 2, 4]))
    items = N * H_v * vsplit
    grid_pipe = int(min(items, rng.integers(1, 300)))
    text = f"{N} {H_qk} {H_v} {P} {grid_recur} {grid_pipe} {vsplit} {int(use_idx)}\n"
    text += " ".join(map(str, lengths)) + "\n"
    if use_idx:
        text += " ".join(map(str, idx)) + "\n"
    lines = _run(bins["walk"], text).splitlines()
    rows = {}
    for ln in lines:
        f = ln.split()
        rows.setdefault(f[0], []).append(tuple(int(x) for x in f[1:]))
    expect = _expected_recur(N, H_qk, H_v, P, grid_recur, lengths, idx)
    assert rows.get("recur", []) == expect
    assert rows.get("legacy", []) == expect
    # schedule: longest first, ties by index; the given order beyond 4,096
    order = [r[1] for r in rows["order"]]
    want = list(range(N)) if N > 4096 else sorted(range(N), key=lambda i: (-lengths[i], i))
    assert order == want
    # chunk-kernel items: each (rank, head, value block) exactly once, with its fields
    cu = np.concatenate([[0], np.cumsum(lengths)])
    seen = sorted(r[2] for r in rows["pipe"])
    assert seen == list(range(items))
    for b, pss, item, n, h, vb, nch, slot, beg, ln in rows["pipe"]:
        rank, rest = divmod(item, H_v * vsplit)
        assert (n, h, vb) == (want[rank], rest // vsplit, rest % vsplit)
        assert (beg, ln) == (int(cu[n]), int(lengths[n]))
        ok_slot = idx is None or 0 <= idx[n] < P
        assert nch == ((ln + 63) // 64 if (ln > 8 and ok_slot) else 0)
        assert slot == (n if idx is None else idx[n])
    # the slot -> unit map is a bijection, and each workgroup's units of one
    # q/k head sit on one XCD when the stride is a multiple of 8
    for units in (1, 7, 31, 32, 33, 64, 100, 257, 1024):
        for grp in (4, 8, 16):
            assert sorted(_slot_unit(s, units, grp) for s in range(units)) == list(range(units))
            full = units // (8 * grp) * 8 * grp
            xcd = {}
            for s in range(full):
                xcd.setdefault(_slot_unit(s, units, grp) // grp, set()).add(s % 8)
            assert all(len(v) == 1 for v in xcd.values())
    # logical_item is a bijection of [0, total)
    for key in ("logical2", "logical8"):
        by_total = {}
        for total, bid, item in rows[key]:
            by_total.setdefault(total, []).append(item)
        for total, its in by_total.items():
            assert sorted(its) == list(range(total)), (key, total)


@pytest.mark.parametrize("seed", range(6))
def test_malformed_cu_seqlens_stays_in_bounds(bins, seed):
    """Every kernel takes a sequence's tokens from seq_span: for any cu_seqlens,
    valid or not, the span lies inside [0, T), and for a valid one it is the
    plain difference; cu_seqlens_breaks flags exactly the malformed arrays (the
    kernels set bit 2 of the fault word from it).  Host build only: no GPU run
    is ever given a malformed cu_seqlens."""
    rng = np.random.default_rng(2000 + seed)
    for trial in range(40):
        N = int(rng.integers(1, 30))
        T = int(rng.integers(0, 500))
        if trial % 4 == 0:  # valid
            cut = np.sort(rng.integers(0, T + 1, size=N - 1)) if N > 1 else np.zeros(0, np.int64)
            cu = np.concatenate([[0], cut, [T]]).astype(np.int64)
        else:  # arbitrary, including negative, decreasing and past-the-end offsets
            cu = rng.integers(-50, T + 100, size=N + 1)
            if trial % 4 == 1:
                cu = np.sort(cu)
        text = "spans\n%d %d\n%s\n" % (N, T, " ".join(map(str, cu)))
        rows = {}
        for ln in _run(bins["walk"], text).splitlines():
            f = ln.split()
            rows.setdefault(f[0], []).append(tuple(int(x) for x in f[1:]))
        valid = cu[0] == 0 and cu[N] == T and bool(np.all(np.diff(cu) >= 0))
        assert (not any(b for _, b in rows["breaks"])) == valid
        for n, beg, ln in rows["span"]:
            assert 0 <= beg <= T and 0 <= ln and beg + ln <= T
            if valid:
                assert (beg, ln) == (int(cu[n]), int(cu[n + 1] - cu[n]))
