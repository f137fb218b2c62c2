"""Helpers for the GPU parity tests: move seeded inputs to the device, call the
HIP library through its binding (the C ABI), bring results back, and measure
errors against the fp64 oracle.

Gates (from the workload statement): outputs max-abs <= 2e-2; states relative
Frobenius error <= 1e-3, taken per (sequence, value head) -- the worst unit
must pass, which is stricter than the global ratio."""
from __future__ import annotations

import sys

import numpy as np

OUT_TOL = 2e-2
STATE_TOL = 1e-3

# (test, check, what, error) of every parity check in this run, printed at the
# end of the session by the terminal-summary hook in conftest.py.
RESULTS = []


def record(check, what, err):
    import os

    test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
    RESULTS.append((test, check, what, err))


def device():
    import torch

    if not torch.cuda.is_available():
        raise RuntimeError("GPU test run without a visible GPU")
    return torch.device("cuda:0")


def note(msg: str) -> None:
    """Print and flush, so the case is named even if the next GPU step dies."""
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(x, dev, bf16=False):
    from paper_2607_17979_amd.workloads import to_torch

    return to_torch(x, dev, bf16=bf16)


def bf16_np(t) -> np.ndarray:
    """torch bf16 tensor -> numpy uint16 bit patterns (host)."""
    import torch

    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def max_abs(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref))) if got.size else 0.0


def rel_frob_units(got, ref):
    """Per-unit ||got - ref||_F / ||ref||_F over the last two axes; returns the
    array of unit errors (0 where both are zero)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.sqrt(np.sum((got - ref) ** 2, axis=(-2, -1)))
    den = np.sqrt(np.sum(ref ** 2, axis=(-2, -1)))
    out = np.where(den > 0, num / np.where(den > 0, den, 1.0), num)
    return out


def check_outputs(got_bits, ref, what=""):
    from oracle.gdn_ref import to_f64

    err = max_abs(to_f64(got_bits), ref)
    note(f"  {what} outputs max-abs {err:.3e} (gate {OUT_TOL})")
    record("outputs max-abs", what, err)
    assert err <= OUT_TOL, f"{what}: output max-abs {err:.3e} > {OUT_TOL}"
    return err


def check_states(got, ref, what=""):
    errs = rel_frob_units(got, ref)
    worst = float(np.max(errs)) if errs.size else 0.0
    glob = float(np.linalg.norm(np.asarray(got, np.float64) - ref) / max(np.linalg.norm(ref), 1e-300))
    note(f"  {what} states rel-Frobenius worst unit {worst:.3e}, global {glob:.3e} (gate {STATE_TOL})")
    record("states rel-F worst unit", what, worst)
    assert worst <= STATE_TOL, f"{what}: state rel-Frobenius {worst:.3e} > {STATE_TOL}"
    return worst
