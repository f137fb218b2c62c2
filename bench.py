"""Benchmark of the Gated DeltaNet hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step of the default workload is one pass of the whole hot path over one
batch of synthetic input:
  * gdn_decode on a batch of 64 sequences (32 value heads sharing 16 q/k heads,
    d = 128, fp32 states [64, 32, 128, 128] updated in place), launched once
    for each of four independent state buffers (the decode states of four
    layers, 4 x 128 MiB, more than the 256 MB last-level cache holds), and
  * gdn_prefill_varlen on 16 packed sequences with lengths uniform in
    [128, 2048] (same heads, chunk 64, zero initial states).
Inputs are resident in HBM before timing starts.

The JSON line's ``value`` is the decode kernel's achieved HBM bandwidth
(algorithmic bytes / kernel time, HIP events on the launch stream); the
``prefill`` object carries tokens/s and MFMA utilisation.  ``roofline`` is the
decode kernel against HBM peak; ``prefill.roofline`` the prefill launch against
the bf16 MFMA peak.  Other workloads (``--workload``) print the same format.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, TFLOP/s
METRIC = "decode: achieved HBM GB/s (% peak); prefill: tokens/s and MFMA util %"


# --- algorithmic work ------------------------------------------------------------

def decode_bytes(B, H_qk, H_v, D):
    """State read + write (fp32), q/k (bf16, one read per q/k head), v and o
    (bf16), g and beta (fp32)."""
    return (2 * B * H_v * D * D * 4 + 2 * B * H_qk * D * 2 + 2 * B * H_v * D * 2
            + 2 * B * H_v * 4)


def prefill_flops(T, H_v, D, C):
    """Dense chunked-form FLOPs per token: 2 H_v (4 C D + 3 D^2) (the C x C
    products K K^T, Q K^T, T W, (M o QK^T) U and the D x D products K S^T,
    Q S^T and the state update, each counted once, no hi/lo split)."""
    return T * 2 * H_v * (4 * C * D + 3 * D * D)


def prefill_bytes(T, N, H_qk, H_v, D, init_state):
    per_tok = 2 * H_qk * D * 2 + 2 * H_v * D * 2 + 2 * H_v * 4
    st = N * H_v * D * D * 4 * (2 if init_state else 1)
    return T * per_tok + st


# --- helpers ---------------------------------------------------------------------

def measured_traffic(kernel: str):
    """HBM bytes per launch of ``kernel`` from profiles/hbm_traffic.txt (FETCH_SIZE +
    WRITE_SIZE from rocprofv3, scaled by a plain-copy calibration), or None when
    the kernel's source has changed since those counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hbm_traffic.txt")
    try:
        rec = json.load(open(path))[kernel]
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, KeyError, ValueError):
        return None
    if hashlib.sha256(src).hexdigest()[:16] != rec.get("source_sha256_16"):
        return None
    return rec.get("hbm_bytes_per_launch")


def _dev_inputs_decode(d, dev):
    from paper_2607_17979_amd.workloads import to_torch

    return dict(q=to_torch(d.q, dev, True), k=to_torch(d.k, dev, True), v=to_torch(d.v, dev, True),
                g=to_torch(d.g, dev), beta=to_torch(d.beta, dev))


def _dev_inputs_prefill(p, dev):
    from paper_2607_17979_amd.workloads import to_torch

    return dict(q=to_torch(p.q, dev, True), k=to_torch(p.k, dev, True), v=to_torch(p.v, dev, True),
                g=to_torch(p.g, dev), beta=to_torch(p.beta, dev), cu=to_torch(p.cu_seqlens, dev),
                init=to_torch(p.initial_state, dev))


class Decode:
    """``per_step`` decode launches per call, each on the next of ``nbuf`` state
    buffers (independent layers of a model), so successive launches cannot be
    served from the last-level cache and the event pair around the call
    amortises its own overhead."""

    def __init__(self, dev, B, H_qk, H_v, D, seed, nbuf, per_step=1, n_inputs=1):
        import torch
        from paper_2607_17979_amd import workloads as wl

        self.B, self.H_qk, self.H_v, self.D = B, H_qk, H_v, D
        self.host = wl.decode_inputs(seed, B, H_qk, H_v, D)
        # launch i takes input set i % n_inputs (fresh q, k, v, g, beta per step)
        self.xs = [_dev_inputs_decode(self.host, dev)] + [
            _dev_inputs_decode(wl.decode_step_inputs(seed, s, B, H_qk, H_v, D), dev)
            for s in range(1, n_inputs)]
        self.states = [wl.to_torch(self.host.state, dev) for _ in range(nbuf)]
        self.o = torch.empty((B, H_v, D), dtype=torch.bfloat16, device=dev)
        self.i = 0
        self.per_step = per_step
        self.bytes = decode_bytes(B, H_qk, H_v, D)

    def __call__(self):
        from paper_2607_17979_amd import gdn

        for _ in range(self.per_step):
            x = self.xs[self.i % len(self.xs)]
            gdn.gdn_decode(x["q"], x["k"], x["v"], x["g"], x["beta"],
                           self.states[self.i % len(self.states)], self.o)
            self.i += 1


class DecodeIndexed:
    """``per_step`` gdn_decode_indexed launches per call on a pool of
    ``nbuf`` x B slots: launch i updates the B distinct slots of index set
    i % nbuf (the index sets are disjoint shuffles of the pool), so, as for
    Decode, successive launches stream their states from HBM."""

    def __init__(self, dev, B, H_qk, H_v, D, seed, nbuf=4, per_step=4):
        import numpy as np
        import torch
        from paper_2607_17979_amd import workloads as wl

        self.B, self.H_qk, self.H_v, self.D = B, H_qk, H_v, D
        self.host = wl.decode_inputs(seed, B, H_qk, H_v, D)
        self.x = _dev_inputs_decode(self.host, dev)
        self.pool = torch.cat([wl.to_torch(self.host.state, dev) for _ in range(nbuf)])
        perm = np.random.default_rng(seed).permutation(nbuf * B).astype(np.int32)
        self.idx = [torch.as_tensor(perm[i * B:(i + 1) * B], device=dev) for i in range(nbuf)]
        self.o = torch.empty((B, H_v, D), dtype=torch.bfloat16, device=dev)
        self.i = 0
        self.per_step = per_step
        self.bytes = decode_bytes(B, H_qk, H_v, D) + 4 * B

    def __call__(self):
        from paper_2607_17979_amd import gdn

        x = self.x
        for _ in range(self.per_step):
            gdn.gdn_decode_indexed(x["q"], x["k"], x["v"], x["g"], x["beta"], self.pool,
                                   self.idx[self.i % len(self.idx)], self.o)
            self.i += 1


class MultiToken:
    """A multi-token decode step: ``N`` sequences of ``len`` new tokens each,
    states updated in place, through gdn_decode_multitoken (``via_prefill``
    False) or gdn_prefill_varlen with initial_state is final_state.
    ``per_step`` launches per call, each on the next of ``nbuf`` state
    buffers, as for Decode."""

    def __init__(self, dev, w, nbuf=4, per_step=4, via_prefill=False):
        import torch
        from paper_2607_17979_amd import gdn
        from paper_2607_17979_amd import workloads as wl

        self.N, self.Tn, self.H_qk, self.H_v, self.D = w["N"], w["len"], w["H_qk"], w["H_v"], w["D"]
        self.T = self.N * self.Tn
        self.host = wl.prefill_inputs(w["seed"], [self.Tn] * self.N, self.H_qk, self.H_v, self.D,
                                      state_std=w["state_std"])
        self.x = _dev_inputs_prefill(self.host, dev)
        self.states = [wl.to_torch(self.host.initial_state, dev) for _ in range(nbuf)]
        self.o = torch.empty((self.T, self.H_v, self.D), dtype=torch.bfloat16, device=dev)
        ws = gdn.gdn_prefill_workspace_size(self.N, self.T, self.H_v, self.D, self.D, w["chunk"])
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=dev)
        self.chunk = w["chunk"]
        self.i = 0
        self.per_step = per_step
        self.via_prefill = via_prefill
        self.bytes = prefill_bytes(self.T, self.N, self.H_qk, self.H_v, self.D, True)

    def __call__(self):
        from paper_2607_17979_amd import gdn

        x = self.x
        for _ in range(self.per_step):
            st = self.states[self.i % len(self.states)]
            if self.via_prefill:
                gdn.gdn_prefill_varlen(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], st, st, self.o,
                                       chunk=self.chunk, workspace=self.ws)
            else:
                gdn.gdn_decode_multitoken(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], st, self.o,
                                          workspace=self.ws)
            self.i += 1


class Prefill:
    def __init__(self, dev, lengths, H_qk, H_v, D, C, seed, state_std):
        import torch
        from paper_2607_17979_amd import gdn
        from paper_2607_17979_amd import workloads as wl

        self.host = wl.prefill_inputs(seed, lengths, H_qk, H_v, D, state_std=state_std)
        self.x = _dev_inputs_prefill(self.host, dev)
        N, T = len(lengths), int(sum(lengths))
        self.N, self.T, self.H_qk, self.H_v, self.D, self.C = N, T, H_qk, H_v, D, C
        self.fin = torch.empty((N, H_v, D, D), dtype=torch.float32, device=dev)
        self.o = torch.empty((T, H_v, D), dtype=torch.bfloat16, device=dev)
        ws = gdn.gdn_prefill_workspace_size(N, T, H_v, D, D, C)
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=dev)
        self.flops = prefill_flops(T, H_v, D, C)
        self.bytes = prefill_bytes(T, N, H_qk, H_v, D, state_std is not None)

    def __call__(self):
        from paper_2607_17979_amd import gdn

        x = self.x
        gdn.gdn_prefill_varlen(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu"], x["init"],
                               self.fin, self.o, chunk=self.C, workspace=self.ws)


SETTLE = {"seconds": 0.0, "steps": 0}


def _settle(parts, seconds):
    """Untimed steps for about ``seconds`` of wall time before the warm-up:
    the GPU clocks take about 20 steps of this MFMA-heavy workload to reach
    their sustained level, so a short --warmup alone would time the ramp.
    The length is reported in the JSON line (``settle``)."""
    import torch

    n, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(5):
            for p in parts:
                p()
        n += 5
        torch.cuda.synchronize()
    SETTLE["seconds"] += time.perf_counter() - t0
    SETTLE["steps"] += n


def _time_parts(parts, steps, warmup, settle_s=0.0):
    """Settle the clocks (``settle_s`` seconds of untimed steps), run
    ``warmup`` then ``steps`` steps of all parts in order; HIP event times on
    torch's current stream (the stream the library launches on) and the wall
    time of the timed steps.  With one part, one event pair brackets all timed
    steps (back-to-back launches, nothing recorded between them); with several,
    each part of each step has its own pair, so that the parts can be told
    apart.  Returns (ms_per_step, [avg ms per part])."""
    import torch

    if settle_s > 0:
        _settle(parts, settle_s)
    for _ in range(warmup):
        for p in parts:
            p()
    torch.cuda.synchronize()
    if len(parts) == 1:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record()
        for _ in range(steps):
            parts[0]()
        e1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return wall * 1e3 / steps, [e0.elapsed_time(e1) / steps]
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in parts] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        for j, p in enumerate(parts):
            evs[s][j][0].record()
            p()
            evs[s][j][1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [sum(evs[s][j][0].elapsed_time(evs[s][j][1]) for s in range(steps)) / steps
           for j in range(len(parts))]
    return wall * 1e3 / steps, per


def _time_graph(fn, launches, replays, warmup):
    """Capture ``launches`` calls of ``fn`` in one HIP graph and time ``replays``
    replays with HIP events on the replay stream; returns the median ms per
    call.  Removes the host's per-launch cost, which dominates for small decode
    batches."""
    import statistics
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(warmup):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(launches):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    ts = []
    for _ in range(replays):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return statistics.median(ts) / launches


def _host_threads():
    """(os.cpu_count(), BLAS/OpenMP threads numpy's libraries would use)."""
    try:
        from threadpoolctl import threadpool_info

        blas = max((d.get("num_threads", 1) for d in threadpool_info()), default=1)
    except Exception:  # threadpoolctl missing: report the environment's setting
        blas = int(os.environ.get("OMP_NUM_THREADS", "1") or 1)
    return os.cpu_count() or 1, blas


def _cpu_baseline_decode(dec, budget_s=10.0):
    """The fp64 oracle's decode (as it stands) timed on the host: repeated full
    calls on the same batch until about ``budget_s`` of CPU time.  The oracle
    is vectorised over all (sequence, head) units of the step by numpy; its
    einsum row dots run on one thread (numpy's einsum does not call BLAS for
    these shapes), so ``cores`` is 1."""
    import oracle.gdn_ref as ref

    h = dec.host
    n, t0 = 0, time.perf_counter()
    while True:
        ref.decode(h.q, h.k, h.v, h.g, h.beta, h.state)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    ncpu, blas = _host_threads()
    return dict(value=n * dec.bytes / el / 1e9, unit="GB/s", cores=1, host_cpus=ncpu, blas_threads=blas,
                kind="oracle",
                sample=f"{n} full decode calls of the timed batch ({dec.B} x {dec.H_v} heads), "
                       f"{el:.1f} s; numpy fp64, vectorised over the units of the step, one thread "
                       f"(host has {ncpu} CPUs)")


def _cpu_baseline_prefill(pre, budget_s=10.0):
    """The oracle's prefill on a bounded sample: whole sequences of the timed
    batch (all value heads of a sequence advance together, the oracle's token
    loop vectorised across the independent heads), longest first, until about
    ``budget_s``; tokens/s = tokens of the sequences done / seconds (units are
    independent, so time is linear in the sample)."""
    import numpy as np
    import oracle.gdn_ref as ref

    h = pre.host
    cu = h.cu_seqlens
    lens = np.diff(cu)
    order = sorted(range(pre.N), key=lambda i: -int(lens[i]))
    tokens, seqs, t0 = 0, 0, time.perf_counter()
    while True:
        n = order[seqs % pre.N]
        ref.prefill_units(h.q, h.k, h.v, h.g, h.beta, cu, [(n, hh) for hh in range(pre.H_v)],
                          h.initial_state)
        tokens += int(lens[n])
        seqs += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    ncpu, blas = _host_threads()
    return dict(value=tokens / el, unit="tokens/s", cores=1, host_cpus=ncpu, blas_threads=blas,
                kind="oracle",
                sample=f"{seqs} whole sequences ({tokens} tokens x {pre.H_v} heads, the heads of a "
                       f"sequence vectorised in numpy fp64, one thread; host has {ncpu} CPUs), {el:.1f} s")


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50, help="untimed warm-up steps")
    ap.add_argument("--settle-s", type=float, default=0.5,
                    help="seconds of untimed steps before the warm-up, so that the clocks reach their "
                         "sustained level (about 20 steps of the default workload); reported in the output")
    ap.add_argument("--workload", default="decode_b64+prefill_varlen16",
                    choices=["decode_b64+prefill_varlen16", "decode_b64", "decode_sweep",
                             "prefill_varlen16", "prefill_long2x64k", "decode_multitoken",
                             "decode_indexed", "copy_calibration"])
    ap.add_argument("--batch", type=int, default=None, help="decode_sweep: one batch size only")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU (asked for --gpus {args.gpus}); its "
              "kernels would shard by (sequence, head) across GPUs with no exchange, which is "
              "not built", file=sys.stderr)
        return 2

    import torch

    from paper_2607_17979_amd import workloads as wl
    from paper_2607_17979_amd.build import LIB_PATH

    if not os.path.exists(LIB_PATH):
        from paper_2607_17979_amd.build import build

        build()
    dev = torch.device("cuda:0")
    W = wl.WORKLOADS
    out = dict(metric=METRIC, n_gpus=1, steps=args.steps, warmup=args.warmup,
               higher_is_better=True, scaling="weak", vs_baseline=None, data="synthetic")
    print(f"# bench {args.workload}: setting up inputs", file=sys.stderr, flush=True)
    if args.workload == "copy_calibration":
        # A plain device-to-device copy of a known size: the reference for scaling
        # the FETCH_SIZE / WRITE_SIZE counters into HBM bytes.
        nbytes = 1 << 30
        src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        ms_step, per = _time_parts([lambda: dst.copy_(src)], args.steps, args.warmup)
        gbs = 2 * nbytes / (per[0] * 1e-3) / 1e9
        out.update(value=gbs, unit="GB/s", ms_per_step=ms_step, dtype="f32",
                   config=dict(workload="copy_calibration", bytes_read=nbytes, bytes_written=nbytes))
        out["settle"] = dict(seconds=round(SETTLE["seconds"], 3), steps=SETTLE["steps"])
        print(json.dumps(out), flush=True)
        return 0

    parts, names = [], []
    dec = pre = None
    if args.workload in ("decode_b64+prefill_varlen16", "decode_b64"):
        w = W["decode_b64"]
        dec = Decode(dev, w["B"], w["H_qk"], w["H_v"], w["D"], w["seed"], nbuf=4, per_step=4)
        parts.append(dec)
        names.append("decode")
    if args.workload in ("decode_b64+prefill_varlen16", "prefill_varlen16"):
        w = W["prefill_varlen16"]
        lengths = wl.varlen_lengths(w["seed"], w["N"], w["len_lo"], w["len_hi"])
        pre = Prefill(dev, lengths, w["H_qk"], w["H_v"], w["D"], w["chunk"], w["seed"], w["state_std"])
        parts.append(pre)
        names.append("prefill")
    if args.workload == "prefill_long2x64k":
        w = W["prefill_long2x64k"]
        pre = Prefill(dev, [w["len"]] * w["N"], w["H_qk"], w["H_v"], w["D"], w["chunk"], w["seed"],
                      w["state_std"])
        parts.append(pre)
        names.append("prefill")

    if args.workload == "decode_indexed":
        w = W["decode_b64"]
        di = DecodeIndexed(dev, w["B"], w["H_qk"], w["H_v"], w["D"], w["seed"])
        ms_step, per = _time_parts([di], args.steps, args.warmup, args.settle_s)
        t = per[0] * 1e-3 / di.per_step
        gbs = di.bytes / t / 1e9
        out.update(value=gbs, unit="GB/s", ms_per_step=ms_step, dtype="f32", us_per_launch=t * 1e6,
                   roofline=dict(bound="hbm", achieved=gbs, peak=HBM_PEAK_GBS, unit="GB/s",
                                 frac=gbs / HBM_PEAK_GBS, traffic=None,
                                 kernel="gdn::decode_kernel<128,1,true>", bytes_per_launch=di.bytes),
                   config=dict(workload="decode_indexed", B=di.B, pool_slots=int(di.pool.shape[0]),
                               H_qk=di.H_qk, H_v=di.H_v, d=di.D, launches_per_step=di.per_step))
        out["settle"] = dict(seconds=round(SETTLE["seconds"], 3), steps=SETTLE["steps"])
        print(json.dumps(out), flush=True)
        return 0

    if args.workload == "decode_multitoken":
        mt = MultiToken(dev, W["decode_multitoken"])
        # the same step through gdn_prefill_varlen (one more launch, which finds
        # nothing to do), timed first, for comparison
        mtp = MultiToken(dev, W["decode_multitoken"], via_prefill=True)
        _, per_p = _time_parts([mtp], args.steps, args.warmup, args.settle_s)
        ms_step, per = _time_parts([mt], args.steps, args.warmup, args.settle_s)
        t = per[0] * 1e-3 / mt.per_step
        gbs = mt.bytes / t / 1e9
        out.update(value=gbs, unit="GB/s", ms_per_step=ms_step, dtype="f32",
                   tokens_per_s=mt.T / t, us_per_launch=t * 1e6,
                   us_per_call_via_prefill_varlen=per_p[0] * 1e3 / mtp.per_step,
                   roofline=dict(bound="hbm", achieved=gbs, peak=HBM_PEAK_GBS, unit="GB/s",
                                 frac=gbs / HBM_PEAK_GBS, traffic=None,
                                 kernel="gdn::recur::prefill_recur_kernel (token by token; "
                                        "sequences of at most 8 tokens)",
                                 bytes_per_launch=mt.bytes),
                   config=dict(workload="decode_multitoken (gdn_decode_multitoken)", N=mt.N,
                               tokens_per_sequence=mt.Tn,
                               H_qk=mt.H_qk, H_v=mt.H_v, d=mt.D, state_buffers=len(mt.states),
                               launches_per_step=mt.per_step, in_place=True))
        out["settle"] = dict(seconds=round(SETTLE["seconds"], 3), steps=SETTLE["steps"])
        print(json.dumps(out), flush=True)
        return 0

    if args.workload == "decode_sweep":
        w = W["decode_sweep"]
        batches = [args.batch] if args.batch else list(w["batches"])
        lines = []
        for B in batches:
            nbuf = max(1, min(4, (512 << 20) // (B * w["H_v"] * w["D"] * w["D"] * 4)))
            d = Decode(dev, B, w["H_qk"], w["H_v"], w["D"], w["seed"] + B, nbuf=nbuf, n_inputs=8)
            # eager: one host launch per step, HIP events around each
            _, per = _time_parts([d], w["steps"], args.warmup)
            # graph: the steps captured once and replayed (the kernel without host launch cost)
            ms_graph = _time_graph(d, w["steps"], 5, args.warmup)
            gbs = d.bytes / (ms_graph * 1e-3) / 1e9
            lines.append(dict(batch=B, us_per_step=ms_graph * 1e3, GBs=gbs, frac=gbs / HBM_PEAK_GBS,
                              us_per_step_eager=per[0] * 1e3,
                              GBs_eager=d.bytes / (per[0] * 1e-3) / 1e9, state_buffers=nbuf))
            print(f"# decode B={B}: graph {ms_graph*1e3:.2f} us/step ({gbs:.1f} GB/s); "
                  f"eager {per[0]*1e3:.2f} us/step", file=sys.stderr, flush=True)
        big = lines[-1]
        out.update(value=big["GBs"], unit="GB/s", ms_per_step=big["us_per_step"] / 1e3,
                   steps=w["steps"], dtype="f32",
                   config=dict(workload=f"decode sweep, batches {batches} x {w['steps']} steps "
                                        f"(captured in a HIP graph, replayed), "
                                        f"H_v={w['H_v']}/H_qk={w['H_qk']}, d={w['D']}",
                               sweep=lines),
                   roofline=dict(bound="hbm", achieved=big["GBs"], peak=HBM_PEAK_GBS, unit="GB/s",
                                 frac=big["frac"], traffic=None))
        out["settle"] = dict(seconds=round(SETTLE["seconds"], 3), steps=SETTLE["steps"])
        print(json.dumps(out), flush=True)
        return 0

    print(f"# bench: timing {args.steps} steps after {args.warmup} warmup", file=sys.stderr, flush=True)
    ms_step, per = _time_parts(parts, args.steps, args.warmup, args.settle_s)
    times = dict(zip(names, per))
    out["ms_per_step"] = ms_step
    cfg = {}
    if dec is not None:
        times["decode"] /= dec.per_step  # per launch
        gbs = dec.bytes / (times["decode"] * 1e-3) / 1e9
        out.update(value=gbs, unit="GB/s", dtype="f32")
        out["roofline"] = dict(bound="hbm", achieved=gbs, peak=HBM_PEAK_GBS, unit="GB/s",
                               frac=gbs / HBM_PEAK_GBS, traffic=measured_traffic("decode_kernel"),
                               kernel="gdn::decode_kernel<128,1>",
                               bytes_per_launch=dec.bytes, us_per_launch=times["decode"] * 1e3)
        cfg["decode"] = dict(B=dec.B, H_qk=dec.H_qk, H_v=dec.H_v, d=dec.D, state_buffers=len(dec.states),
                             launches_per_step=dec.per_step)
    if pre is not None:
        t = times["prefill"] * 1e-3
        tflops = pre.flops / t / 1e12
        pobj = dict(tokens_per_s=pre.T / t, us_per_call=t * 1e6, tokens=pre.T, sequences=pre.N,
                    algorithmic_tflops=tflops, mfma_util=tflops / BF16_PEAK_TFLOPS,
                    hbm_GBs=pre.bytes / t / 1e9,
                    roofline=dict(bound="mfma", achieved=tflops, peak=BF16_PEAK_TFLOPS,
                                  unit="TFLOP/s", frac=tflops / BF16_PEAK_TFLOPS,
                                  traffic=measured_traffic("prefill_kernel"),
                                  kernel="gdn::pipe::prefill_pipe_kernel<NS,NVT,NO> (+ the token-by-token launch, which writes the schedule; the launcher picks the variant from N*H_v and the CU count)",
                                  flops_per_launch=pre.flops))
        out["prefill"] = pobj
        cfg["prefill"] = dict(N=pre.N, T=pre.T, H_qk=pre.H_qk, H_v=pre.H_v, d=pre.D, chunk=pre.C,
                              initial_state=pre.host.initial_state is not None)
        if dec is None:
            out.update(value=pre.T / t, unit="tokens/s", dtype="bf16-mfma/f32")
            out["roofline"] = pobj["roofline"]
    out["config"] = dict(workload=args.workload, **cfg)
    if not args.no_cpu_baseline:
        print("# bench: timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        if dec is not None:
            out["cpu_baseline"] = _cpu_baseline_decode(dec)
            if pre is not None:
                out["prefill"]["cpu_baseline"] = _cpu_baseline_prefill(pre)
        else:
            out["cpu_baseline"] = _cpu_baseline_prefill(pre)
    out["settle"] = dict(seconds=round(SETTLE["seconds"], 3), steps=SETTLE["steps"])
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
