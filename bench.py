"""Benchmark of the MI355X row softmax: one JSON line on stdout.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload KEY]
                    [--no-cpu-baseline] [--no-extra-workloads]

A step is one softmax_fwd call (every stage of the path: load, row max,
shift, clip, exp, row sum, reciprocal scale, store) over the whole workload
matrix.  The headline workload is the long-row one, 64 x 262144 (134 MB of
traffic per call, tied with the vocabulary workload as the largest of the
five); the vocabulary workload, 512 x 32768, gets the same roofline and CPU
baseline objects under ``graded``, and the other three shapes are reported
under ``other_workloads``.  Inputs sit in HBM before the timed region starts.
Each step uses a different (x, y) pair out of a rotation set of at least
1 GiB, so no step finds its input in the 256 MB last-level (MALL) cache left
warm by earlier steps; every x_k holds the same seeded matrix.

Timing: the K steps are captured once into a HIP graph (torch.cuda.CUDAGraph)
on a dedicated stream.  After W eager warmup steps and one untimed replay,
the graph is replayed, untimed, until at least SETTLE_S seconds of GPU work
have run (the GPU's clocks drop while the host prepares each workload, and
take tens of milliseconds to come back up; a window timed right after the
preparation measured up to 10% slower), FIRST_SETTLE_S for the first
workload of the process, which starts from an idle GPU.  Then the measurement is:
synchronise; replay the graph once untimed (a pre-roll
that keeps the GPU busy while the host queues the rest); record the start
event; replay the graph (exactly K steps, with every gap between them);
record the stop event; synchronise.  Starting the event behind queued work
keeps the host's submission time of the timed replay out of the window.
The same steps launched one by one from Python, also behind a pre-roll, are
reported as ``eager``.  The roofline object uses the algorithmic traffic of
one call (8 bytes per element: one fp32 read of x, one fp32 write of y)
divided by the step time; these workloads take one launch per step.
``cpu_baseline`` times the float64 oracle on the host, ``cpu_fp32_baseline``
a plain single-thread fp32 C loop.

Counter passes (FETCH_SIZE, WRITE_SIZE, and optionally occupancy) use two
extra modes:

    rocprofv3 --pmc FETCH_SIZE -d DIR/fetch -o run -- python3 bench.py --pmc-run --workload KEY
    rocprofv3 --pmc WRITE_SIZE -d DIR/write -o run -- python3 bench.py --pmc-run --workload KEY
    rocprofv3 --pmc OccupancyPercent SQ_WAVES GRBM_GUI_ACTIVE -d DIR/occ -o run \
        -- python3 bench.py --pmc-run --workload KEY
    python3 bench.py --summarize-pmc DIR --workload KEY

The summary (profiles/pmc_KEY.json and .md) scales each counter by what it
reads for the library's copy kernel on the same number of bytes; ``traffic``
in the JSON line comes from it only while the kernel sources are unchanged.
A kernel-trace run of this script (``rocprofv3 --kernel-trace --stats``)
summarised with ``--summarize-trace`` gives profiles/trace_bench.json, whose
per-kernel median, p10 and p90 the JSON line repeats under the same rule.
"""
from __future__ import annotations

import argparse
import csv
import ctypes
import glob
import hashlib
import json
import math
import os
import platform
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, 8 TB/s
ROTATE_BYTES = 1 << 30          # >= 4x the 256 MB MALL
METRIC = "softmax rows/s and achieved HBM GB/s (% of MI355X peak), fp32, 1 GPU"
DEFAULT_WORKLOAD = "longrow_64x262144"
GRADED = ("longrow_64x262144", "vocab_512x32768")   # >= 32 MB of logits each
CSRC = os.path.join(ROOT, "paper_1904_12380_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
TRACE_JSON = os.path.join(PROFILES, "trace_bench.json")


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def kernel_source_sha256() -> str:
    """Hash of the HIP sources: counter and trace summaries are tied to it."""
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(CSRC, "*"))):
        if path.endswith((".hip", ".hpp", ".h")):
            h.update(os.path.basename(path).encode())
            with open(path, "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def machine_state() -> dict:
    """Clocks, power and performance level from rocm-smi (read-only queries),
    so that differences between machines and runs can be told apart."""
    out: dict = {}
    cmd = ["rocm-smi", "--showclocks", "--showpower", "--showmaxpower", "--showperflevel",
           "--json"]
    try:
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=30)
        doc = json.loads(r.stdout) if r.stdout.strip().startswith("{") else {}
        card = next((v for k, v in doc.items() if k.startswith("card")), {})
        keep = ("sclk", "mclk", "fclk", "socclk", "power", "perf")
        out = {k: v for k, v in card.items() if any(t in k.lower() for t in keep)}
        if not out:
            out = {"raw": r.stdout.strip()[-400:]}
    except Exception as e:  # rocm-smi missing or failed: record why
        out = {"error": repr(e)}
    return out


class Rotation:
    """K (x, y) pairs of the workload resident in HBM, at least 1 GiB."""

    def __init__(self, torch, x_host: np.ndarray):
        dev = torch.device("cuda:0")
        pair_bytes = 8 * x_host.size
        self.n = max(2, math.ceil(ROTATE_BYTES / pair_bytes))
        x0 = torch.from_numpy(x_host).to(dev)
        self.xs = [x0.clone() for _ in range(self.n)]
        self.ys = [torch.empty_like(x0) for _ in range(self.n)]

    def pair(self, i):
        return self.xs[i % self.n], self.ys[i % self.n]


def warm_clocks(sm, torch, seconds: float = 0.3) -> None:
    """Untimed: keep the GPU streaming for a moment, so that the first timed
    workload does not run while clocks are still ramping up from idle."""
    x = torch.zeros(1 << 26, device="cuda:0")      # 256 MB
    y = torch.empty_like(x)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            sm.softmax_copy_probe(x, out=y)
        torch.cuda.synchronize()
    del x, y


SETTLE_S = 0.05
# The first timed workload of the process starts from an idle GPU (sclk
# about 170 MHz before the run): it settles longer.  With 0.05 s a session
# measured the headline's graph window at 22.7 us per step against 21.9-22.1
# for the same kernel in the modes timed right after it.
FIRST_SETTLE_S = 0.5
_settled = False


def time_steps(torch, launch, steps: int, warmup: int) -> tuple[float, float]:
    """Graph-replayed and eager ms per step of launch(i, stream), each timed
    over exactly `steps` steps behind a queued pre-roll, after untimed
    replays that let the clocks settle (see the module docstring).  Returns
    (graph ms per step, eager ms per step)."""
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        for i in range(warmup):
            launch(i, stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(steps):
                launch(i, stream)
        g.replay()                  # first replay, untimed
        torch.cuda.synchronize()
        global _settled
        settle_s = SETTLE_S if _settled else FIRST_SETTLE_S
        _settled = True
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < settle_s:   # clocks settle, untimed
            for _ in range(4):
                g.replay()
            torch.cuda.synchronize()
        g.replay()                  # pre-roll, untimed
        start.record(stream)
        g.replay()                  # the timed steps
        stop.record(stream)
        torch.cuda.synchronize()
        graph_ms = start.elapsed_time(stop) / steps
        g.replay()                  # pre-roll for the eager steps
        start.record(stream)
        for i in range(steps):
            launch(i, stream)
        stop.record(stream)
        torch.cuda.synchronize()
        eager_ms = start.elapsed_time(stop) / steps
    del g
    return graph_ms, eager_ms


def time_gpu(sm, torch, w: workloads.Workload, x_host: np.ndarray, steps: int, warmup: int,
             check: bool = True, memcpy: bool = False) -> dict:
    rot = Rotation(torch, x_host)
    labels = torch.from_numpy(workloads.generate_labels(w.key)).to(rot.xs[0].device)
    losses = [torch.empty(w.rows, device=rot.xs[0].device) for _ in range(rot.n)]
    plan = sm.softmax_plan(w.rows, w.cols, rot.xs[0].data_ptr(), rot.ys[0].data_ptr())

    def fwd(i, s):
        x, y = rot.pair(i)
        sm.softmax_fwd(x, out=y, stream=s)

    def cpy(i, s):
        x, y = rot.pair(i)
        sm.softmax_copy_probe(x, out=y, stream=s)

    def cpy_inplace(i, s):
        # the copy kernel with y == x: the same read-then-write of each line
        # as an in-place softmax, with no arithmetic
        _, y = rot.pair(i)
        sm.softmax_copy_probe(y, out=y, stream=s)

    def d2d(i, s):
        x, y = rot.pair(i)
        y.copy_(x)          # hipMemcpyAsync device to device

    # The fixed cost of one launch that reads and then writes: the copy
    # kernel on 4 KiB, same stream and graph timing.
    tiny_x = torch.zeros(1024, device=rot.xs[0].device)
    tiny_y = torch.empty_like(tiny_x)

    def tiny(i, s):
        sm.softmax_copy_probe(tiny_x, out=tiny_y, stream=s)

    def fwd_inplace(i, s):
        # in place on y_k, which holds finite softmax outputs of earlier steps
        _, y = rot.pair(i)
        sm.softmax_fwd(y, out=y, stream=s)

    def fwd_noclip(i, s):
        x, y = rot.pair(i)
        sm.softmax_fwd_clip(x, float("-inf"), out=y, stream=s)

    def fwd_approx(i, s):
        x, y = rot.pair(i)
        sm.softmax_fwd_approx(x, out=y, stream=s)

    def fwd_log(i, s):
        x, y = rot.pair(i)
        sm.softmax_log_fwd(x, out=y, stream=s)

    def fwd_nll(i, s):
        x, _ = rot.pair(i)
        sm.softmax_nll_fwd(x, labels, out=losses[i % rot.n], stream=s)

    ms, eager_ms = time_steps(torch, fwd, steps, warmup)
    inplace_ms, _ = time_steps(torch, fwd_inplace, steps, warmup)
    copy_ms, _ = time_steps(torch, cpy, steps, warmup)
    copy_inplace_ms, _ = time_steps(torch, cpy_inplace, steps, warmup)
    memcpy_ms = time_steps(torch, d2d, steps, warmup)[0] if memcpy else None
    floor_ms = time_steps(torch, tiny, steps, warmup)[0] if memcpy else None
    noclip_ms, _ = time_steps(torch, fwd_noclip, steps, warmup)
    approx_ms, _ = time_steps(torch, fwd_approx, steps, warmup)
    log_ms, _ = time_steps(torch, fwd_log, steps, warmup)
    nll_ms, _ = time_steps(torch, fwd_nll, steps, warmup)
    nll_bytes = 4 * w.rows * w.cols + 12 * w.rows   # x read, labels read, losses written

    max_rel = None
    if check:
        # Re-run once on pair 0 and check sampled rows against the oracle.
        import oracle
        x0, y0 = rot.pair(0)
        sm.softmax_fwd(x0, out=y0)
        torch.cuda.synchronize()
        rng = np.random.default_rng(0)
        rows = np.unique(rng.integers(0, w.rows, size=min(w.rows, 16)))
        dev = y0.device
        y = y0[torch.from_numpy(rows).to(dev)].cpu().numpy().astype(np.float64)
        want = oracle.softmax_clipped(x_host[rows])
        max_rel = float(np.max(np.abs(y - want) / want))
        if max_rel > 4e-6:
            raise SystemExit(f"bench output failed parity on {w.key}: {max_rel:.3e}")
    nbuf = rot.n
    del rot
    torch.cuda.empty_cache()

    gbps = w.algorithmic_bytes / (ms * 1e-3) / 1e9
    return {
        "ms_per_step": ms,
        "rows_per_s": w.rows / (ms * 1e-3),
        "elements_per_s": w.elements / (ms * 1e-3),
        "hbm_gbps": gbps,
        "frac_of_peak": gbps / HBM_PEAK_GBPS,
        "eager_ms_per_step": eager_ms,
        "eager_hbm_gbps": w.algorithmic_bytes / (eager_ms * 1e-3) / 1e9,
        "in_place_ms_per_step": inplace_ms,
        "in_place_hbm_gbps": w.algorithmic_bytes / (inplace_ms * 1e-3) / 1e9,
        "copy_ms_per_step": copy_ms,
        "copy_gbps": w.algorithmic_bytes / (copy_ms * 1e-3) / 1e9,
        "copy_in_place_ms_per_step": copy_inplace_ms,
        "softmax_over_copy_time": ms / copy_ms,
        "memcpy_ms_per_step": memcpy_ms,
        "launch_floor_ms_per_step": floor_ms,
        "noclip_ms_per_step": noclip_ms,
        "noclip_hbm_gbps": w.algorithmic_bytes / (noclip_ms * 1e-3) / 1e9,
        "approx_exp_ms_per_step": approx_ms,
        "approx_exp_hbm_gbps": w.algorithmic_bytes / (approx_ms * 1e-3) / 1e9,
        "log_softmax_ms_per_step": log_ms,
        "log_softmax_hbm_gbps": w.algorithmic_bytes / (log_ms * 1e-3) / 1e9,
        "nll_ms_per_step": nll_ms,
        "nll_algorithmic_bytes": nll_bytes,
        "nll_hbm_gbps": nll_bytes / (nll_ms * 1e-3) / 1e9,
        "rotation_buffers": nbuf,
        "plan": plan,
        "sampled_max_rel_err": max_rel,
    }


FP32_MATRIX_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix-core peak


# The kernel softmax_attention_fwd runs on the DAM tile (d = dv = 200, 49 or
# 50 keys, 128-bit operands).
ATTENTION_KERNEL = "smx::k_attention_pp<4, false, 200>"


def time_attention(sm, torch, key: str, steps: int, warmup: int) -> dict:
    """The fused attention on the DAM Q, K, V: graph-replayed steps over a
    rotation of at least 1 GiB of (Q, K, V, O) sets, plus the same problem
    done unfused for comparison (hipBLAS batched products around
    softmax_fwd, with K^T made contiguous outside the timed region)."""
    wa = workloads.ATTENTION_WORKLOADS[key]
    q, k, v = workloads.generate_qkv(key)
    dev = torch.device("cuda:0")
    nset = max(2, math.ceil(ROTATE_BYTES / wa.algorithmic_bytes))
    q0, k0, v0 = (torch.from_numpy(a).to(dev) for a in (q, k, v))
    sets = [(q0.clone(), k0.clone(), v0.clone(),
             torch.empty((wa.batch, wa.lq, wa.dv), device=dev)) for _ in range(nset)]

    def fused(i, s):
        qq, kk, vv, oo = sets[i % nset]
        sm.softmax_attention_fwd(qq, kk, vv, scale=wa.scale, out=oo, stream=s)

    ms, eager_ms = time_steps(torch, fused, steps, warmup)
    # parity of the timed output on sampled batch elements
    import oracle
    torch.cuda.synchronize()
    pick = np.random.default_rng(0).choice(wa.batch, 32, replace=False)
    got = sets[0][3][torch.from_numpy(pick).to(dev)].cpu().numpy().astype(np.float64)
    want = oracle.attention_clipped(q[pick], k[pick], v[pick], wa.scale)
    err = float(np.max(np.abs(got - want)) / np.max(np.abs(want)))
    if err > 1e-4:
        raise SystemExit(f"attention output failed parity: normwise {err:.3e}")

    # unfused: S = bmm(Q, K^T) * scale, P = softmax_fwd(S), O = bmm(P, V)
    kt = [st[1].transpose(1, 2).contiguous() for st in sets]
    ss = [torch.empty((wa.batch, wa.lq, wa.lk), device=dev) for _ in range(nset)]

    def unfused(i, s):
        qq, _, vv, oo = sets[i % nset]
        sc = ss[i % nset]
        torch.bmm(qq, kt[i % nset], out=sc)
        sc.mul_(wa.scale)
        sm.softmax_fwd(sc.view(-1, wa.lk), out=sc.view(-1, wa.lk), stream=s)
        torch.bmm(sc, vv, out=oo)

    unfused_ms, _ = time_steps(torch, unfused, steps, warmup)
    del sets, kt, ss
    torch.cuda.empty_cache()
    gbps = wa.algorithmic_bytes / (ms * 1e-3) / 1e9
    tflops = wa.flops / (ms * 1e-3) / 1e12
    traffic, traffic_note = load_traffic(key)
    return {
        "workload": key, "batch": wa.batch, "lq": wa.lq, "lk": wa.lk, "d": wa.d, "dv": wa.dv,
        "ms_per_step": ms, "eager_ms_per_step": eager_ms,
        "batches_per_s": wa.batch / (ms * 1e-3),
        "algorithmic_bytes_per_launch": wa.algorithmic_bytes, "hbm_gbps": gbps,
        "frac_of_hbm_peak": gbps / HBM_PEAK_GBPS,
        "flops_per_launch": wa.flops, "tflops": tflops,
        "frac_of_fp32_matrix_peak": tflops / FP32_MATRIX_PEAK_TFLOPS,
        "unfused_ms_per_step": unfused_ms, "fused_speedup": unfused_ms / ms,
        "sampled_normwise_err": err, "rotation_sets": nset,
        "traffic": traffic,
        **({"traffic_note": traffic_note} if traffic_note else {}),
        "kernel": ATTENTION_KERNEL,
        "kernel_trace": kernel_trace_stats(ATTENTION_KERNEL, None),
    }


def time_cpu_oracle(x: np.ndarray, budget_s: float) -> dict:
    """float64 oracle (numpy, one thread) on whole passes over the matrix,
    repeated until `budget_s` of wall time is spent."""
    import oracle
    passes, t0 = 0, time.perf_counter()
    while True:
        oracle.softmax_clipped(x)
        passes += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per = el / passes
    return {"value": x.shape[0] / per, "unit": "rows/s", "cores": 1, "kind": "oracle",
            "sample": f"{passes} full passes over the {x.shape[0]}x{x.shape[1]} matrix "
                      f"({el:.1f} s), numpy float64, one thread",
            "seconds_per_pass": per, "cpu_model": cpu_model(),
            "host_cores_available": os.cpu_count()}


def time_cpu_fp32(x: np.ndarray, budget_s: float) -> dict | None:
    so = os.path.join(ROOT, "oracle", "libcpu_fp32_baseline.so")
    if not os.path.exists(so):
        return None
    lib = ctypes.CDLL(so)
    lib.cpu_softmax_fp32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_int64]
    y = np.empty_like(x)
    passes, t0 = 0, time.perf_counter()
    while True:
        lib.cpu_softmax_fp32(x.ctypes.data, y.ctypes.data, x.shape[0], x.shape[1])
        passes += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    per = el / passes
    return {"value": x.shape[0] / per, "unit": "rows/s", "cores": 1, "kind": "fp32_c_loop",
            "sample": f"{passes} full passes ({el:.1f} s), gcc -O2, one thread",
            "gbps": 8 * x.size / per / 1e9}


def pmc_summary_path(key: str, ext: str, tag: str = "") -> str:
    return os.path.join(PROFILES, f"pmc_{key}{'_' + tag if tag else ''}.{ext}")


def load_traffic(key: str) -> tuple[float | None, str | None]:
    """HBM bytes per launch from the committed counter summary, or None when
    there is none or the kernel sources changed since it was taken."""
    path = pmc_summary_path(key, "json")
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        doc = json.load(f)
    if doc.get("source_sha256") != kernel_source_sha256():
        return None, "kernel changed since the counters were taken"
    return doc["traffic_bytes_per_launch"], None


class AttentionCounters:
    """An attention workload seen by the counter passes: the copy kernel that
    calibrates the counters moves as many floats as Q, K and V hold."""

    def __init__(self, key: str):
        self.wa = workloads.ATTENTION_WORKLOADS[key]
        self.key = key
        wa = self.wa
        self.elements = wa.batch * (wa.lq * wa.d + wa.lk * wa.d + wa.lk * wa.dv)
        self.algorithmic_bytes = wa.algorithmic_bytes


def pmc_run_attention(sm, torch, wc: AttentionCounters, launches: int) -> None:
    """Launches for a counter pass on the fused attention: `launches` calls,
    then as many copy-kernel calls over the bytes of Q, K and V."""
    wa = wc.wa
    dev = torch.device("cuda:0")
    q, k, v = (torch.from_numpy(a).to(dev) for a in workloads.generate_qkv(wc.key))
    o = torch.empty((wa.batch, wa.lq, wa.dv), device=dev)
    for _ in range(launches):
        sm.softmax_attention_fwd(q, k, v, scale=wa.scale, out=o)
    torch.cuda.synchronize()
    src = torch.cat([q.reshape(-1), k.reshape(-1), v.reshape(-1)])
    dst = torch.empty_like(src)
    for _ in range(launches):
        sm.softmax_copy_probe(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"pmc_run": wc.key, "launches": launches}), flush=True)


def pmc_run(sm, torch, w: workloads.Workload, launches: int, in_place: bool = False) -> None:
    """Launches for a counter pass: `launches` softmax calls on the rotation,
    then as many copy-kernel calls over the same bytes.  With in_place, the
    softmax calls run with y == x on the rotation's y buffers, which first
    receive a copy of x (copy-kernel calls over the same bytes, so the copy
    kernel's per-dispatch counters are unchanged)."""
    rot = Rotation(torch, workloads.generate(w.key))
    if in_place:
        for i in range(rot.n):
            x, y = rot.pair(i)
            sm.softmax_copy_probe(x, out=y)
        torch.cuda.synchronize()
    for i in range(launches):
        x, y = rot.pair(i)
        if in_place:
            sm.softmax_fwd(y, out=y)
        else:
            sm.softmax_fwd(x, out=y)
    torch.cuda.synchronize()
    for i in range(launches):
        x, y = rot.pair(i)
        sm.softmax_copy_probe(x, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"pmc_run": w.key, "launches": launches}), flush=True)


def _counter_rows(directory: str):
    """(kernel name, counter name, value per dispatch) from a rocprofv3 pass:
    counter_collection.csv (--output-format csv) or the rocpd database."""
    files = glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)
    for path in files:
        with open(path) as f:
            for r in csv.DictReader(f):
                yield r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"])
    if files:
        return
    dbs = glob.glob(os.path.join(directory, "**", "*.db"), recursive=True)
    if not dbs:
        raise SystemExit(f"no counter output under {directory}")
    import sqlite3
    for path in dbs:
        con = sqlite3.connect(path)
        try:
            for name, cname, val in con.execute(
                    "select kernel_name, counter_name, value from counters_collection"):
                yield name, cname, float(val)
        finally:
            con.close()


def summarize_pmc(directory: str, w: workloads.Workload, command: str, tag: str = "") -> dict:
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the softmax
    kernel and of the copy kernel, scaled by the copy kernel's reading for
    its known byte count (4 * elements read, 4 * elements written)."""
    per = {}
    subs = ["fetch", "write"] + [d for d in ("occ", "sq")
                                 if os.path.isdir(os.path.join(directory, d))]
    for sub in subs:
        for name, cname, val in _counter_rows(os.path.join(directory, sub)):
            key = "copy" if "k_copy" in name else ("softmax" if "smx::k_" in name else None)
            if key is None:
                continue
            per.setdefault((key, cname, name), []).append(val)
    agg = {}
    for (key, cname, name), vals in per.items():
        agg.setdefault(key, {})[cname] = float(np.median(vals))
        agg[key].setdefault("kernels", set()).add(name.split("(")[0])
    bytes_each_way = 4.0 * w.elements
    scale_fetch = bytes_each_way / (agg["copy"]["FETCH_SIZE"] * 1024.0)
    scale_write = bytes_each_way / (agg["copy"]["WRITE_SIZE"] * 1024.0)
    fetch_b = agg["softmax"]["FETCH_SIZE"] * 1024.0 * scale_fetch
    write_b = agg["softmax"]["WRITE_SIZE"] * 1024.0 * scale_write
    doc = {
        "workload": w.key,
        "softmax_kernels": sorted(agg["softmax"]["kernels"]),
        "source_sha256": kernel_source_sha256(),
        "softmax_fetch_kib_per_dispatch": agg["softmax"]["FETCH_SIZE"],
        "softmax_write_kib_per_dispatch": agg["softmax"]["WRITE_SIZE"],
        "copy_fetch_kib_per_dispatch": agg["copy"]["FETCH_SIZE"],
        "copy_write_kib_per_dispatch": agg["copy"]["WRITE_SIZE"],
        "copy_bytes_each_way": bytes_each_way,
        "scale_fetch": scale_fetch,
        "scale_write": scale_write,
        "traffic_fetch_bytes_per_launch": fetch_b,
        "traffic_write_bytes_per_launch": write_b,
        "traffic_bytes_per_launch": fetch_b + write_b,
        "algorithmic_bytes_per_launch": float(w.algorithmic_bytes),
        "traffic_over_algorithmic": (fetch_b + write_b) / w.algorithmic_bytes,
        "command": command,
        "tag": tag,
    }
    if "sq" in subs:
        names = sorted({c for k in ("softmax", "copy") for c in agg[k]
                        if c.startswith(("SQ_", "GRBM_", "TCC_", "TCP_", "TA_", "TD_"))
                        and c not in ("FETCH_SIZE", "WRITE_SIZE")})
        doc["sq_counters_median_per_dispatch"] = {
            k: {c: agg[k].get(c) for c in names} for k in ("softmax", "copy")}
    if "occ" in subs:
        for key in ("softmax", "copy"):
            doc[f"{key}_occupancy_percent"] = agg[key].get("OccupancyPercent")
            doc[f"{key}_sq_waves_per_dispatch"] = agg[key].get("SQ_WAVES")
            doc[f"{key}_grbm_gui_active_cycles"] = agg[key].get("GRBM_GUI_ACTIVE")
    os.makedirs(PROFILES, exist_ok=True)
    with open(pmc_summary_path(w.key, "json", tag), "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    with open(pmc_summary_path(w.key, "md", tag), "w") as f:
        f.write(f"# HBM traffic counters: {', '.join(doc['softmax_kernels'])} on {w.key}"
                f"{' (' + tag.replace('_', ' ') + ')' if tag else ''}\n\n")
        f.write("Commands (from the repository root on the GPU machine):\n\n```\n"
                f"{command}\n```\n\n")
        f.write("| quantity | softmax kernel | copy kernel (same bytes) |\n|---|---|---|\n")
        f.write("| FETCH_SIZE KiB/dispatch (median) | "
                f"{doc['softmax_fetch_kib_per_dispatch']:.1f} | "
                f"{doc['copy_fetch_kib_per_dispatch']:.1f} |\n")
        f.write("| WRITE_SIZE KiB/dispatch (median) | "
                f"{doc['softmax_write_kib_per_dispatch']:.1f} | "
                f"{doc['copy_write_kib_per_dispatch']:.1f} |\n\n")
        f.write(f"Copy kernel moves {bytes_each_way:.0f} bytes each way; scale factors "
                f"fetch {scale_fetch:.4f}, write {scale_write:.4f}.\n\n")
        f.write(f"Scaled traffic per launch: fetch {fetch_b:.0f} B + write {write_b:.0f} B = "
                f"{fetch_b + write_b:.0f} B; algorithmic {w.algorithmic_bytes} B; ratio "
                f"{doc['traffic_over_algorithmic']:.4f}.\n\n")
        if "occ" in subs:
            f.write("Occupancy pass (OccupancyPercent = 400 * SQ_WAVE_CYCLES / "
                    "GRBM_GUI_ACTIVE / CUs / 32, the profiler's derived counter: mean "
                    "resident waves per CU over the dispatch as % of 32):\n\n"
                    "| quantity | softmax kernel | copy kernel |\n|---|---|---|\n")
            for label, k in (("OccupancyPercent (median)", "occupancy_percent"),
                             ("SQ_WAVES per dispatch", "sq_waves_per_dispatch"),
                             ("GRBM_GUI_ACTIVE cycles", "grbm_gui_active_cycles")):
                a, b = doc[f"softmax_{k}"], doc[f"copy_{k}"]
                f.write(f"| {label} | {a if a is None else round(a, 1)} | "
                        f"{b if b is None else round(b, 1)} |\n")
        if "sq_counters_median_per_dispatch" in doc:
            sq = doc["sq_counters_median_per_dispatch"]
            f.write("\nSQ / GRBM pass (median per dispatch; cycle counters are summed "
                    "over the XCDs' sequencers as the profiler reports them):\n\n"
                    "| counter | softmax kernel | copy kernel |\n|---|---|---|\n")
            for c in sq["softmax"]:
                a, b = sq["softmax"][c], sq["copy"][c]
                f.write(f"| {c} | {a if a is None else round(a, 1)} | "
                        f"{b if b is None else round(b, 1)} |\n")
            f.write("\n")
        f.write(f"Kernel sources sha256: {doc['source_sha256']}\n")
    return doc


def summarize_trace(directory: str, command: str, bench_json: str | None) -> str:
    """profiles/trace_bench.{md,json} from a rocprofv3 --kernel-trace --stats
    run of this script: per (kernel, grid) dispatch durations (median, p10,
    p90, mean) and register / LDS usage, the per-kernel stats table, and the
    step times the same run printed."""
    traces = glob.glob(os.path.join(directory, "**", "*kernel_trace.csv"), recursive=True)
    stats = glob.glob(os.path.join(directory, "**", "*kernel_stats.csv"), recursive=True)
    if not traces or not stats:
        raise SystemExit(f"no kernel_trace.csv / kernel_stats.csv under {directory}")
    groups: dict = {}
    with open(traces[0]) as f:
        for r in csv.DictReader(f):
            if "smx::" not in r["Kernel_Name"]:
                continue
            key = (r["Kernel_Name"].split("(")[0].replace("void ", ""), int(r["Grid_Size_X"]))
            g = groups.setdefault(key, {"d": [], "res": r})
            g["d"].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    with open(stats[0]) as f:
        rows = list(csv.DictReader(f))
    bench = None
    if bench_json:
        with open(bench_json) as f:
            bench = json.loads(f.read().strip().splitlines()[-1])
    doc = {"source_sha256": kernel_source_sha256(), "command": command, "kernels": []}
    for (name, grid), g in sorted(groups.items()):
        r = g["res"]
        # Runs of calls more than 0.5 s apart are reported apart: the same
        # launch shape can come from different parts of the run (the unfused
        # attention reference calls softmax_fwd on the DAM shape).
        calls = sorted(g["d"])
        runs = [[calls[0]]]
        for c in calls[1:]:
            if c[0] - runs[-1][-1][1] > 500_000_000:
                runs.append([])
            runs[-1].append(c)
        for k, run in enumerate(runs):
            d = np.array([(e - b) / 1e3 for b, e in run])
            doc["kernels"].append({
                "kernel": name, "grid_threads": grid, "run": k + 1, "runs": len(runs),
                "calls": int(d.size), "median_us": float(np.median(d)),
                "p10_us": float(np.percentile(d, 10)), "p90_us": float(np.percentile(d, 90)),
                "mean_us": float(d.mean()), "vgpr": r["VGPR_Count"], "sgpr": r["SGPR_Count"],
                "lds_bytes": r["LDS_Block_Size"], "scratch_bytes": r["Scratch_Size"]})
    if bench:
        doc["bench_line"] = {"workload": bench["config"]["workload"],
                             "ms_per_step": bench["ms_per_step"],
                             "graded": {k: v["ms_per_step"] for k, v in bench["graded"].items()}}
    os.makedirs(PROFILES, exist_ok=True)
    with open(TRACE_JSON, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    path = TRACE_JSON[:-5] + ".md"
    with open(path, "w") as f:
        f.write("# Kernel trace of bench.py\n\n")
        f.write(f"Command (repository root, GPU machine):\n\n```\n{command}\n```\n\n")
        f.write("Per dispatch, grouped by kernel and grid (eager and graph-replayed "
                "launches together; durations are the profiler's begin-to-end times). "
                "The last template argument of the softmax kernels is the mode: 0 "
                "softmax_fwd, 1 no clip, 2 approximate exponential, 3 log-softmax, 4 "
                "negative log-likelihood.  A shape seen in separate parts of the run is "
                "split into runs: the second run of the DAM-shaped k_packed mode 0 is "
                "the unfused attention reference (softmax_fwd between two hipBLAS "
                "products).\n\n")
        f.write("| kernel | grid threads | run | calls | median us | p10 us | p90 us | "
                "mean us | VGPR | SGPR | LDS B | scratch B |\n"
                "|---|---|---|---|---|---|---|---|---|---|---|---|\n")
        for k in doc["kernels"]:
            f.write(f"| `{k['kernel']}` | {k['grid_threads']} | {k['run']}/{k['runs']} | "
                    f"{k['calls']} | {k['median_us']:.2f} | {k['p10_us']:.2f} | "
                    f"{k['p90_us']:.2f} | {k['mean_us']:.2f} | {k['vgpr']} | {k['sgpr']} | "
                    f"{k['lds_bytes']} | {k['scratch_bytes']} |\n")
        f.write("\nrocprofv3 --stats table (all kernels of the run):\n\n")
        f.write("| kernel | calls | average us | min us | max us |\n|---|---|---|---|---|\n")
        for r in rows:
            f.write(f"| `{r['Name'].split('(')[0][:120]}` | {r['Calls']} | "
                    f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                    f"{float(r['MaxNs']) / 1e3:.2f} |\n")
        if bench:
            f.write(f"\nThe same run's JSON line: {bench['config']['workload']} "
                    f"{bench['ms_per_step'] * 1e3:.2f} us per step by HIP events "
                    f"(graph replay); graded: ")
            f.write(", ".join(f"{k} {v['ms_per_step'] * 1e3:.2f} us"
                              for k, v in bench["graded"].items()))
            f.write("; other workloads: ")
            f.write(", ".join(f"{k} {v['ms_per_step'] * 1e3:.2f} us"
                              for k, v in bench["other_workloads"].items()))
            f.write(".  Event time per step includes the gap between consecutive "
                    "kernels; the profiler's durations do not.\n")
        f.write(f"\nKernel sources sha256: {doc['source_sha256']}\n")
    return path


def kernel_trace_stats(kernel: str, grid_threads: int | None) -> dict | None:
    """Median / p10 / p90 of one kernel shape (any grid when grid_threads is
    None) from profiles/trace_bench.json, if the kernel sources still hash to
    what the trace was taken with."""
    if not os.path.exists(TRACE_JSON):
        return None
    with open(TRACE_JSON) as f:
        doc = json.load(f)
    if doc.get("source_sha256") != kernel_source_sha256():
        return {"note": "kernel changed since the trace was taken"}
    for k in doc["kernels"]:
        if (k["kernel"] == kernel and grid_threads in (None, k["grid_threads"])
                and k["run"] == 1):
            return {kk: k[kk] for kk in ("median_us", "p10_us", "p90_us", "mean_us", "calls")}
    return None


def plan_kernel_name(plan: dict, cols: int, mode: int = 0) -> str:
    """The demangled template instance softmax_fwd launches for a plan on
    rows of `cols` columns (the row kernels' last argument says whether the
    rows are taken with their phase: 128-bit access to rows that are not
    whole 16-byte strips)."""
    v = plan["elems_per_lane"] // 4
    vec = "true" if plan["vec_width"] == 4 else "false"
    ph = "true" if plan["vec_width"] == 4 and cols % 4 != 0 else "false"
    k = plan["kernel_name"]
    if k == "packed":
        return f"smx::k_packed<{plan['lanes_per_row']}, {plan['elems_per_lane']}, {vec}, {mode}>"
    if k == "group_rows":  # the row groups per step (1 or 2) are not in the plan
        return "smx::k_group_rows"
    if k == "wave_row":
        return f"smx::k_wave_row<{v}, {vec}, {mode}, {ph}>"
    if k == "block_row":
        return f"smx::k_block_row<{plan['block_threads']}, {v}, {vec}, {mode}, {ph}>"
    return f"smx::k_split_onepass<{plan['block_threads']}, {v}, {vec}, {mode}, {ph}>"


def roofline(w, res: dict, traffic, traffic_note, plan: dict) -> dict:
    ms = res["ms_per_step"]
    name = plan_kernel_name(plan, w.cols)
    return {
        "bound": "hbm",
        "achieved": res["hbm_gbps"],
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": res["frac_of_peak"],
        "traffic": traffic,
        "traffic_note": traffic_note,
        "algorithmic_bytes_per_launch": w.algorithmic_bytes,
        "kernel": name,
        "launches_per_step": plan["launches"],
        "launch_duration_us": ms * 1e3 / plan["launches"],
        "kernel_trace": kernel_trace_stats(name, plan["grid"] * plan["block_threads"]),
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    choices=list(workloads.WORKLOADS) + list(workloads.ATTENTION_WORKLOADS),
                    help="the headline softmax workload (attention workloads: counter "
                         "passes only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra-workloads", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--pmc-run", action="store_true",
                    help="only launch the kernels for a rocprofv3 counter pass")
    ap.add_argument("--pmc-launches", type=int, default=20)
    ap.add_argument("--pmc-in-place", action="store_true",
                    help="counter pass with y == x (softmax workloads)")
    ap.add_argument("--pmc-tag", default="",
                    help="suffix of the summary's file name (--summarize-pmc)")
    ap.add_argument("--summarize-pmc", metavar="DIR",
                    help="write profiles/pmc_<workload>.{json,md} from DIR/fetch and DIR/write")
    ap.add_argument("--pmc-command", default="", help="commands recorded in the summary")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="write profiles/trace_bench.{json,md} from a kernel-trace run")
    ap.add_argument("--trace-json", help="JSON line printed by the traced run")
    args = ap.parse_args()

    if args.workload in workloads.ATTENTION_WORKLOADS:
        w = AttentionCounters(args.workload)
        if not (args.pmc_run or args.summarize_pmc):
            print("attention workloads are timed inside the default run; use them with "
                  "--pmc-run or --summarize-pmc", file=sys.stderr)
            return 2
    else:
        w = workloads.WORKLOADS[args.workload]
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace, args.pmc_command, args.trace_json))
        return 0
    if args.summarize_pmc:
        doc = summarize_pmc(args.summarize_pmc, w, args.pmc_command, args.pmc_tag)
        print(json.dumps(doc), flush=True)
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the softmax rows are independent, so a "
              "multi-GPU run would shard rows with no communication; run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch

    import paper_1904_12380_amd as sm
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    sm.load_library()

    if args.pmc_run:
        if isinstance(w, AttentionCounters):
            pmc_run_attention(sm, torch, w, args.pmc_launches)
        else:
            pmc_run(sm, torch, w, args.pmc_launches, in_place=args.pmc_in_place)
        return 0

    machine_before = machine_state()
    warm_clocks(sm, torch)
    order = [w.key] + [k for k in GRADED if k != w.key]
    if not args.no_extra_workloads:
        order += [k for k in workloads.WORKLOADS if k not in order]
    results: dict = {}
    inputs: dict = {}
    for key in order:
        wk = workloads.WORKLOADS[key]
        log(f"[bench] timing {key}: {args.warmup} warmup + {args.steps} steps (graph replay)")
        x = workloads.generate(key)
        r = time_gpu(sm, torch, wk, x, args.steps, args.warmup, memcpy=(key == w.key))
        results[key] = r
        if key in GRADED or key == w.key:
            inputs[key] = x
        log(f"[bench] {key}: {r['ms_per_step'] * 1e3:.2f} us/step, {r['hbm_gbps']:.0f} GB/s "
            f"({r['frac_of_peak']:.3f} of peak; eager {r['eager_ms_per_step'] * 1e3:.2f} us, "
            f"in place {r['in_place_ms_per_step'] * 1e3:.2f} us, copy "
            f"{r['copy_ms_per_step'] * 1e3:.2f} us, no clip "
            f"{r['noclip_ms_per_step'] * 1e3:.2f} us, approx exp "
            f"{r['approx_exp_ms_per_step'] * 1e3:.2f} us, log "
            f"{r['log_softmax_ms_per_step'] * 1e3:.2f} us, nll {r['nll_ms_per_step'] * 1e3:.2f} us)")

    attention = None
    if not args.no_extra_workloads:
        akey = next(iter(workloads.ATTENTION_WORKLOADS))
        log(f"[bench] timing fused attention {akey}")
        attention = time_attention(sm, torch, akey, args.steps, args.warmup)
        log(f"[bench] {akey}: {attention['ms_per_step'] * 1e3:.2f} us/step, "
            f"{attention['hbm_gbps']:.0f} GB/s, {attention['tflops']:.1f} TFLOP/s; unfused "
            f"{attention['unfused_ms_per_step'] * 1e3:.2f} us")
    machine_after = machine_state()

    def rounded(d: dict) -> dict:
        return {k: (float(f"{v:.6g}") if isinstance(v, float) else v)
                for k, v in d.items() if k != "plan"}

    graded = {}
    cpu_main = cpu32_main = None
    for key in [k for k in order if k in GRADED or k == w.key]:
        wk = workloads.WORKLOADS[key]
        r = results[key]
        traffic, note = load_traffic(key)
        entry = rounded(r)
        entry["plan"] = r["plan"]
        entry["roofline"] = roofline(wk, r, traffic, note, r["plan"])
        entry["cpu_baseline"] = entry["cpu_fp32_baseline"] = None
        if not args.no_cpu_baseline:
            log(f"[bench] CPU oracle baseline on {key}")
            entry["cpu_baseline"] = time_cpu_oracle(inputs[key], args.cpu_budget)
            log(f"[bench] CPU fp32 baseline on {key}")
            entry["cpu_fp32_baseline"] = time_cpu_fp32(inputs[key], min(args.cpu_budget, 5.0))
        if key == w.key:
            cpu_main, cpu32_main = entry["cpu_baseline"], entry["cpu_fp32_baseline"]
        if key in GRADED:
            graded[key] = entry

    main_res = results[w.key]
    x = inputs[w.key]
    ms = main_res["ms_per_step"]
    plan = main_res["plan"]
    traffic, traffic_note = load_traffic(w.key)
    extra = {}
    for key, r in results.items():
        if key in GRADED or key == w.key:
            continue
        extra[key] = rounded(r)
        extra[key]["kernel"] = r["plan"]["kernel_name"]
        extra[key]["launches_per_step"] = r["plan"]["launches"]
        extra[key]["store_delay_ns"] = r["plan"]["store_delay_ns"]
    out = {
        "metric": METRIC,
        "value": main_res["rows_per_s"],
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.key, "rows": w.rows, "cols": w.cols, "seed": w.seed,
                   "input_sha256": workloads.sha256_f32(x),
                   "kernel": plan["kernel_name"], "launches_per_step": plan["launches"],
                   "chunks_per_row": plan["chunks_per_row"],
                   "store_delay_ns": plan["store_delay_ns"],
                   "rotation_buffers": main_res["rotation_buffers"],
                   "timing": "HIP graph of the timed steps on a dedicated stream, HIP "
                             "events recorded behind a queued pre-roll replay"},
        "elements_per_s": main_res["elements_per_s"],
        "hbm_gbps": main_res["hbm_gbps"],
        "roofline": roofline(w, main_res, traffic, traffic_note, plan),
        "cpu_baseline": cpu_main,
        "cpu_fp32_baseline": cpu32_main,
        "graded": graded,
        "eager": {"ms_per_step": main_res["eager_ms_per_step"],
                  "hbm_gbps": main_res["eager_hbm_gbps"]},
        "in_place": {"ms_per_step": main_res["in_place_ms_per_step"],
                     "hbm_gbps": main_res["in_place_hbm_gbps"],
                     "what": "softmax_fwd with y == x, on the rotation's y buffers"},
        "copy_ceiling": {"gbps": main_res["copy_gbps"],
                         "ms_per_step": main_res["copy_ms_per_step"],
                         "softmax_over_copy_time": main_res["softmax_over_copy_time"],
                         "memcpy_d2d_ms_per_step": main_res["memcpy_ms_per_step"],
                         "memcpy_d2d_gbps": w.algorithmic_bytes
                         / (main_res["memcpy_ms_per_step"] * 1e-3) / 1e9,
                         "launch_floor_ms_per_step": main_res["launch_floor_ms_per_step"],
                         "launch_floor_what": "softmax_copy_probe on 4 KiB: the fixed cost "
                                              "of one graph-replayed launch that reads, "
                                              "then writes"},
        "no_clip": {"ms_per_step": main_res["noclip_ms_per_step"],
                    "hbm_gbps": main_res["noclip_hbm_gbps"],
                    "what": "softmax_fwd_clip with clip_lo = -inf, same rotation and timing"},
        "log_softmax": {"ms_per_step": main_res["log_softmax_ms_per_step"],
                        "hbm_gbps": main_res["log_softmax_hbm_gbps"],
                        "what": "softmax_log_fwd (log of the clipped softmax), same rotation "
                                "and timing"},
        "nll": {"ms_per_step": main_res["nll_ms_per_step"],
                "hbm_gbps": main_res["nll_hbm_gbps"],
                "algorithmic_bytes_per_launch": main_res["nll_algorithmic_bytes"],
                "what": "softmax_nll_fwd (per-row loss of a label; x read once, 4 B "
                        "written per row), same rotation and timing"},
        "approx_exp": {"ms_per_step": main_res["approx_exp_ms_per_step"],
                       "hbm_gbps": main_res["approx_exp_hbm_gbps"],
                       "what": "softmax_fwd_approx (single-instruction fp32 exponential), "
                               "same rotation and timing"},
        "sampled_max_rel_err": main_res["sampled_max_rel_err"],
        "machine": {"before": machine_before, "after": machine_after,
                    "gpu": torch.cuda.get_device_name(0),
                    "compute_units": torch.cuda.get_device_properties(0).multi_processor_count},
        "other_workloads": extra,
        "fused_attention": attention,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
