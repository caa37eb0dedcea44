"""Split rows: the exchange table, the store schedule and the planned entry.

Rows longer than 32768 columns are spread over several workgroups that
combine partial (max, sum) pairs through a region of a static device table
claimed per launch (include/softmax_mi355x.h, softmax_fwd "Scratch").  These
tests check, against the float64 oracle, that this needs no allocation and
no host-side state: a first call made under stream capture, more than 64
streams, calls on several streams at once and graphs replayed at the same
time; that every region is back at rest and no wait gave up afterwards; that
the store delay changes no output bit; and that every kernel family reached
through softmax_fwd_planned matches the oracle.
"""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
import paper_1904_12380_amd as sm
import workloads

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
REL_TOL = 4e-6
SUM_TOL = 1e-5


def log(msg):
    print(msg, flush=True)


def _torch():
    import torch
    return torch


def check(x, y, what):
    want = oracle.softmax_clipped(x)
    y64 = y.astype(np.float64)
    rel = float(np.max(np.abs(y64 - want) / want))
    assert rel <= REL_TOL, (what, rel)
    assert float(np.max(np.abs(y64.sum(axis=1) - 1.0))) <= SUM_TOL, what
    return rel


def assert_exchange_at_rest():
    _torch().cuda.synchronize()
    st = sm.softmax_exchange_status()
    log(f"[exchange] status {st}")
    assert st == {"join_give_ups": 0, "wait_give_ups": 0, "entries_in_use": 0}, st


CAPTURE_FIRST = r"""
import json, sys
sys.path.insert(0, {root!r})
import numpy as np, torch
import oracle, workloads
import paper_1904_12380_amd as sm
dev = torch.device("cuda:0")
x = workloads.random_logits(6, 262144, seed=21, kind="offset")
xt = torch.from_numpy(x).to(dev)
yg = torch.empty_like(xt)
s = torch.cuda.Stream()
g = torch.cuda.CUDAGraph()
# the library's first call in this process is made under capture
with torch.cuda.graph(g, stream=s):
    sm.softmax_fwd(xt, out=yg, stream=s)
want = oracle.softmax_clipped(x)
errs = []
for rep in range(3):
    yg.fill_(-1.0)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    y = yg.cpu().numpy().astype(np.float64)
    errs.append(float(np.max(np.abs(y - want) / want)))
print(json.dumps({{"errs": errs, "status": sm.softmax_exchange_status()}}), flush=True)
"""


def test_first_call_under_capture():
    """A fresh process whose first library call (a long-row one) is made
    under stream capture: the capture succeeds and every replay matches the
    oracle."""
    log("[exchange] first call under capture (child process)")
    code = CAPTURE_FIRST.format(root=ROOT)
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         timeout=180)
    assert res.returncode == 0, res.stdout + res.stderr
    out = json.loads(res.stdout.strip().splitlines()[-1])
    log(f"[exchange] child: {out}")
    assert max(out["errs"]) <= REL_TOL
    assert out["status"] == {"join_give_ups": 0, "wait_give_ups": 0, "entries_in_use": 0}


def test_more_than_64_streams_no_device_sync():
    """80 streams, each with its own long-row call queued before any
    synchronisation: all correct, and the table back at rest."""
    torch = _torch()
    log("[exchange] 80 streams")
    dev = torch.device("cuda:0")
    rows, cols = 3, 70000
    xs, ys, streams = [], [], []
    for i in range(80):
        x = workloads.random_logits(rows, cols, seed=100 + i, kind="offset")
        xs.append(x)
        xt = torch.from_numpy(x).to(dev)
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        streams.append(s)
        ys.append((xt, torch.empty_like(xt)))
    for (xt, yt), s in zip(ys, streams):
        sm.softmax_fwd(xt, out=yt, stream=s)
    torch.cuda.synchronize()
    for i, ((xt, yt), x) in enumerate(zip(ys, xs)):
        check(x, yt.cpu().numpy(), f"stream {i}")
    assert_exchange_at_rest()


def test_concurrent_streams_and_graph_replays():
    """Two captured graphs replayed on two streams while eager long-row calls
    run on a third: every output bitwise equal to its eager reference."""
    torch = _torch()
    log("[exchange] concurrent graphs + eager")
    dev = torch.device("cuda:0")
    shapes = [(64, 262144), (512, 65536), (7, 1048580)]
    xs = [torch.from_numpy(workloads.random_logits(r, c, seed=r + c, kind="normal")).to(dev)
          for r, c in shapes]
    ref = [sm.softmax_fwd(x) for x in xs]
    torch.cuda.synchronize()
    for x, r, (rows, cols) in zip(xs, ref, shapes):
        check(x.cpu().numpy(), r.cpu().numpy(), f"eager {rows}x{cols}")
    outs = [torch.empty_like(x) for x in xs]
    graphs, gstreams = [], []
    for i in range(2):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(3):
                sm.softmax_fwd(xs[i], out=outs[i], stream=s)
        graphs.append(g)
        gstreams.append(s)
    s3 = torch.cuda.Stream()
    for rep in range(4):
        for o in outs:
            o.fill_(-1.0)
        torch.cuda.synchronize()
        for g, s in zip(graphs, gstreams):
            with torch.cuda.stream(s):
                g.replay()
        for _ in range(3):
            sm.softmax_fwd(xs[2], out=outs[2], stream=s3)
        torch.cuda.synchronize()
        for o, r in zip(outs, ref):
            assert torch.equal(o.view(torch.int32), r.view(torch.int32)), rep
    assert_exchange_at_rest()


@pytest.mark.parametrize("key", ["vocab_512x32768", "longrow_64x262144", "classifier_4096x1000"])
def test_store_delay_changes_no_bit(key):
    """The store schedule only moves the stores in time: the library's
    kernel for each workload with its own delay, with none, with 9 us and
    with 50 us gives bitwise the output of softmax_fwd."""
    torch = _torch()
    log(f"[exchange] store delay {key}")
    x = torch.from_numpy(workloads.generate(key)).to(torch.device("cuda:0"))
    rows, cols = x.shape
    p = sm.softmax_plan(rows, cols, x.data_ptr(), x.data_ptr() + (1 << 40))
    plan = dict(kernel_name=p["kernel_name"], vec_width=p["vec_width"],
                block_threads=p["block_threads"], elems_per_lane=p["elems_per_lane"])
    base = sm.softmax_fwd(x)
    for delay in (-1, 0, 9000, 50000):
        y = sm.softmax_fwd_planned(x, dict(plan, store_delay_ns=delay))
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int32), base.view(torch.int32)), delay
    check(x.cpu().numpy(), base.cpu().numpy(), key)
    assert_exchange_at_rest()


PLANNED = [
    ("packed", 4, {}, [(1000, 50), (333, 17), (77, 64), (501, 65), (333, 250), (64, 256)]),
    ("packed", 1, {}, [(129, 65), (70, 255)]),
    ("group_rows", 4, {}, [(1000, 52), (333, 16), (77, 256), (9, 4), (4099, 8)]),
    ("wave_row", 4, {}, [(300, 52), (257, 1000), (9, 4096)]),
    ("wave_row", 1, {}, [(130, 1001), (5, 2047)]),
    ("wave_row", 4, {}, [(17, 2049), (9, 4093)]),
    ("block_row", 4, {}, [(5, 8189), (6, 4097), (7, 2051)]),
    ("block_row", 4, {}, [(64, 1000), (9, 8192), (5, 32768)]),
    ("block_row", 1, {}, [(20, 999), (5, 32767)]),
    ("split_row", 4, dict(block_threads=256, elems_per_lane=32), [(33, 1000), (9, 32768),
                                                                  (3, 262144)]),
    ("split_row", 4, dict(block_threads=512, elems_per_lane=32), [(17, 40000), (3, 1048576)]),
    ("split_row", 4, dict(block_threads=512, elems_per_lane=64), [(6, 65536), (2, 2097152)]),
    ("split_row", 1, dict(block_threads=256, elems_per_lane=32), [(11, 8193), (3, 100003)]),
    ("split_row", 4, dict(block_threads=256, elems_per_lane=32), [(11, 8193), (3, 100003),
                                                                  (5, 65533)]),
    ("split_row", 4, dict(block_threads=512, elems_per_lane=32), [(3, 100003), (2, 1048573)]),
    ("split_row", 1, dict(block_threads=512, elems_per_lane=32), [(3, 1048577)]),
]


@pytest.mark.parametrize("kernel,vec,extra,shapes", PLANNED,
                         ids=[f"{k}-{v}-{e.get('block_threads', '')}x{e.get('elems_per_lane', '')}"
                              for k, v, e, _ in PLANNED])
def test_planned_kernels_match_oracle(kernel, vec, extra, shapes):
    """Each kernel family through softmax_fwd_planned, on shapes outside the
    range the default dispatch sends it (split rows of one chunk, block rows
    of 999 columns, ...), against the oracle."""
    torch = _torch()
    dev = torch.device("cuda:0")
    for rows, cols in shapes:
        log(f"[planned] {kernel} vec{vec} {extra} {rows}x{cols}")
        x = workloads.random_logits(rows, cols, seed=rows * 31 + cols, kind="clip_heavy")
        n = rows * cols
        if vec == 4:
            xt = torch.from_numpy(x).to(dev)
            yt = torch.empty_like(xt)
        else:   # 4 bytes past a 16-byte boundary: 32-bit access only
            xb = torch.empty(n + 4, dtype=torch.float32, device=dev)
            yb = torch.empty(n + 4, dtype=torch.float32, device=dev)
            xb[1:n + 1] = torch.from_numpy(x.reshape(-1)).to(dev)
            xt, yt = xb[1:n + 1].view(rows, cols), yb[1:n + 1].view(rows, cols)
        sm.softmax_fwd_planned(xt, dict(kernel_name=kernel, vec_width=vec, **extra), out=yt)
        torch.cuda.synchronize()
        check(x, yt.cpu().numpy(), f"{kernel} {rows}x{cols}")
    assert_exchange_at_rest()


def test_plan_geometry_on_device():
    """Grid, launches and store delay for the workloads, on this device."""
    torch = _torch()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    p = sm.softmax_plan(115200, 50)
    assert p["kernel_name"] == "packed" and p["grid"] == 6 * cus and p["launches"] == 1
    assert p["store_delay_ns"] == 0
    p = sm.softmax_plan(4096, 1000)
    assert p["kernel_name"] == "wave_row" and p["grid"] == 1024 and p["store_delay_ns"] == 0
    p = sm.softmax_plan(512, 32768)
    assert p["kernel_name"] == "split_row" and p["chunks_per_row"] == 4
    assert p["grid"] == 2048 and p["launches"] == 1
    assert 8000 < p["store_delay_ns"] < 10000
    p = sm.softmax_plan(512, 32765)              # row phase: 128-bit, scheduled stores
    assert p["vec_width"] == 4 and p["chunks_per_row"] == 4 and p["store_delay_ns"] > 0
    p = sm.softmax_plan(512, 32765, (1 << 44) + 4, 1 << 45)   # 32-bit access: no schedule
    assert p["vec_width"] == 1 and p["store_delay_ns"] == 0
    p = sm.softmax_plan(512, 32767)              # the phase would add a chunk: 32-bit
    assert p["vec_width"] == 1 and p["chunks_per_row"] == 4
    p = sm.softmax_plan(64, 262144)
    assert p["chunks_per_row"] == 16 and p["launches"] == 1 and p["grid"] == 1024
    assert 8000 < p["store_delay_ns"] < 10000
    p = sm.softmax_plan(7, 262144)               # 7 MiB of reads: no delay
    assert p["store_delay_ns"] == 0
    p = sm.softmax_plan(10000, 262144)       # several one-pass launches
    per_launch = p["grid"] // p["chunks_per_row"]
    assert per_launch * p["chunks_per_row"] == p["grid"]
    assert p["launches"] == -(-10000 // per_launch)
    p = sm.softmax_plan(2, 1 << 30)          # two passes per batch of rows
    assert p["launches"] % 2 == 0
