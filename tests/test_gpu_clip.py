"""GPU parity for the clip bound as a parameter (softmax_fwd_clip), through the
C ABI, against the float64 oracle at the same bound.

Bar per element: |y - y_ref| <= 4e-6 * y_ref + 2^-148.  The absolute term is
two steps of the smallest fp32 denormal: without the clip (or with a bound
below -87) outputs can be denormal or 0, where fp32 has no relative
precision left.  Per row: |sum_j y_ij - 1| <= 1e-5.  NaN rows must match the
oracle's NaN rows exactly.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_1904_12380_amd as sm
import workloads

pytestmark = pytest.mark.gpu

REL_TOL = 4e-6
ABS_TOL = 2.0 ** -148
SUM_TOL = 1e-5
NEG_INF = float("-inf")
BOUNDS = [-48.0, -64.0, -80.0, -87.0, -87.5, -100.0, -120.0, -200.0, NEG_INF]


def _torch():
    import torch
    return torch


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_clip(x: np.ndarray, lo: float) -> np.ndarray:
    torch = _torch()
    xt = torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")
    yt = sm.softmax_fwd_clip(xt, lo)
    torch.cuda.synchronize()
    return yt.cpu().numpy()


def check_clip(x: np.ndarray, y: np.ndarray, lo: float, what: str) -> float:
    want = oracle.softmax_clipped(x, lo)
    y64 = y.astype(np.float64)
    assert np.array_equal(np.isnan(y64), np.isnan(want)), what
    fin = np.isfinite(want)
    err = np.abs(y64[fin] - want[fin])
    bound = REL_TOL * want[fin] + ABS_TOL
    if err.size and np.any(err > bound):
        k = int(np.argmax(err / bound))
        idx = np.unravel_index(np.flatnonzero(fin)[k], y.shape)
        pytest.fail(f"{what} lo={lo}: err {err[k]:.3e} > {bound[k]:.3e} at {idx}: "
                    f"got {y64[idx]!r}, want {want[idx]!r}, x={x[idx]!r}, "
                    f"rowmax={x[idx[0]].max()!r}")
    rows_ok = np.all(fin, axis=1)
    if rows_ok.any():
        assert float(np.abs(y64[rows_ok].sum(axis=1) - 1.0).max()) <= SUM_TOL, what
    big = fin & (want >= 2.0 ** -126)
    return float((np.abs(y64[big] - want[big]) / want[big]).max()) if big.any() else 0.0


# One shape per kernel family and path: packed (G = 1, 4), grouped aligned
# rows (G = 16, 32), wave per row, block per row, one-pass split (small and
# large chunks), two-pass split.
SHAPES = [(1000, 50), (257, 7), (1001, 64), (300, 100), (64, 1000), (5, 8192), (3, 100003),
          (2, 1048577), (1, 2097153)]


@pytest.mark.parametrize("rows,cols", SHAPES)
def test_bounds_on_every_kernel(rows, cols):
    log(f"[clip] bounds {rows}x{cols}")
    for kind in ("clip_heavy", "normal"):
        x = workloads.random_logits(rows, cols, seed=rows + cols, kind=kind, scale=30.0)
        for lo in BOUNDS:
            worst = check_clip(x, run_clip(x, lo), lo, f"{rows}x{cols} {kind}")
            log(f"[clip] {rows}x{cols} {kind} lo={lo}: max rel err (normal range) {worst:.3e}")


@pytest.mark.parametrize("key", list(workloads.WORKLOADS))
def test_workloads_without_clip(key):
    """The five workloads with the clip off (the paper's optimised functor)."""
    log(f"[clip] workload {key}, no clip")
    x = workloads.generate(key)
    worst = check_clip(x, run_clip(x, NEG_INF), NEG_INF, key)
    log(f"[clip] {key} no clip: max rel err {worst:.3e}")


@pytest.mark.parametrize("key", ["dam_attention_115200x50", "classifier_4096x1000",
                                 "vocab_512x32768", "longrow_64x262144"])
def test_default_bound_is_softmax_fwd_bitwise(key):
    torch = _torch()
    x = torch.from_numpy(workloads.generate(key)).to("cuda:0")
    a = sm.softmax_fwd(x)
    b = sm.softmax_fwd_clip(x, -64.0)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("rows,cols", [(33, 1001), (131, 7), (3, 100003)])
def test_misaligned_without_clip(rows, cols):
    torch = _torch()
    log(f"[clip] misaligned {rows}x{cols}")
    x = workloads.random_logits(rows, cols, seed=cols, kind="clip_heavy")
    n = rows * cols
    xb = torch.empty(n + 4, dtype=torch.float32, device="cuda:0")
    yb = torch.empty(n + 4, dtype=torch.float32, device="cuda:0")
    xb[1:n + 1] = torch.from_numpy(x.reshape(-1)).to("cuda:0")
    xv, yv = xb[1:n + 1].view(rows, cols), yb[1:n + 1].view(rows, cols)
    assert sm.softmax_plan(rows, cols, xv.data_ptr(), yv.data_ptr())["vec_width"] == 1
    sm.softmax_fwd_clip(xv, NEG_INF, out=yv)
    torch.cuda.synchronize()
    check_clip(x, yv.cpu().numpy(), NEG_INF, f"misaligned {rows}x{cols}")


@pytest.mark.parametrize("cols", [5, 50, 1000, 8192, 70000])
def test_nonfinite_rows_without_clip(cols):
    """No clip: -inf entries give exactly 0, NaN and +inf rows are NaN, an
    all -inf row is NaN."""
    rng = np.random.default_rng(cols)
    x = rng.standard_normal((5, cols)).astype(np.float32)
    x[0, cols // 2] = np.nan
    x[1, cols // 3] = np.inf
    x[2, :] = -np.inf
    x[3, ::2] = -np.inf
    y = run_clip(x, NEG_INF)
    assert np.all(np.isnan(y[:3]))
    assert np.all(y[3, ::2] == 0.0)
    check_clip(x, y, NEG_INF, f"nonfinite {cols}")


def test_one_hot_rows_without_clip():
    """A row with one finite entry and -inf elsewhere is exactly one-hot."""
    for cols in (7, 50, 1000, 8192, 100003):
        x = np.full((3, cols), -np.inf, dtype=np.float32)
        for i in range(3):
            x[i, (i * 977) % cols] = 3.5 * i
        y = run_clip(x, NEG_INF)
        want = np.zeros_like(y)
        for i in range(3):
            want[i, (i * 977) % cols] = 1.0
        assert np.array_equal(y, want), cols


def test_exp_probe_wide_range():
    """The kernels' exp without a clip, over shifted logits down to -110,
    against float64 exp: 2 ulp where the result is a normal fp32, and below
    2^-126 the same 2 ulp relative plus half a denormal step (2^-150), the
    final rounding onto the denormal grid."""
    torch = _torch()
    rng = np.random.default_rng(98)
    n = 1 << 21
    m = rng.uniform(-40.0, 40.0, n).astype(np.float32)
    d = np.concatenate([rng.uniform(-110.0, 0.0, n - 8192),
                        rng.uniform(-87.5, -87.2, 4096), rng.uniform(-104.0, -103.5, 4096)])
    x = (m.astype(np.float64) + d).astype(np.float32)
    for lo in (NEG_INF, -100.0, -87.5):
        e = sm.softmax_exp_probe(torch.from_numpy(x).to("cuda:0"),
                                 torch.from_numpy(m).to("cuda:0"), clip_lo=lo).cpu().numpy()
        want = oracle.exp_clipped(x.astype(np.float64) - m.astype(np.float64), lo)
        e64 = e.astype(np.float64)
        normal = want >= 2.0 ** -126
        rel = float((np.abs(e64[normal] - want[normal]) / want[normal]).max())
        assert rel <= 4.0 * 2.0 ** -24, (lo, rel)
        sub = ~normal
        err = np.abs(e64[sub] - want[sub])
        assert np.all(err <= 2.0 ** -150 + 4.0 * 2.0 ** -24 * want[sub]), (lo, float(err.max()))
        log(f"[clip] exp probe lo={lo}: max rel err {rel:.3e}, "
            f"max abs err below 2^-126 {float(err.max()):.3e}")


def test_invalid_bounds_raise():
    torch = _torch()
    x = torch.zeros(4, 8, device="cuda:0")
    for lo in (float("nan"), -47.0, 0.0, float("inf")):
        with pytest.raises(sm.SoftmaxError):
            sm.softmax_fwd_clip(x, lo)


def test_graph_capture_without_clip():
    """A captured no-clip call replays bit-identical to the eager call."""
    torch = _torch()
    x = torch.from_numpy(workloads.random_logits(64, 262144, seed=3,
                                                 kind="clip_heavy")).to("cuda:0")
    want = sm.softmax_fwd_clip(x, NEG_INF)
    torch.cuda.synchronize()
    yg = torch.empty_like(x)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        sm.softmax_fwd_clip(x, NEG_INF, out=yg, stream=s)
    for rep in range(3):
        yg.fill_(-1.0)
        sm.softmax_fwd(x)                   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(yg.view(torch.int32), want.view(torch.int32)), rep


def test_bounds_on_three_chunk_block_rows():
    """Rows of 20480 columns with about 0.8 rows per compute unit take one
    1024-thread workgroup per row (8 strips per lane) rather than the split
    kernel; every bound on that instance."""
    import torch
    rows = torch.cuda.get_device_properties(0).multi_processor_count * 204 // 256
    cols = 20480
    p = sm.softmax_plan(rows, cols)
    assert p["kernel_name"] == "block_row" and p["elems_per_lane"] == 32, p
    log(f"[clip] bounds on block rows {rows}x{cols}")
    for kind in ("clip_heavy", "normal"):
        x = workloads.random_logits(rows, cols, seed=rows + 7, kind=kind, scale=30.0)
        for lo in BOUNDS:
            worst = check_clip(x, run_clip(x, lo), lo, f"{rows}x{cols} {kind}")
            log(f"[clip] {rows}x{cols} {kind} lo={lo}: max rel err (normal range) {worst:.3e}")
