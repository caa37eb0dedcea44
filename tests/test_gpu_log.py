"""GPU parity for the log of the clipped softmax (softmax_log_fwd), through
the C ABI, against ``oracle.log_softmax_clipped``.

Bar, from the arithmetic: the row sum carries the softmax path's rounding
(under 2e-6 relative), ln S comes from v_log_f32 (1 ulp of log2 S, at most
2.4e-7 |ln S|, and ln S <= ln(cols)), and c - ln S is rounded once to fp32
(half an ulp, 6e-8 |y|).  So per element

    |y - y*| <= 2e-6 + 2.5e-7 * (|y*| + ln(cols)),

-inf exactly where the oracle gives -inf, NaN exactly where it gives NaN.
"""
import math
import sys

import numpy as np
import pytest

import oracle
import paper_1904_12380_amd as sm
import workloads

pytestmark = pytest.mark.gpu
NEG_INF = float("-inf")


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_log(x, lo):
    import torch
    xt = torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")
    y = sm.softmax_log_fwd(xt, lo)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check_log(x, y, lo, what):
    want = oracle.log_softmax_clipped(x, lo)
    y64 = y.astype(np.float64)
    assert np.array_equal(np.isnan(y64), np.isnan(want)), what
    assert np.array_equal(np.isneginf(y64), np.isneginf(want)), what
    fin = np.isfinite(want)
    err = np.abs(y64[fin] - want[fin])
    bound = 2e-6 + 2.5e-7 * (np.abs(want[fin]) + math.log(max(x.shape[1], 1)))
    if err.size and np.any(err > bound):
        k = int(np.argmax(err / bound))
        idx = np.unravel_index(np.flatnonzero(fin)[k], want.shape)
        pytest.fail(f"{what} lo={lo}: err {err[k]:.3e} > {bound[k]:.3e} at {idx}: "
                    f"got {y64[idx]!r} want {want[idx]!r}")
    return float((err / bound).max()) if err.size else 0.0


@pytest.mark.parametrize("key", list(workloads.WORKLOADS))
def test_workloads(key):
    x = workloads.generate(key)
    for lo in (-64.0, NEG_INF):
        r = check_log(x, run_log(x, lo), lo, key)
        log(f"[log] {key} lo={lo}: worst error / bound {r:.3f}")


SHAPES = [(1000, 50), (257, 7), (64, 1000), (5, 8192), (9, 3000), (3, 100003), (2, 1048577),
          (1, 2097153)]


@pytest.mark.parametrize("rows,cols", SHAPES)
def test_shapes(rows, cols):
    for kind in ("clip_heavy", "normal", "offset"):
        x = workloads.random_logits(rows, cols, seed=rows * 13 + cols, kind=kind, scale=30.0)
        for lo in (-64.0, -90.0, NEG_INF):
            r = check_log(x, run_log(x, lo), lo, f"{rows}x{cols} {kind}")
        log(f"[log] {rows}x{cols} {kind}: worst error / bound {r:.3f}")


@pytest.mark.parametrize("rows,cols", [(33, 1001), (131, 7), (3, 100003)])
def test_misaligned_and_in_place(rows, cols):
    import torch
    x = workloads.random_logits(rows, cols, seed=cols, kind="clip_heavy")
    n = rows * cols
    xb = torch.empty(n + 4, dtype=torch.float32, device="cuda:0")
    xb[1:n + 1] = torch.from_numpy(x.reshape(-1)).to("cuda:0")
    xv = xb[1:n + 1].view(rows, cols)
    assert sm.softmax_plan(rows, cols, xv.data_ptr(), xv.data_ptr())["vec_width"] == 1
    sm.softmax_log_fwd(xv, NEG_INF, out=xv)          # misaligned and in place
    torch.cuda.synchronize()
    check_log(x, xv.cpu().numpy(), NEG_INF, f"misaligned in place {rows}x{cols}")


@pytest.mark.parametrize("cols", [5, 50, 1000, 8192, 70000])
def test_nonfinite_rows(cols):
    rng = np.random.default_rng(cols + 1)
    x = rng.standard_normal((5, cols)).astype(np.float32)
    x[0, cols // 2] = np.nan
    x[1, cols // 3] = np.inf
    x[2, :] = -np.inf
    x[3, ::2] = -np.inf
    for lo in (-64.0, NEG_INF):
        y = run_log(x, lo)
        assert np.all(np.isnan(y[:3]))
        check_log(x, y, lo, f"nonfinite {cols} lo={lo}")
    assert np.all(run_log(x, NEG_INF)[3, ::2] == -np.inf)


def test_uniform_rows():
    """Uniform rows give -ln N, to within the bound (ln N comes from
    v_log_f32)."""
    for n in (1, 3, 50, 1000, 4096, 32768, 262144):
        x = np.full((2, n), -3.25, dtype=np.float32)
        check_log(x, run_log(x, -64.0), -64.0, f"uniform {n}")
        if n == 1:
            assert np.all(run_log(x, -64.0) == 0.0)


def test_exp_of_log_is_softmax():
    """exp of the log outputs matches softmax_fwd's probabilities."""
    import torch
    x = workloads.generate("classifier_4096x1000")
    ylog = run_log(x, -64.0).astype(np.float64)
    p = sm.softmax_fwd(torch.from_numpy(x).to("cuda:0")).cpu().numpy().astype(np.float64)
    assert np.max(np.abs(np.exp(ylog) - p) / p) <= 2e-5
