"""GPU parity for the fused negative log-likelihood (softmax_nll_fwd),
through the C ABI, against ``oracle.nll_clipped``.

Bar, from the arithmetic (the loss is minus one log-softmax output, and
negation is exact): per row

    |loss - loss*| <= 2e-6 + 2.5e-7 * (|loss*| + ln(cols)),

+inf exactly where the oracle gives +inf and NaN exactly where it gives NaN
(labels outside the row, NaN rows).  The loss is also checked against
minus softmax_log_fwd's output at the label: bit for bit where both modes
take the same row sum.
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


def run_nll(x, labels, lo):
    import torch
    xt = torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")
    lt = torch.from_numpy(np.ascontiguousarray(labels, dtype=np.int64)).to("cuda:0")
    y = sm.softmax_nll_fwd(xt, lt, lo)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check_nll(x, labels, loss, lo, what):
    want = oracle.nll_clipped(x, labels, lo)
    got = loss.astype(np.float64)
    assert got.shape == want.shape, what
    assert np.array_equal(np.isnan(got), np.isnan(want)), what
    assert np.array_equal(np.isposinf(got), np.isposinf(want)), what
    fin = np.isfinite(want)
    err = np.abs(got[fin] - want[fin])
    bound = 2e-6 + 2.5e-7 * (np.abs(want[fin]) + math.log(max(x.shape[1], 1)))
    if err.size and np.any(err > bound):
        k = int(np.argmax(err / bound))
        i = np.flatnonzero(fin)[k]
        pytest.fail(f"{what} lo={lo}: err {err[k]:.3e} > {bound[k]:.3e} at row {i}: "
                    f"got {got[i]!r} want {want[i]!r} (label {labels[i]})")
    return float((err / bound).max()) if err.size else 0.0


@pytest.mark.parametrize("key", list(workloads.WORKLOADS))
def test_workloads(key):
    x = workloads.generate(key)
    t = workloads.generate_labels(key)
    for lo in (-64.0, NEG_INF):
        r = check_nll(x, t, run_nll(x, t, lo), lo, key)
        log(f"[nll] {key} lo={lo}: worst error / bound {r:.3f}")


# Every kernel bucket: packed rows (G = 1, 2, 4), one wavefront per row,
# one workgroup per row, one-pass split rows (both chunk sizes) and the
# two-pass fallback.
SHAPES = [(1000, 50), (257, 7), (130, 17), (64, 64), (64, 1000), (9, 3000), (5, 8192),
          (3, 100003), (2, 1048577), (1, 2097153)]


@pytest.mark.parametrize("rows,cols", SHAPES)
def test_shapes(rows, cols):
    rng = np.random.default_rng(rows * 7 + cols)
    for kind in ("clip_heavy", "normal", "offset"):
        x = workloads.random_logits(rows, cols, seed=rows * 13 + cols, kind=kind, scale=30.0)
        t = rng.integers(0, cols, size=rows, dtype=np.int64)
        t[0] = 0
        t[-1] = cols - 1
        for lo in (-64.0, -90.0, NEG_INF):
            r = check_nll(x, t, run_nll(x, t, lo), lo, f"{rows}x{cols} {kind}")
        log(f"[nll] {rows}x{cols} {kind}: worst error / bound {r:.3f}")


@pytest.mark.parametrize("rows,cols", [(33, 1001), (131, 7), (3, 100003), (2, 40000)])
def test_misaligned_rows(rows, cols):
    """x 4 bytes past a 16-byte boundary: the 32-bit access paths."""
    import torch
    x = workloads.random_logits(rows, cols, seed=cols, kind="clip_heavy")
    t = np.random.default_rng(cols).integers(0, cols, size=rows, dtype=np.int64)
    n = rows * cols
    xb = torch.empty(n + 4, dtype=torch.float32, device="cuda:0")
    xb[1:n + 1] = torch.from_numpy(x.reshape(-1)).to("cuda:0")
    xv = xb[1:n + 1].view(rows, cols)
    assert sm.softmax_plan(rows, cols, xv.data_ptr(), xv.data_ptr())["vec_width"] == 1
    loss = sm.softmax_nll_fwd(xv, torch.from_numpy(t).to("cuda:0"), NEG_INF)
    torch.cuda.synchronize()
    check_nll(x, t, loss.cpu().numpy(), NEG_INF, f"misaligned {rows}x{cols}")


@pytest.mark.parametrize("cols", [5, 50, 1000, 8192, 70000])
def test_labels_out_of_range_and_nonfinite_rows(cols):
    rng = np.random.default_rng(cols + 3)
    x = rng.standard_normal((8, cols)).astype(np.float32)
    x[0, cols // 2] = np.nan
    x[1, cols // 3] = np.inf
    x[2, :] = -np.inf
    x[3, 1] = -np.inf
    t = np.array([0, 0, 0, 1, -1, cols, 1 << 40, cols - 1], dtype=np.int64)
    for lo in (-64.0, NEG_INF):
        y = run_nll(x, t, lo)
        assert np.all(np.isnan(y[:3])) and np.all(np.isnan(y[4:7])) and np.isfinite(y[7])
        check_nll(x, t, y, lo, f"nonfinite {cols} lo={lo}")
    assert run_nll(x, t, NEG_INF)[3] == np.inf


@pytest.mark.parametrize("key", ["dam_attention_115200x50", "classifier_4096x1000",
                                 "vocab_512x32768", "longrow_64x262144"])
def test_minus_log_softmax_at_label(key):
    """The loss is minus softmax_log_fwd's output at the label: bit for bit
    where both modes take the same row sum, and within the shared bound
    where they do not: on the 1024-thread row kernel (vocab rows), where the
    NLL folds its sums in as the loads land and the log mode reduces the
    loaded row, and on long rows, where the NLL's one-pass chunks are twice
    as wide."""
    import torch
    x = torch.from_numpy(workloads.generate(key)).to("cuda:0")
    t = torch.from_numpy(workloads.generate_labels(key)).to("cuda:0")
    cols = x.shape[1]
    for lo in (-64.0, NEG_INF):
        loss = sm.softmax_nll_fwd(x, t, lo)
        ylog = sm.softmax_log_fwd(x, lo)
        picked = ylog.gather(1, t.view(-1, 1)).view(-1)
        torch.cuda.synchronize()
        if key not in ("vocab_512x32768", "longrow_64x262144"):
            assert torch.equal(loss.view(torch.int32), (-picked).view(torch.int32)), (key, lo)
        else:
            a = loss.double().cpu().numpy()
            b = (-picked).double().cpu().numpy()
            bound = 2.0 * (2e-6 + 2.5e-7 * (np.abs(a) + math.log(cols)))
            assert np.all(np.abs(a - b) <= bound), (key, lo)


@pytest.mark.parametrize("rows,cols", [(3, 100003), (64, 262144), (2, 1048580), (70, 500000)])
def test_long_rows_interleaved_with_other_modes(rows, cols):
    """Long rows of every mode share the exchange table: each launch claims a
    region and the last of its workgroups returns it to rest (for the loss,
    the merging workgroup), so softmax, log-softmax and loss calls in any
    order on one stream all stay within their bounds, and afterwards no wait
    gave up and no region is left claimed.  70 x 500000 takes several
    one-pass launches per call."""
    import torch
    x = workloads.random_logits(rows, cols, seed=cols + rows, kind="clip_heavy")
    t = np.random.default_rng(cols).integers(0, cols, size=rows, dtype=np.int64)
    xt = torch.from_numpy(x).to("cuda:0")
    tt = torch.from_numpy(t).to("cuda:0")
    want_nll = oracle.nll_clipped(x, t, -64.0)
    sample = np.random.default_rng(rows).integers(0, rows, size=min(rows, 2))
    want_y = oracle.softmax_clipped(x[sample], -64.0)
    for rep in range(3):
        loss = sm.softmax_nll_fwd(xt, tt)
        y = sm.softmax_fwd(xt)
        loss2 = sm.softmax_nll_fwd(xt, tt)
        ylog = sm.softmax_log_fwd(xt)
        torch.cuda.synchronize()
        assert torch.equal(loss.view(torch.int32), loss2.view(torch.int32)), rep
        check_nll(x, t, loss.cpu().numpy(), -64.0, f"interleaved {rows}x{cols} rep {rep}")
        got = y.cpu().numpy()[sample].astype(np.float64)
        assert np.all(np.abs(got - want_y) <= 4e-6 * want_y), rep
        picked = ylog.gather(1, tt.view(-1, 1)).view(-1)
        a = loss.double().cpu().numpy()
        b = (-picked).double().cpu().numpy()
        bound = 2.0 * (2e-6 + 2.5e-7 * (np.abs(a) + math.log(cols)))
        assert np.all(np.abs(a - b) <= bound), rep
    torch.cuda.synchronize()
    st = sm.softmax_exchange_status()
    assert st == {"join_give_ups": 0, "wait_give_ups": 0, "entries_in_use": 0}, st


def test_uniform_rows():
    """Uniform rows give ln N for every label, within the bound."""
    for n in (1, 3, 50, 1000, 4096, 32768, 262144):
        x = np.full((3, n), 2.5, dtype=np.float32)
        t = np.array([0, n // 2, n - 1], dtype=np.int64)
        check_nll(x, t, run_nll(x, t, -64.0), -64.0, f"uniform {n}")


def test_deterministic_and_graph_replay():
    import torch
    key = "vocab_512x32768"
    x = torch.from_numpy(workloads.generate(key)).to("cuda:0")
    t = torch.from_numpy(workloads.generate_labels(key)).to("cuda:0")
    a = sm.softmax_nll_fwd(x, t)
    b = sm.softmax_nll_fwd(x, t)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    og = torch.empty_like(a)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        sm.softmax_nll_fwd(x, t, out=og, stream=s)
    for rep in range(3):
        og.fill_(-1.0)
        sm.softmax_nll_fwd(x, t, out=b)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(og.view(torch.int32), a.view(torch.int32)), rep


def test_bad_arguments_raise():
    import torch
    x = torch.zeros(4, 8, device="cuda:0")
    t = torch.zeros(4, dtype=torch.int64, device="cuda:0")
    with pytest.raises(sm.SoftmaxError):
        sm.softmax_nll_fwd(x, t, clip_lo=-1.0)
    with pytest.raises(sm.SoftmaxError):
        sm.softmax_nll_fwd(torch.zeros(4, 0, device="cuda:0"), t)
    with pytest.raises(TypeError):
        sm.softmax_nll_fwd(x, t.to(torch.int32))
    with pytest.raises(ValueError):
        sm.softmax_nll_fwd(x, t[:3])
