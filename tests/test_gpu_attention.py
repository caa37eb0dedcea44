"""GPU parity for the fused softmax attention (softmax_attention_fwd) through
the C ABI, against the float64 oracle ``oracle.attention_clipped``.

Bar, derived from the arithmetic (fp32 matrix-core products, the library's
softmax): with u = 2^-24, per query i

    delta_i = (d + 2) u * max_k |scale| sum_t |Q_it K_kt|      (score error)

bounds the absolute error of every score of row i, so each weight is within
a relative 2 delta_i + 4e-6 of the exact weight (the 4e-6 is the softmax
bar), and each output within

    (2 delta_i + 4e-6 + (lk + 2) u) * sum_k P_ik |V_kc|  +  2^-148

of the exact output (the last term covers denormal outputs without a clip).
"""
import sys

import numpy as np
import pytest

import oracle
import paper_1904_12380_amd as sm
import workloads

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def _torch():
    import torch
    return torch


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_attn(q, k, v, scale, lo=-64.0):
    torch = _torch()
    dev = "cuda:0"
    o = sm.softmax_attention_fwd(torch.from_numpy(q).to(dev), torch.from_numpy(k).to(dev),
                                 torch.from_numpy(v).to(dev), scale=scale, clip_lo=lo)
    torch.cuda.synchronize()
    return o.cpu().numpy()


def bound(q, k, v, scale, lo):
    """Per-element error bound of the docstring, and the float64 oracle."""
    q64, k64, v64 = (a.astype(np.float64) for a in (q, k, v))
    want = oracle.attention_clipped(q, k, v, scale, lo)
    lk, d = k.shape[1], q.shape[2]
    absdot = np.abs(scale) * np.matmul(np.abs(q64), np.abs(k64).transpose(0, 2, 1))
    delta = (d + 2) * U * absdot.max(axis=2, keepdims=True)           # [b, lq, 1]
    s = np.matmul(q64, k64.transpose(0, 2, 1)) * float(scale)
    p = oracle.softmax_clipped(s.reshape(-1, lk), lo).reshape(s.shape)
    mass = np.matmul(p, np.abs(v64))                                   # sum_k P |V|
    tol = (2.0 * delta + 4e-6 + (lk + 2) * U) * mass + 2.0 ** -148
    return want, tol


def check(q, k, v, scale, lo, what):
    got = run_attn(q, k, v, scale, lo).astype(np.float64)
    want, tol = bound(q, k, v, scale, lo)
    assert got.shape == want.shape, what
    assert np.array_equal(np.isnan(got), np.isnan(want)), what
    fin = np.isfinite(want)
    err = np.abs(got[fin] - want[fin])
    if np.any(err > tol[fin]):
        i = int(np.argmax(err / tol[fin]))
        idx = np.unravel_index(np.flatnonzero(fin)[i], want.shape)
        pytest.fail(f"{what}: err {err[i]:.3e} > bound {tol[fin][i]:.3e} at {idx}: "
                    f"got {got[idx]!r} want {want[idx]!r}")
    ratio = float((err / tol[fin]).max()) if err.size else 0.0
    rel = float((err / np.maximum(np.abs(want[fin]), 1e-30)).max()) if err.size else 0.0
    return ratio, rel


def test_dam_workload():
    key = "dam_fused_attention_2304x50x50x200"
    w = workloads.ATTENTION_WORKLOADS[key]
    log(f"[attn] {key}")
    q, k, v = workloads.generate_qkv(key)
    ratio, rel = check(q, k, v, w.scale, -64.0, key)
    log(f"[attn] {key}: worst error / bound {ratio:.3e}, worst rel {rel:.3e}")


# (batch, lq, lk, d, dv): DAM tile, every key-tile count, query blocks past
# 64, d and dv that are not multiples of 4 or 16 (32-bit loads), one-element
# problems and long value rows; last key tiles of 1 to 4 keys (scores of
# those keys on the VALU) and of more (matrix ops).
SHAPES = [(3, 50, 50, 200, 200), (2, 64, 64, 64, 64), (4, 16, 16, 16, 16), (5, 65, 17, 33, 7),
          (7, 3, 5, 8, 250), (2, 100, 64, 128, 16), (1, 1, 64, 1, 1), (1, 1, 1, 1, 1),
          (9, 48, 32, 20, 3), (2, 130, 49, 12, 70), (3, 7, 33, 300, 5),
          (2, 40, 52, 64, 64), (3, 17, 35, 24, 40), (2, 33, 4, 16, 8),
          # the DAM tile with d = dv = 200 known at compile time (ping-pong
          # schedule): 49 and 50 keys, one query, query blocks past 64, and
          # more items than CUs (workgroups of 1, 2 and 3 items)
          (5, 50, 49, 200, 200), (2, 1, 50, 200, 200), (3, 130, 50, 200, 200),
          (4, 64, 49, 200, 200), (600, 50, 50, 200, 200), (300, 100, 49, 200, 200)]


@pytest.mark.parametrize("b,lq,lk,d,dv", SHAPES)
def test_shapes(b, lq, lk, d, dv):
    log(f"[attn] shape {b}x{lq}x{lk}x{d}x{dv}")
    q, k, v = workloads.random_qkv(b, lq, lk, d, dv, seed=b * 1000 + lq + lk + d + dv)
    scale = float(np.float32(1.0 / np.sqrt(d)))
    ratio, _ = check(q, k, v, scale, -64.0, f"{b}x{lq}x{lk}x{d}x{dv}")
    log(f"[attn] {b}x{lq}x{lk}x{d}x{dv}: worst error / bound {ratio:.3e}")


@pytest.mark.parametrize("lo", [-64.0, -90.0, float("-inf")])
def test_clip_active(lo):
    """Large scores, so that many weights fall below the clip (or to 0)."""
    q, k, v = workloads.random_qkv(6, 50, 50, 64, 40, seed=17, scale=4.0)
    ratio, _ = check(q, k, v, 1.0, lo, f"clip {lo}")
    log(f"[attn] clip {lo}: worst error / bound {ratio:.3e}")


def test_zero_dimension_scores():
    """d = 0: every score is 0, so each output row is the mean of V's rows."""
    torch = _torch()
    b, lq, lk, dv = 3, 10, 7, 5
    v = workloads.random_qkv(b, 1, lk, 1, dv, seed=3)[2]
    vt = torch.from_numpy(v).to("cuda:0")
    e = torch.empty((b, lq, 0), device="cuda:0")
    ke = torch.empty((b, lk, 0), device="cuda:0")
    o = sm.softmax_attention_fwd(e, ke, vt, scale=1.0).cpu().numpy().astype(np.float64)
    want = np.broadcast_to(v.astype(np.float64).mean(axis=1, keepdims=True), o.shape)
    assert np.max(np.abs(o - want)) <= 1e-6 * np.max(np.abs(want))


def test_misaligned_inputs():
    """q and k 4 bytes past a 16-byte boundary: the 32-bit load path."""
    torch = _torch()
    b, lq, lk, d, dv = 4, 50, 50, 200, 200
    q, k, v = workloads.random_qkv(b, lq, lk, d, dv, seed=23)
    dev = "cuda:0"

    def shifted(a):
        buf = torch.empty(a.size + 4, dtype=torch.float32, device=dev)
        buf[1:a.size + 1] = torch.from_numpy(a.reshape(-1)).to(dev)
        return buf[1:a.size + 1].view(a.shape)

    qs, ks = shifted(q), shifted(k)
    assert qs.data_ptr() % 16 == 4
    scale = float(np.float32(1.0 / np.sqrt(d)))
    o = sm.softmax_attention_fwd(qs, ks, torch.from_numpy(v).to(dev), scale=scale)
    torch.cuda.synchronize()
    got = o.cpu().numpy().astype(np.float64)
    want, tol = bound(q, k, v, scale, -64.0)
    assert np.all(np.abs(got - want) <= tol)


def test_nonfinite_inputs():
    """A NaN in a query row makes that output row NaN; an inf in V makes its
    column NaN or inf exactly where the oracle's is."""
    q, k, v = workloads.random_qkv(2, 20, 30, 16, 8, seed=29)
    q[0, 3, 5] = np.nan
    v[1, 7, 2] = np.inf
    got = run_attn(q, k, v, 0.25)
    want = oracle.attention_clipped(q, k, v, 0.25)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    assert np.array_equal(np.isinf(got), np.isinf(want))
    assert np.all(np.isnan(got[0, 3]))


def test_nonfinite_inputs_dam_tile():
    """The same on the DAM tile (50 keys, d = dv = 200): padding keys read a
    zero row, and an inf in the first columns of a key row must not reach
    the previous key's score through the masked last block of d."""
    q, k, v = workloads.random_qkv(3, 50, 50, 200, 200, seed=31)
    q[0, 7, 199] = np.nan
    k[1, 12, 3] = np.inf
    v[2, 49, 150] = -np.inf
    got = run_attn(q, k, v, float(np.float32(1.0 / np.sqrt(200))))
    want = oracle.attention_clipped(q, k, v, float(np.float32(1.0 / np.sqrt(200))))
    assert np.array_equal(np.isnan(got), np.isnan(want))
    assert np.array_equal(np.isinf(got), np.isinf(want))
    fin = np.isfinite(want)
    assert np.all(np.abs(got[fin] - want[fin]) <= 1e-4 * np.abs(want[fin]).max())
    assert np.all(np.isnan(got[0, 7]))


def test_deterministic_and_graph_replay():
    torch = _torch()
    q, k, v = (torch.from_numpy(a).to("cuda:0") for a in
               workloads.generate_qkv("dam_fused_attention_2304x50x50x200"))
    a = sm.softmax_attention_fwd(q, k, v)
    b = sm.softmax_attention_fwd(q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    og = torch.empty_like(a)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        sm.softmax_attention_fwd(q, k, v, out=og, stream=s)
    for rep in range(3):
        og.fill_(-1.0)
        sm.softmax_attention_fwd(q, k, v, out=b)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(og.view(torch.int32), a.view(torch.int32)), rep


def test_bad_arguments_raise():
    torch = _torch()
    q = torch.zeros(2, 5, 8, device="cuda:0")
    k = torch.zeros(2, 65, 8, device="cuda:0")
    v = torch.zeros(2, 65, 4, device="cuda:0")
    with pytest.raises(sm.SoftmaxError):
        sm.softmax_attention_fwd(q, k, v)              # 65 keys
    with pytest.raises(sm.SoftmaxError):
        sm.softmax_attention_fwd(q, k[:, :8].contiguous(), v[:, :8].contiguous(),
                                 scale=float("nan"))
