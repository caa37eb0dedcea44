"""Dense scan of the kernels' exponential against float64 on the host.

Every fp32 x in [-64, 0] goes through the accurate clipped exponential of
softmax_fwd (softmax_exp_probe with m = 0, so the shift is exact and the
scan measures the exponential itself), and every fp32 t in [-126, 0]
through the bare v_exp_f32 instruction (2^t) that the routine builds on.
The error of each output is measured in units in the last place of the
exact value (the fp32 spacing at |exact|), with the exact value from
float64 exp / exp2 on the host (error far below 2^-29 fp32 ulp).

The clipped exponential's stated bound is 1.5 ulp (sm_device.hpp); the
header states the measured maxima of both (on MI355X: 1.2685 ulp at
x = -8.426096 for the clipped exponential, 0.7827 ulp at t = -0.750096 for
v_exp_f32, and at most 1.2451 ulp on the shifted scans).
"""
import concurrent.futures as cf
import sys

import numpy as np
import pytest

import oracle
import paper_1904_12380_amd as sm

pytestmark = pytest.mark.gpu

CHUNK = 1 << 24          # values per GPU launch and host batch
WORKERS = 8              # host threads (numpy releases the GIL)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def ulp32_of(w: np.ndarray) -> np.ndarray:
    """fp32 spacing at |w| (w > 0, normal in fp32): 2^(floor(log2 w) - 23),
    built from the float64 exponent field so that no rounding to fp32 can
    move it into the next binade."""
    e64 = (w.view(np.int64) >> 52) & 0x7FF
    return ((e64 - 23) << 52).view(np.float64)


def _ulp_err(bits_lo: int, e: np.ndarray, ref) -> tuple[float, int]:
    x = np.arange(bits_lo, bits_lo + e.size, dtype=np.uint32).view(np.float32)
    w = ref(x.astype(np.float64))
    err = np.abs(e.astype(np.float64) - w) / ulp32_of(w)
    i = int(np.argmax(err))
    return float(err[i]), bits_lo + i


def scan(torch, bits_lo: int, bits_hi: int, mode: int, ref) -> tuple[float, int]:
    """Max ulp error of softmax_exp_probe (mode) over the fp32 bit patterns
    [bits_lo, bits_hi) (negative numbers: patterns from 0x80000000 up)."""
    dev = torch.device("cuda:0")
    worst, where = 0.0, bits_lo
    pool = cf.ThreadPoolExecutor(WORKERS)
    futs = []
    for lo in range(bits_lo, bits_hi, CHUNK):
        n = min(CHUNK, bits_hi - lo)
        # bit patterns as int32 (they are >= 2^31, so shift into range first)
        xb = torch.arange(lo - (1 << 32), lo - (1 << 32) + n, dtype=torch.int64, device=dev)
        x = xb.to(torch.int32).view(torch.float32)
        m = torch.zeros_like(x) if mode != 2 else None
        e = sm.softmax_exp_probe(x, m, approx=mode).cpu().numpy()
        futs.append(pool.submit(_ulp_err, lo, e, ref))
        while len(futs) > 2 * WORKERS:
            err, at = futs.pop(0).result()
            if err > worst:
                worst, where = err, at
    for f in futs:
        err, at = f.result()
        if err > worst:
            worst, where = err, at
    pool.shutdown()
    return worst, where


def _f32(bits: int) -> float:
    return float(np.array([bits], dtype=np.uint32).view(np.float32)[0])


def test_clipped_exp_dense_scan():
    """Every fp32 x in [-64, 0]: exp(max(x - 0, -64)) within 1.5 ulp."""
    import torch
    lo, hi = 0x80000000, 0xC2800000 + 1      # -0 ... -64
    log(f"[exp scan] clipped exp, {hi - lo} values")
    worst, at = scan(torch, lo, hi, 0, oracle.exp_clipped)
    log(f"[exp scan] clipped exp: max {worst:.4f} ulp at x = {_f32(at)!r}")
    assert worst <= 1.5


def _ordered(f: np.float32) -> int:
    """fp32 -> integer preserving order (-0 and +0 both map to 0)."""
    b = int(np.array([f], dtype=np.float32).view(np.uint32)[0])
    return b if b < 0x80000000 else -(b & 0x7FFFFFFF)


def _from_ordered(k: np.ndarray) -> np.ndarray:
    bits = np.where(k >= 0, k, 0x80000000 | (-k)).astype(np.uint32)
    return bits.view(np.float32)


def test_clipped_exp_scan_with_shift():
    """x - m not representable in fp32: every 128th fp32 x of [m - 64, m]
    for a few row maxima m (the binary64 shift of the routine)."""
    import torch
    dev = torch.device("cuda:0")
    worst = 0.0
    for mval in (37.25, -12.125, 1000.5, 3.0e-3, -57.75):
        m32 = np.float32(mval)
        lo32 = np.float32(float(m32) - 64.0)
        k = np.arange(_ordered(lo32), _ordered(m32) + 1, 128, dtype=np.int64)
        x = _from_ordered(k)
        xt = torch.from_numpy(np.ascontiguousarray(x)).to(dev)
        mt = torch.full_like(xt, float(m32))
        e = sm.softmax_exp_probe(xt, mt).cpu().numpy().astype(np.float64)
        w = oracle.exp_clipped(x.astype(np.float64) - np.float64(m32))
        err = float(np.max(np.abs(e - w) / ulp32_of(w)))
        log(f"[exp scan] m = {mval}: {x.size} values, max {err:.4f} ulp")
        worst = max(worst, err)
    assert worst <= 1.5


def test_v_exp_f32_dense_scan():
    """Every fp32 t in [-126, 0] through the bare v_exp_f32: its error
    against 2^t, the figure the header states."""
    import torch
    lo, hi = 0x80000000, 0xC2FC0000 + 1      # -0 ... -126
    log(f"[exp scan] v_exp_f32, {hi - lo} values")
    worst, at = scan(torch, lo, hi, 2, np.exp2)
    log(f"[exp scan] v_exp_f32: max {worst:.4f} ulp at t = {_f32(at)!r}")
    assert worst <= 1.0
