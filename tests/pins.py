"""Pins for any implementation of the clipped row softmax.

Each ``pin_*`` function takes ``impl(x: float32 [R, C]) -> float64 [R, C]``
and raises AssertionError when ``impl`` violates a fact fixed by the paper or
by mathematics, not by the oracle's own code:

  * closed forms of the definition (Sec. 1.1 Eq. (1); Sec. 1.2 Fig. 1 with
    the -64 clip of the shifted logits, Sec. 2.1);
  * the two-class special case, which is the logistic function (Sec. 1.1
    calls softmax the multi-class extension of logistic regression), checked
    against ``scipy.special.expit``;
  * a 50-digit ``decimal`` brute force stored in ``tests/golden``;
  * ``torch.softmax`` in float64 where the clip is inactive;
  * invariants: uniform rows, exact shift invariance on dyadic grids, row
    sums, permutation equivariance, monotonicity and the clip's lower bound;
  * the non-finite-input reading.

``tests/test_oracle_pins.py`` runs them on the oracle and
``tests/test_oracle_mutants.py`` shows that planted mistakes fail them.
"""
from __future__ import annotations

import json
import math
import os
from decimal import Decimal

import numpy as np

from workloads import random_logits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
E64 = math.exp(-64.0)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _rel(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b) / np.abs(b)))


def pin_uniform_rows(impl):
    """Equal logits give exactly 1/N (Eq. (1) with all terms equal)."""
    for n in (1, 2, 3, 7, 50, 1000, 4097):
        for v in (0.0, -5.25, 17.0, -1.0e4):
            y = impl(_f32(np.full((3, n), v)))
            assert y.shape == (3, n)
            assert np.all(y == 1.0 / n), (n, v)


def pin_single_class(impl):
    """C = 1 gives exactly 1 for any finite logit."""
    y = impl(_f32([[3.0], [-1.0e4], [0.0], [65.5]]))
    assert np.all(y == 1.0)


def pin_two_class_logistic(impl):
    """C = 2 reduces to the logistic function sigma(a - b) (Sec. 1.1)."""
    from scipy.special import expit
    rng = np.random.default_rng(5)
    a = rng.uniform(-30.0, 30.0, 200)
    b = rng.uniform(-30.0, 30.0, 200)
    x = _f32(np.stack([a, b], axis=1))
    y = impl(x)
    diff = x[:, 0].astype(np.float64) - x[:, 1].astype(np.float64)
    assert _rel(y[:, 0], expit(diff)) < 1e-14
    assert _rel(y[:, 1], expit(-diff)) < 1e-14
    # Beyond the clip: the smaller class is held at e^-64 / (1 + e^-64).
    x = _f32([[0.0, -100.0], [-100.0, 0.0], [5.0, -70.0]])
    y = impl(x)
    lo, hi = E64 / (1.0 + E64), 1.0 / (1.0 + E64)
    assert _rel([y[0, 1], y[1, 0], y[2, 1]], [lo, lo, lo]) < 1e-14
    assert _rel([y[0, 0], y[1, 1], y[2, 0]], [hi, hi, hi]) < 1e-15


def pin_clip_closed_form(impl):
    """The clip of Fig. 1 on the shifted logits, in closed form.

    Row [0, -100, -64, -63.5, -1e4]: clipped shifts [0, -64, -64, -63.5, -64]
    and S = 1 + 3 e^-64 + e^-63.5.  The same row with a common offset and in
    every rotation must give the same (rotated) values."""
    base = np.array([0.0, -100.0, -64.0, -63.5, -1.0e4])
    s = 1.0 + 3.0 * E64 + math.exp(-63.5)
    want = np.array([1.0, E64, E64, math.exp(-63.5), E64]) / s
    for off in (0.0, 37.25, -20.5):
        for r in range(5):
            x = _f32(np.roll(base + off, r)[None, :])
            y = impl(x)[0]
            assert _rel(y, np.roll(want, r)) < 1e-14, (off, r)


def pin_brute_force_decimal(impl):
    """Tiny rows against a 50-digit decimal evaluation (tests/golden)."""
    with open(os.path.join(GOLDEN, "brute_force_rows.json")) as f:
        doc = json.load(f)
    for rec in doc["rows"]:
        x = _f32([[float.fromhex(h) for h in rec["x_hex"]]])
        y = impl(x)[0]
        want = np.array([float(Decimal(v)) for v in rec["y"]])
        assert _rel(y, want) < 1e-14, rec["x_hex"]
        if "y_eq1" in rec:
            want1 = np.array([float(Decimal(v)) for v in rec["y_eq1"]])
            assert _rel(y, want1) < 1e-14


def pin_library_unclipped(impl):
    """Where no shifted logit is below -64, torch.softmax (float64) agrees."""
    import torch
    for (r, c, seed) in ((4, 1000, 1), (33, 50, 2), (2, 5000, 3)):
        x = random_logits(r, c, seed, "normal", 4.0)
        want = torch.softmax(torch.from_numpy(x).double(), dim=-1).numpy()
        assert _rel(impl(x), want) < 1e-13


def pin_shift_invariance(impl):
    """Adding k to a dyadic row leaves every shifted logit bit-identical, so
    the output must be bit-identical too."""
    x = random_logits(6, 257, 7, "dyadic")
    y0 = impl(x)
    for k in (0.5, 2.0, 64.0, 1024.0, -256.0):
        xk = _f32(x.astype(np.float64) + k)
        assert np.array_equal(xk.astype(np.float64) - k, x.astype(np.float64))
        assert np.array_equal(impl(xk), y0), k


def pin_row_sums(impl):
    """Every row sums to 1 (up to float64 rounding)."""
    for (r, c, kind, seed) in ((8, 1000, "normal", 11), (3, 262144, "offset", 12),
                              (16, 50, "clip_heavy", 13), (5, 4099, "uniform", 14)):
        y = impl(random_logits(r, c, seed, kind))
        for row in y:
            assert abs(math.fsum(row) - 1.0) < 1e-13


def pin_permutation_equivariance(impl):
    """Permuting classes permutes the outputs."""
    x = random_logits(4, 301, 21, "clip_heavy")
    perm = np.random.default_rng(22).permutation(301)
    assert _rel(impl(x[:, perm]), impl(x)[:, perm]) < 1e-14


def pin_axis_is_rows(impl):
    """Normalisation runs along each row of a non-square [R, C] matrix."""
    x = random_logits(7, 3, 23, "normal")
    y = impl(x)
    assert y.shape == (7, 3)
    assert np.allclose(y.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert not np.allclose(y.sum(axis=0), 1.0, atol=1e-3)


def pin_monotonicity(impl):
    """Raising one logit never lowers its own output nor raises another's;
    it raises its own output strictly once the raised logit is unclipped."""
    x = random_logits(1, 40, 31, "clip_heavy")
    y0 = impl(x)[0]
    for j in (0, 5, 17, 39):
        x1 = x.copy()
        x1[0, j] += np.float32(3.0)
        y1 = impl(x1)[0]
        others = np.arange(40) != j
        assert y1[j] >= y0[j]
        assert np.all(y1[others] <= y0[others] * (1 + 1e-15))
        if x1[0, j] - x.max() > -64.0:
            assert y1[j] > y0[j]


def pin_lower_bound(impl):
    """The clip keeps every output at or above e^-64 / C (Sec. 2.1: no
    zeros), with equality for clipped entries of a row whose other entries
    are all at the max."""
    x = random_logits(32, 64, 41, "clip_heavy")
    y = impl(x)
    assert np.all(y >= E64 / 64 * (1 - 1e-14))
    x = _f32([[0.0] * 3 + [-500.0]])
    y = impl(x)[0]
    assert _rel(y[3], E64 / (3.0 + E64)) < 1e-14


def pin_nonfinite(impl):
    """Reading of non-finite inputs: NaN or +inf poisons the row; -inf clips
    to e^-64; an all -inf row is NaN."""
    x = _f32([[1.0, np.nan, 0.0],
              [1.0, np.inf, 0.0],
              [-np.inf, -np.inf, -np.inf],
              [0.0, -np.inf, 0.0],
              [0.0, 1.0, 2.0]])
    y = impl(x)
    assert np.all(np.isnan(y[0])) and np.all(np.isnan(y[1]))
    assert np.all(np.isnan(y[2]))
    s = 2.0 + E64
    assert _rel(y[3], [1 / s, E64 / s, 1 / s]) < 1e-14
    assert np.all(np.isfinite(y[4]))


def pin_empty(impl):
    """Empty inputs give empty outputs of the same shape."""
    for shape in ((0, 5), (5, 0), (0, 0)):
        y = impl(np.zeros(shape, dtype=np.float32))
        assert y.shape == shape


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]


# ---------------------------------------------------------------------------
# Pins for the clip bound as a parameter.  Each ``pinc_*`` function takes
# ``impl(x: float32 [R, C], clip_lo: float) -> float64 [R, C]``; clip_lo is
# the lower bound on the shifted logits, and -inf means no clip (the
# optimised functor of Sec. 2.3 Fig. 4, which drops the ValueClip of Fig. 1;
# Sec. 2.1 gives the clip's purpose and its removal).  Outputs can then be
# tiny or 0, so values are compared with a relative bound above 1e-290 and
# an absolute one below.

def _close(got, want, rel=1e-14, tiny=1e-290) -> bool:
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    big = np.abs(want) >= tiny
    ok_big = np.all(np.abs(got[big] - want[big]) <= rel * np.abs(want[big]))
    ok_small = np.all(np.abs(got[~big] - want[~big]) <= tiny)
    return bool(ok_big and ok_small)


def pinc_minus_64_passes_the_default_pins(impl):
    """At clip_lo = -64 the function satisfies every pin of the default
    bound (closed forms, brute force, invariants, non-finite reading)."""
    for pin in ALL_PINS:
        pin(lambda x: impl(x, -64.0))


def pinc_clip_off_matches_library(impl):
    """With no clip the result is plain softmax: scipy.special.softmax in
    float64, on rows whose shifted logits go far below -64 (where any clip
    would change the result) and rows with offsets large enough that exp
    overflows unless the max is subtracted first."""
    from scipy.special import softmax as sp_softmax
    rng = np.random.default_rng(52)
    rows = [rng.uniform(-700.0, 0.0, 64), rng.uniform(-150.0, 10.0, 64),
            800.0 + rng.standard_normal(64), -900.0 + 40.0 * rng.standard_normal(64)]
    x = _f32(np.stack(rows))
    want = sp_softmax(x.astype(np.float64), axis=1)
    y = impl(x, -np.inf)
    assert _close(y, want), "clip off differs from plain softmax"
    assert np.any(y < math.exp(-64.0) / 64), "some outputs must fall below the -64 clip"


def pinc_closed_form(impl):
    """Row [0, L-1, L, L+0.5, -1e4] with bound L: clipped shifts
    [0, L, L, L+0.5, L], S = 1 + 3 e^L + e^(L+0.5); with offsets and in every
    rotation."""
    for lo in (-48.0, -80.5, -100.0, -120.0):
        base = np.array([0.0, lo - 1.0, lo, lo + 0.5, -1.0e4])
        el = math.exp(lo)
        s = 1.0 + 3.0 * el + math.exp(lo + 0.5)
        want = np.array([1.0, el, el, math.exp(lo + 0.5), el]) / s
        for off in (0.0, 37.25, -20.5):
            for r in range(5):
                y = impl(_f32(np.roll(base + off, r)[None, :]), lo)[0]
                assert _close(y, np.roll(want, r)), (lo, off, r)


def pinc_two_class(impl):
    """C = 2 with bound L: the smaller class is e^max(b-a, L) / (1 + that)."""
    from scipy.special import expit
    rng = np.random.default_rng(53)
    a = rng.uniform(-30.0, 30.0, 100)
    b = a - rng.uniform(0.0, 140.0, 100)
    x = _f32(np.stack([a, b], axis=1))
    diff = x[:, 0].astype(np.float64) - x[:, 1].astype(np.float64)
    for lo in (-48.0, -90.0, -np.inf):
        y = impl(x, lo)
        t = np.maximum(-diff, lo)
        assert _close(y[:, 1], np.exp(t) / (1.0 + np.exp(t)))
        assert _close(y[:, 0], expit(-t))


def pinc_brute_force_decimal(impl):
    """Tiny rows against 50-digit decimal at bounds -48, -90, -120 and with
    no clip (tests/golden, y_clip)."""
    with open(os.path.join(GOLDEN, "brute_force_rows.json")) as f:
        doc = json.load(f)
    for rec in doc["rows"]:
        x = _f32([[float.fromhex(h) for h in rec["x_hex"]]])
        for key, vals in rec["y_clip"].items():
            lo = -np.inf if key == "-inf" else float(key)
            want = np.array([float(Decimal(v)) for v in vals])
            assert _close(impl(x, lo)[0], want), (rec["x_hex"], key)


def pinc_lower_bound(impl):
    """Every output is at least e^L / C for a finite bound L; with no clip,
    outputs whose shifted logit is below ln(2^-1074) are exactly 0."""
    x = random_logits(16, 64, 54, "clip_heavy")
    for lo in (-48.0, -90.0):
        assert np.all(impl(x, lo) >= math.exp(lo) / 64 * (1 - 1e-14))
    y = impl(_f32([[0.0, -800.0, -1.0e4, 0.0]]), -np.inf)[0]
    assert y[1] == 0.0 and y[2] == 0.0 and y[0] == 0.5 and y[3] == 0.5


def pinc_nonfinite_clip_off(impl):
    """With no clip: a -inf element gives exactly 0; NaN, +inf and all -inf
    rows are NaN."""
    x = _f32([[1.0, np.nan, 0.0],
              [1.0, np.inf, 0.0],
              [-np.inf, -np.inf, -np.inf],
              [0.0, -np.inf, 0.0]])
    y = impl(x, -np.inf)
    assert np.all(np.isnan(y[:3]))
    assert y[3, 1] == 0.0 and y[3, 0] == 0.5 and y[3, 2] == 0.5


def pinc_bound_is_monotone(impl):
    """Lowering the bound never raises an output that was clipped, and an
    element above both bounds keeps its share of the unclipped mass."""
    x = random_logits(6, 200, 55, "clip_heavy")
    d = x.astype(np.float64) - x.max(axis=1, keepdims=True)
    y48, y90 = impl(x, -48.0), impl(x, -90.0)
    clipped = d < -48.0
    assert np.all(y90[clipped] <= y48[clipped] * (1 + 1e-14))
    free = d >= -48.0
    assert np.all(y90[free] >= y48[free] * (1 - 1e-14))


CLIP_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pinc_")]


# ---------------------------------------------------------------------------
# Pins for the log of the clipped softmax.  Each ``pinl_*`` function takes
# ``impl(x: float32 [R, C], clip_lo: float) -> float64 [R, C]``, the row-wise
# log of softmax_clipped (the log that follows softmax in training is why
# the reference functor clips, Sec. 2.1).

def _close_abs(got, want, tol=1e-13):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    both_inf = np.isneginf(got) & np.isneginf(want)
    ok = both_inf | (np.abs(got - want) <= tol * np.maximum(1.0, np.abs(want)))
    return bool(np.all(ok))


def pinl_library_log_softmax(impl):
    """No clip: scipy.special.log_softmax in float64, on rows whose shifted
    logits reach -800 (where exp underflows but the log must not) and rows
    with large offsets."""
    from scipy.special import log_softmax
    rng = np.random.default_rng(61)
    rows = [rng.uniform(-800.0, 0.0, 64), rng.uniform(-150.0, 10.0, 64),
            800.0 + rng.standard_normal(64), 3.0 * rng.standard_normal(64)]
    x = _f32(np.stack(rows))
    assert _close_abs(impl(x, -np.inf), log_softmax(x.astype(np.float64), axis=1))
    # where no shifted logit is below -64 the -64 clip changes nothing
    x = random_logits(5, 300, 62, "normal", 4.0)
    assert _close_abs(impl(x, -64.0), log_softmax(x.astype(np.float64), axis=1))


def pinl_is_log_of_softmax(impl):
    """exp of the result is the pinned clipped softmax (math.exp per entry,
    where the probability is a normal float64)."""
    x = random_logits(6, 257, 63, "clip_heavy")
    for lo in (-64.0, -90.0):
        y = impl(x, lo)
        p = np.exp(y)
        want = _softmax_reference(x, lo)
        assert np.all(np.abs(p - want) <= 1e-13 * want)


def _softmax_reference(x, lo):
    """Plain loops over the definition (math.fsum), independent of numpy's
    reductions, for the consistency pin."""
    out = np.empty(x.shape)
    for i, row in enumerate(x.astype(np.float64)):
        m = max(row)
        e = [math.exp(max(v - m, lo)) for v in row]
        s = math.fsum(e)
        out[i] = [t / s for t in e]
    return out


def pinl_uniform_and_two_class(impl):
    """Uniform rows give -log N; two classes give the log-sigmoid
    (scipy.special.log_expit of the difference)."""
    from scipy.special import log_expit
    for n in (1, 2, 7, 1000):
        y = impl(_f32(np.full((2, n), 3.5)), -64.0)
        assert _close_abs(y, np.full((2, n), -math.log(n)), 1e-15)
    rng = np.random.default_rng(64)
    a, b = rng.uniform(-30.0, 30.0, 100), rng.uniform(-30.0, 30.0, 100)
    x = _f32(np.stack([a, b], axis=1))
    diff = x[:, 0].astype(np.float64) - x[:, 1].astype(np.float64)
    y = impl(x, -np.inf)
    assert _close_abs(y[:, 0], log_expit(diff)) and _close_abs(y[:, 1], log_expit(-diff))


def pinl_closed_form_clip(impl):
    """Row [0, -100, -64, -63.5, -1e4] at the -64 clip:
    y = c - log(1 + 3 e^-64 + e^-63.5) with c = [0, -64, -64, -63.5, -64];
    rows at a bound of -1 where the clipped terms dominate the sum."""
    x = _f32([[0.0, -100.0, -64.0, -63.5, -1.0e4]])
    ls = math.log1p(3.0 * E64 + math.exp(-63.5))
    want = np.array([[0.0, -64.0, -64.0, -63.5, -64.0]]) - ls
    assert _close_abs(impl(x, -64.0), want, 1e-15)
    # a bound close to the max makes the clip's share of the sum visible:
    # [0, -3, -5] at -1 gives c = [0, -1, -1] and S = 1 + 2/e
    x = _f32([[0.0, -3.0, -5.0], [7.0, 4.0, 2.0]])
    want = np.array([[0.0, -1.0, -1.0]] * 2) - math.log1p(2.0 * math.exp(-1.0))
    assert _close_abs(impl(x, -1.0), want, 1e-15)


def pinl_brute_force_decimal(impl):
    """Tiny rows against 50-digit decimal logs at bounds -48, -64, -90, -120
    and with no clip (tests/golden, logy_clip)."""
    with open(os.path.join(GOLDEN, "brute_force_rows.json")) as f:
        doc = json.load(f)
    for rec in doc["rows"]:
        x = _f32([[float.fromhex(h) for h in rec["x_hex"]]])
        for key, vals in rec["logy_clip"].items():
            lo = -np.inf if key == "-inf" else float(key)
            want = np.array([float(Decimal(v)) for v in vals])
            assert _close_abs(impl(x, lo)[0], want, 1e-14), (rec["x_hex"], key)


def pinl_nonfinite(impl):
    """NaN, +inf and all -inf rows are NaN; a -inf entry gives the clipped
    value c - log S, or -inf with no clip."""
    x = _f32([[1.0, np.nan, 0.0], [1.0, np.inf, 0.0], [-np.inf] * 3, [0.0, -np.inf, 0.0]])
    y = impl(x, -64.0)
    assert np.all(np.isnan(y[:3]))
    ls = math.log(2.0 + E64)
    assert _close_abs(y[3], [-ls, -64.0 - ls, -ls], 1e-15)
    y = impl(x, -np.inf)
    assert np.all(np.isnan(y[:3])) and y[3, 1] == -np.inf
    assert _close_abs(y[3, [0, 2]], [-math.log(2.0)] * 2, 1e-15)


def pinl_shift_invariance(impl):
    """Adding k to a dyadic row leaves every output bit-identical."""
    x = random_logits(4, 129, 65, "dyadic")
    y0 = impl(x, -64.0)
    for k in (0.5, 64.0, -256.0):
        xk = _f32(x.astype(np.float64) + k)
        assert np.array_equal(impl(xk, -64.0), y0), k


LOG_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pinl_")]


# ---------------------------------------------------------------------------
# Pins for the per-row negative log-likelihood of a label under the clipped
# softmax.  Each ``pinn_*`` function takes
# ``impl(x: float32 [R, C], labels: int64 [R], clip_lo: float) -> float64 [R]``.

def _labels(*v):
    return np.asarray(v, dtype=np.int64)


def pinn_library_cross_entropy(impl):
    """No clip: torch's cross_entropy in float64 (reduction 'none'), on rows
    whose shifted logits reach -800 and rows with offsets of +-800; with the
    -64 clip on rows where no shifted logit is below -64."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(71)
    rows = [rng.uniform(-800.0, 0.0, 64), rng.uniform(-150.0, 10.0, 64),
            800.0 + rng.standard_normal(64), -800.0 + 3.0 * rng.standard_normal(64)]
    x = _f32(np.stack(rows))
    t = rng.integers(0, 64, size=4)
    want = F.cross_entropy(torch.from_numpy(x.astype(np.float64)), torch.from_numpy(t),
                           reduction="none").numpy()
    assert _close_abs(impl(x, t, -np.inf), want)
    x = random_logits(6, 300, 72, "normal", 4.0)
    t = rng.integers(0, 300, size=6)
    want = F.cross_entropy(torch.from_numpy(x.astype(np.float64)), torch.from_numpy(t),
                           reduction="none").numpy()
    assert _close_abs(impl(x, t, -64.0), want)


def pinn_uniform_and_two_class(impl):
    """Uniform rows give log N for any label; two classes give the softplus
    of the other class's margin (-log_expit of the label's margin)."""
    from scipy.special import log_expit
    for n in (1, 2, 7, 1000):
        for lab in sorted({0, n // 2, n - 1}):
            y = impl(_f32(np.full((2, n), -2.25)), _labels(lab, lab), -64.0)
            assert _close_abs(y, [math.log(n)] * 2, 1e-15), (n, lab)
    rng = np.random.default_rng(73)
    a, b = rng.uniform(-30.0, 30.0, 100), rng.uniform(-30.0, 30.0, 100)
    x = _f32(np.stack([a, b], axis=1))
    diff = x[:, 0].astype(np.float64) - x[:, 1].astype(np.float64)
    t = rng.integers(0, 2, size=100)
    want = np.where(t == 0, -log_expit(diff), -log_expit(-diff))
    assert _close_abs(impl(x, t, -np.inf), want)


def pinn_closed_form_clip(impl):
    """Row [0, -100, -64, -63.5, -1e4] at the -64 clip, every label:
    loss = log(1 + 3 e^-64 + e^-63.5) - c_label with
    c = [0, -64, -64, -63.5, -64]; and at a bound of -1, where the clipped
    terms change the sum: [0, -3, -5] gives log(1 + 2/e) - c_label with
    c = [0, -1, -1]."""
    x = _f32([[0.0, -100.0, -64.0, -63.5, -1.0e4]] * 5)
    ls = math.log1p(3.0 * E64 + math.exp(-63.5))
    want = ls - np.array([0.0, -64.0, -64.0, -63.5, -64.0])
    assert _close_abs(impl(x, _labels(0, 1, 2, 3, 4), -64.0), want, 1e-15)
    x = _f32([[0.0, -3.0, -5.0]] * 3)
    ls = math.log1p(2.0 * math.exp(-1.0))
    assert _close_abs(impl(x, _labels(0, 1, 2), -1.0), ls - np.array([0.0, -1.0, -1.0]), 1e-15)


def pinn_brute_force_decimal(impl):
    """Tiny rows against the 50-digit decimal logs (tests/golden, logy_clip):
    the loss of label j is minus the log-probability of column j, at every
    stored bound and every label."""
    with open(os.path.join(GOLDEN, "brute_force_rows.json")) as f:
        doc = json.load(f)
    for rec in doc["rows"]:
        row = [float.fromhex(h) for h in rec["x_hex"]]
        n = len(row)
        x = _f32([row] * n)
        t = np.arange(n, dtype=np.int64)
        for key, vals in rec["logy_clip"].items():
            lo = -np.inf if key == "-inf" else float(key)
            want = -np.array([float(Decimal(v)) for v in vals])
            assert _close_abs(impl(x, t, lo), want, 1e-14), (rec["x_hex"], key)


def pinn_label_picks_its_column(impl):
    """For unclipped columns j and k of one row the losses differ by exactly
    x_k - x_j (the shared log-sum cancels); labels are per row, not shared."""
    x = random_logits(1, 40, 74, "normal", 2.0)
    xs = _f32(np.repeat(x, 40, axis=0))
    losses = impl(xs, np.arange(40, dtype=np.int64), -64.0)
    x64 = x[0].astype(np.float64)
    assert np.all(np.abs((losses - losses[0]) - (x64[0] - x64)) <= 1e-12)
    y = impl(_f32([[5.0, 0.0, 0.0], [0.0, 5.0, 0.0]]), _labels(0, 0), -64.0)
    assert y[0] < 0.02 and y[1] > 4.9


def pinn_out_of_range_and_nonfinite(impl):
    """Labels below 0 or at or past the class count give NaN (never a
    wrapped index); a NaN row gives NaN; with no clip a -inf label entry
    gives +inf, with the -64 clip it gives 64 + log S."""
    x = _f32([[1.0, 2.0, 3.0]] * 4)
    y = impl(x, _labels(-1, 3, 1 << 40, 2), -64.0)
    assert np.all(np.isnan(y[:3])) and np.isfinite(y[3])
    x = _f32([[1.0, np.nan, 0.0], [1.0, np.inf, 0.0], [0.0, -np.inf, 0.0], [0.0, -np.inf, 0.0]])
    y = impl(x, _labels(0, 0, 1, 1), -np.inf)
    assert np.isnan(y[0]) and np.isnan(y[1]) and y[2] == np.inf and y[3] == np.inf
    y = impl(x[2:], _labels(1, 0), -64.0)
    assert _close_abs(y, [64.0 + math.log(2.0 + E64), math.log(2.0 + E64)], 1e-15)


NLL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pinn_")]
