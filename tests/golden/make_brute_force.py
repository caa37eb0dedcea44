"""Write brute_force_rows.json: tiny rows evaluated in 50-digit decimal.

The expected values here come from Python's ``decimal`` module alone (its
``exp`` is correctly rounded at the context precision), not from the oracle
and not from the GPU path.  They pin the float64 oracle to the definition:

  * Sec. 1.1, Eq. (1): y_j = e^{x_j} / sum_i e^{x_i}, evaluated directly with
    no max shift for rows where no shifted logit is below -64;
  * Sec. 1.2, Fig. 1 with the -64 clip on the shifted logits (the reading of
    Sec. 2.1 used throughout), evaluated as
    y_j = exp(max(x_j - M, -64)) / sum_i exp(max(x_i - M, -64)).

Each row is also evaluated with other clip bounds (``y_clip``): -48, -90,
-120 and -inf (no clip, the optimised functor of Sec. 2.3 Fig. 4, which
drops the ValueClip, Sec. 2.1), and its logarithm ``logy_clip``,
c_j - ln(sum_k exp(c_k)), at those bounds and at -64 (the log that the clip
exists for, Sec. 2.1).

Inputs are fp32 values stored as exact hex strings.  Run from the repo root:
    python tests/golden/make_brute_force.py
"""
from __future__ import annotations

import json
import os
from decimal import Decimal, getcontext

import numpy as np

getcontext().prec = 50
CLIP = Decimal(-64)
OTHER_CLIPS = {"-48": Decimal(-48), "-90": Decimal(-90), "-120": Decimal(-120),
               "-inf": Decimal("-Infinity")}


def _rows() -> list[list[float]]:
    rng = np.random.default_rng(20190429)
    rows: list[list[float]] = []
    # unclipped random rows of every width 1..8
    for c in range(1, 9):
        for scale in (1.0, 6.0):
            rows.append(list(np.float32(scale * rng.standard_normal(c))))
    # rows with large common offsets (shift must not matter)
    for off in (-50.0, 33.5, 80.0):
        rows.append(list(np.float32(off + rng.standard_normal(5))))
    # rows where the clip is active, and boundary values around -64
    rows.append([0.0, -100.0, -64.0, -63.5, -1.0e4])
    rows.append([10.0, -54.0, -53.999996185302734, -54.000003814697266, 9.0])
    rows.append([-3.0, -70.0, -2.0, -66.5, -67.0, -65.99999237060547])
    rows.append(list(np.float32(rng.uniform(-150.0, 0.0, 8))))
    rows.append(list(np.float32(rng.uniform(-150.0, 0.0, 7))))
    # ties and signed zeros
    rows.append([2.5, 2.5, 2.5, -1.0])
    rows.append([0.0, -0.0, -0.0, 0.0])
    # rows whose shifted logits reach the denormal and underflow range of
    # fp32 exponentials (e^-87.3 and e^-103.3), for the lower clip bounds
    rows.append([0.0, -88.0, -95.5, -103.0, -104.5, -110.0, -1.0e4])
    rows.append(list(np.float32(rng.uniform(-130.0, 0.0, 8))))
    return [[float(np.float32(v)) for v in r] for r in rows]


def clipped_softmax_decimal(row: list[float], clip: Decimal = CLIP) -> list[Decimal]:
    xs = [Decimal(v) for v in row]            # exact: fp32 -> Decimal
    m = max(xs)
    cs = [max(x - m, clip) for x in xs]
    es = [c.exp() for c in cs]
    s = sum(es, Decimal(0))
    return [e / s for e in es]


def log_softmax_decimal(row: list[float], clip: Decimal = CLIP) -> list[Decimal]:
    """c_j - ln(sum_k exp(c_k)) with c = max(x - M, clip), in decimal."""
    xs = [Decimal(v) for v in row]
    m = max(xs)
    cs = [max(x - m, clip) for x in xs]
    s = sum((c.exp() for c in cs), Decimal(0))
    ls = s.ln()
    return [c - ls for c in cs]


def eq1_softmax_decimal(row: list[float]) -> list[Decimal]:
    xs = [Decimal(v) for v in row]
    es = [x.exp() for x in xs]
    s = sum(es, Decimal(0))
    return [e / s for e in es]


def main() -> None:
    out = []
    for row in _rows():
        y = clipped_softmax_decimal(row)
        m = max(row)
        clip_active = any(Decimal(v) - Decimal(m) < CLIP for v in row)
        rec = {
            "x_hex": [float(v).hex() for v in row],
            "y": [format(v, ".30e") for v in y],
            "clip_active": clip_active,
            "y_clip": {k: [format(v, ".30e") for v in clipped_softmax_decimal(row, c)]
                       for k, c in OTHER_CLIPS.items()},
            "logy_clip": {k: [format(v, ".30e") for v in log_softmax_decimal(row, c)]
                          for k, c in dict(OTHER_CLIPS, **{"-64": CLIP}).items()},
        }
        if not clip_active:
            y1 = eq1_softmax_decimal(row)
            # Eq. (1) without a shift and the shifted form agree to ~1e-45.
            assert all(abs(a - b) <= Decimal("1e-40") * b for a, b in zip(y, y1))
            rec["y_eq1"] = [format(v, ".30e") for v in y1]
        out.append(rec)
    doc = {
        "what": "clipped row softmax of tiny fp32 rows in 50-digit decimal",
        "cites": "Sec. 1.1 Eq. (1); Sec. 1.2 Fig. 1 (clip of the shifted "
                 "logits, bound -64; y_clip: other bounds and no clip); "
                 "Sec. 2.1; Sec. 2.3 Fig. 4",
        "generator": "tests/golden/make_brute_force.py (decimal only)",
        "rows": out,
    }
    path = os.path.join(os.path.dirname(__file__), "brute_force_rows.json")
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    print(f"wrote {len(out)} rows to {path}")


if __name__ == "__main__":
    main()
