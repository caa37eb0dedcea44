"""Write attention_cases.json: tiny attention problems in 50-digit decimal.

Expected values come from Python's ``decimal`` module alone (not from the
oracle, not from the GPU path): for fp32 inputs Q [lq, d], K [lk, d],
V [lk, dv] and an fp32 scale,

    s_ij = scale * sum_t Q_it K_jt
    p_ij = exp(max(s_ij - max_j s_ij, L)) / sum_j exp(max(s_ij - max_j s_ij, L))
    o_ic = sum_j p_ij V_jc

with L = -64 (the clip of the softmax step, Sec. 1.2 Fig. 1) and with no
clip (Sec. 2.3 Fig. 4).  Every fp32 value converts to Decimal exactly.
Run from the repo root:
    python tests/golden/make_attention_brute_force.py
"""
from __future__ import annotations

import json
import os
from decimal import Decimal, getcontext

import numpy as np

getcontext().prec = 50
CLIPS = {"-64": Decimal(-64), "-inf": Decimal("-Infinity")}


def _cases():
    rng = np.random.default_rng(19042019)
    out = []
    for (lq, lk, d, dv, spread) in ((1, 1, 1, 1, 1.0), (2, 3, 4, 2, 1.0), (3, 4, 5, 3, 2.0),
                                    (2, 5, 3, 4, 6.0), (4, 2, 6, 1, 1.0)):
        q = rng.standard_normal((lq, d)) * spread
        k = rng.standard_normal((lk, d)) * spread
        v = rng.standard_normal((lk, dv))
        out.append((np.float32(q), np.float32(k), np.float32(v), np.float32(1.0 / np.sqrt(d))))
    # a case where the clip is active: one key dominates by far
    q = np.float32([[12.0, 0.0], [0.0, 12.0]])
    k = np.float32([[12.0, 0.0], [0.0, 12.0], [-3.0, 1.0]])
    v = np.float32([[1.0, 2.0], [3.0, -4.0], [0.5, 0.25]])
    out.append((q, k, v, np.float32(1.0)))
    return out


def attention_decimal(q, k, v, scale, clip):
    lq, d = q.shape
    lk, dv = v.shape
    sc = Decimal(float(scale))
    o = []
    for i in range(lq):
        s = [sc * sum((Decimal(float(q[i, t])) * Decimal(float(k[j, t])) for t in range(d)),
                      Decimal(0)) for j in range(lk)]
        m = max(s)
        e = [max(x - m, clip).exp() for x in s]
        tot = sum(e, Decimal(0))
        p = [x / tot for x in e]
        o.append([sum((p[j] * Decimal(float(v[j, c])) for j in range(lk)), Decimal(0))
                  for c in range(dv)])
    return o


def main() -> None:
    recs = []
    for q, k, v, scale in _cases():
        rec = {"q_hex": [[float(x).hex() for x in r] for r in q],
               "k_hex": [[float(x).hex() for x in r] for r in k],
               "v_hex": [[float(x).hex() for x in r] for r in v],
               "scale_hex": float(scale).hex(),
               "o": {key: [[format(x, ".30e") for x in r] for r in attention_decimal(q, k, v, scale, c)]
                     for key, c in CLIPS.items()}}
        recs.append(rec)
    doc = {"what": "softmax attention of tiny fp32 problems in 50-digit decimal",
           "cites": "softmax step: Sec. 1.1 Eq. (1), Sec. 1.2 Fig. 1 (clip -64), "
                    "Sec. 2.3 Fig. 4 (no clip); attention of the DAM model (Sec. 1)",
           "generator": "tests/golden/make_attention_brute_force.py (decimal only)",
           "cases": recs}
    path = os.path.join(os.path.dirname(__file__), "attention_cases.json")
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    print(f"wrote {len(recs)} cases to {path}")


if __name__ == "__main__":
    main()
