"""Pins for any implementation of softmax attention over small tiles.

Each ``pina_*`` function takes ``impl(q, k, v, scale, clip_lo) -> float64
[batch, lq, dv]`` (q [batch, lq, d], k [batch, lk, d], v [batch, lk, dv],
fp32) and raises AssertionError when ``impl`` violates a fact that does not
come from the oracle's own code:

  * torch's scaled_dot_product_attention in float64 where the clip is
    inactive (a library special case);
  * closed forms: all-zero queries give the mean of the value rows; a
    dominant key clipped at -64 gives weights 1/(1 + n e^-64) and
    e^-64/(1 + n e^-64);
  * a 50-digit decimal brute force of tiny problems (tests/golden);
  * identity values (V = I) give the softmax weights themselves, checked
    against plain loops over the definition;
  * invariants: permuting keys together with their values, linearity in V,
    and rows of queries computed one at a time.

The softmax step is the paper's (Sec. 1.1 Eq. (1), clip of Sec. 1.2 Fig. 1,
no clip as in Sec. 2.3 Fig. 4); the attention around it is the DAM model's
scaled dot-product attention (Sec. 1).
"""
from __future__ import annotations

import json
import math
import os
from decimal import Decimal

import numpy as np

from workloads import random_qkv

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
E64 = math.exp(-64.0)


def _f32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _normwise(got, want) -> float:
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    return float(np.max(np.abs(got - want)) / max(np.max(np.abs(want)), 1e-300))


def pina_library_sdpa(impl):
    """Clip inactive (scores within 64 of their row max): torch's
    scaled_dot_product_attention in float64 gives the same result."""
    import torch
    for (b, lq, lk, d, dv, seed) in ((3, 50, 50, 200, 200, 1), (2, 7, 13, 16, 5, 2),
                                     (4, 1, 64, 32, 48, 3)):
        q, k, v = random_qkv(b, lq, lk, d, dv, seed)
        scale = float(np.float32(1.0 / math.sqrt(d)))
        want = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q).double(), torch.from_numpy(k).double(),
            torch.from_numpy(v).double(), scale=scale).numpy()
        assert _normwise(impl(q, k, v, scale, -64.0), want) < 1e-13, (b, lq, lk, d, dv)


def pina_zero_queries_average_values(impl):
    """Q = 0 makes every score 0, so every output row is the mean of V's
    rows."""
    _, k, v = random_qkv(2, 5, 9, 8, 6, 4)
    q = np.zeros((2, 5, 8), dtype=np.float32)
    o = impl(q, k, v, 0.5, -64.0)
    want = np.broadcast_to(v.astype(np.float64).mean(axis=1, keepdims=True), o.shape)
    assert _normwise(o, want) < 1e-15


def pina_dominant_key_clipped(impl):
    """Query i aligned with key i only: s_ii = 900, all other scores 0, so
    with the -64 clip the weights are 1/(1 + 3 e^-64) and e^-64/(1 + 3 e^-64);
    with no clip the other keys get e^-900 = 0 in float64.  With V = I the
    output is the weight matrix itself, compared element by element."""
    key = 30.0 * np.eye(4)
    q, k = _f32(key[None]), _f32(key[None])
    w_hi, w_lo = 1.0 / (1.0 + 3.0 * E64), E64 / (1.0 + 3.0 * E64)
    p = np.full((4, 4), w_lo) + np.eye(4) * (w_hi - w_lo)
    eye = _f32(np.eye(4)[None])
    got = impl(q, k, eye, 1.0, -64.0)[0]
    assert np.all(np.abs(got - p) <= 1e-14 * p), got
    assert np.array_equal(impl(q, k, eye, 1.0, -np.inf)[0], np.eye(4))
    v = _f32(np.arange(16, dtype=np.float64).reshape(1, 4, 4) - 5.0)
    assert _normwise(impl(q, k, v, 1.0, -64.0)[0], p @ v[0].astype(np.float64)) < 1e-15


def pina_brute_force_decimal(impl):
    """Tiny problems against 50-digit decimal, with the -64 clip and with no
    clip (tests/golden/attention_cases.json)."""
    with open(os.path.join(GOLDEN, "attention_cases.json")) as f:
        doc = json.load(f)
    for rec in doc["cases"]:
        q = _f32([[[float.fromhex(h) for h in r] for r in rec["q_hex"]]])
        k = _f32([[[float.fromhex(h) for h in r] for r in rec["k_hex"]]])
        v = _f32([[[float.fromhex(h) for h in r] for r in rec["v_hex"]]])
        scale = float.fromhex(rec["scale_hex"])
        for key, rows in rec["o"].items():
            lo = -np.inf if key == "-inf" else float(key)
            want = np.array([[float(Decimal(x)) for x in r] for r in rows])
            got = impl(q, k, v, scale, lo)[0]
            assert np.all(np.abs(got - want) <= 1e-14 * np.abs(want) + 1e-15), (key, got, want)


def pina_identity_values_give_weights(impl):
    """V = I (lk = dv) returns the softmax weights; checked against plain
    loops over the definition with math.fsum."""
    q, k, _ = random_qkv(2, 3, 6, 5, 6, 5, scale=3.0)
    v = _f32(np.broadcast_to(np.eye(6), (2, 6, 6)))
    scale = 0.75
    got = impl(q, k, v, scale, -64.0)
    for b in range(2):
        for i in range(3):
            s = [scale * math.fsum(float(q[b, i, t]) * float(k[b, j, t]) for t in range(5))
                 for j in range(6)]
            m = max(s)
            e = [math.exp(max(x - m, -64.0)) for x in s]
            tot = math.fsum(e)
            want = [x / tot for x in e]
            assert _normwise(got[b, i], want) < 1e-14


def pina_key_permutation(impl):
    """Permuting the keys together with their value rows changes nothing."""
    q, k, v = random_qkv(3, 4, 11, 7, 5, 6, scale=2.0)
    perm = np.random.default_rng(7).permutation(11)
    a = impl(q, k, v, 0.4, -64.0)
    b = impl(q, k[:, perm], v[:, perm], 0.4, -64.0)
    assert _normwise(b, a) < 1e-14


def pina_linear_in_values(impl):
    """O(V1 + V2) = O(V1) + O(V2) for the same queries and keys (V1, V2 on a
    2^-10 grid, so V1 + V2 is exact in fp32)."""
    q, k, _ = random_qkv(2, 6, 9, 4, 7, 8)
    rng = np.random.default_rng(9)
    v1 = _f32(np.round(rng.standard_normal((2, 9, 7)) * 1024.0) / 1024.0)
    v2 = _f32(np.round(rng.standard_normal((2, 9, 7)) * 1024.0) / 1024.0)
    v12 = _f32(v1.astype(np.float64) + v2.astype(np.float64))
    assert np.array_equal(v12.astype(np.float64), v1.astype(np.float64) + v2.astype(np.float64))
    lhs = impl(q, k, v12, 0.5, -64.0)
    rhs = impl(q, k, v1, 0.5, -64.0) + impl(q, k, v2, 0.5, -64.0)
    assert _normwise(lhs, rhs) < 1e-14


def pina_query_rows_independent(impl):
    """Each output row depends only on its own query: one query at a time
    gives the same rows; the batch axis is independent too."""
    q, k, v = random_qkv(3, 5, 8, 6, 4, 10, scale=2.0)
    full = impl(q, k, v, 0.3, -64.0)
    for i in range(5):
        part = impl(_f32(q[:, i:i + 1]), k, v, 0.3, -64.0)
        assert _normwise(part[:, 0], full[:, i]) < 1e-15
    one = impl(_f32(q[1:2]), _f32(k[1:2]), _f32(v[1:2]), 0.3, -64.0)
    assert _normwise(one[0], full[1]) < 1e-15


def pina_empty(impl):
    """Empty batch, query or value dimensions give empty outputs."""
    for (b, lq, lk, d, dv) in ((0, 3, 4, 5, 6), (2, 0, 4, 5, 6), (2, 3, 4, 5, 0)):
        q, k, v = random_qkv(b, lq, lk, d, dv, 11)
        assert impl(q, k, v, 1.0, -64.0).shape == (b, lq, dv)


ATTN_PINS = [v for k_, v in sorted(globals().items()) if k_.startswith("pina_")]
