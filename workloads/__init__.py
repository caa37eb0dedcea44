"""Seeded synthetic inputs for the row-softmax workloads.

This module only draws random numbers and shapes them into logits matrices.
It performs none of the softmax arithmetic, so both the float64 oracle and the
GPU path can take their inputs from here without sharing any of the method.

The paper measures softmax inside inference of the Deep Attention Matching
(DAM) model (Sec. 1 and Sec. 3); its model, data and figure values are not
available, so every workload below is synthetic.  Each one is shaped like a
use the paper names: DAM attention rows, classifier rows, NLP vocabulary rows,
plus a long-row case.  Draw order is fixed and uses numpy's PCG64
(``default_rng(seed)``); values are drawn in float64 and cast once to float32
(round to nearest even).

The DAM-style scores are formed as Q.K^T / sqrt(200) from 200-dim standard
normal vectors that are first rounded to multiples of 2^-10.  With that
rounding every product and every partial sum of the 200-term dot product is
exact in float64, so the result does not depend on the summation order that
a BLAS or einsum kernel happens to use on a given host CPU.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

__all__ = ["Workload", "WORKLOADS", "generate", "sha256_f32", "random_logits",
           "generate_labels", "AttentionWorkload", "ATTENTION_WORKLOADS", "generate_qkv",
           "random_qkv"]


@dataclass(frozen=True)
class Workload:
    key: str
    rows: int
    cols: int
    seed: int
    description: str

    @property
    def elements(self) -> int:
        return self.rows * self.cols

    @property
    def algorithmic_bytes(self) -> int:
        """One fp32 read of x and one fp32 write of y per element."""
        return 8 * self.rows * self.cols


WORKLOADS: dict[str, Workload] = {
    w.key: w
    for w in (
        Workload("plumbing_64x1000", 64, 1000, 0,
                 "uniform(-10, 10) logits, 64 rows x 1000 classes"),
        Workload("dam_attention_115200x50", 115200, 50, 1,
                 "DAM-style attention scores: 256 batch x 9 turns x 50 queries "
                 "rows over 50 keys; score = q.k / sqrt(200)"),
        Workload("classifier_4096x1000", 4096, 1000, 2,
                 "N(0, 3^2) classifier logits with one true class boosted by +8"),
        Workload("vocab_512x32768", 512, 32768, 3,
                 "N(0, 2^2) vocabulary logits; 5% of entries set to -1e4, "
                 "5 rows with a single +80 outlier"),
        Workload("longrow_64x262144", 64, 262144, 4,
                 "N(0,1) + per-row offset uniform(-50, 50), 64 rows x 262144"),
    )
}

# Short aliases by position (1-based, in the order above).
_BY_INDEX = {i + 1: k for i, k in enumerate(WORKLOADS)}


def _resolve(key) -> Workload:
    if isinstance(key, int):
        key = _BY_INDEX[key]
    return WORKLOADS[key]


def _dam_qk(rng: np.random.Generator) -> tuple[np.ndarray, np.ndarray]:
    """DAM query and key vectors, [2304, 50, 200] each, standard normal
    rounded to multiples of 2^-10 (exact in fp32)."""
    batch_turns, q, k, dim = 2304, 50, 50, 200
    qv = rng.standard_normal((batch_turns, q, dim))
    kv = rng.standard_normal((batch_turns, k, dim))
    qv = np.round(qv * 1024.0) / 1024.0
    kv = np.round(kv * 1024.0) / 1024.0
    return qv, kv


def _dam_scores(rng: np.random.Generator) -> np.ndarray:
    batch_turns, q, k = 2304, 50, 50
    qv, kv = _dam_qk(rng)
    s = np.matmul(qv, kv.transpose(0, 2, 1))
    s = s / np.sqrt(200.0)
    return s.reshape(batch_turns * q, k)


def generate(key) -> np.ndarray:
    """Return the float32 [rows, cols] logits matrix for a workload.

    ``key`` is a workload name from ``WORKLOADS`` or its 1-based position.
    """
    w = _resolve(key)
    rng = np.random.default_rng(w.seed)
    if w.key == "plumbing_64x1000":
        x = rng.uniform(-10.0, 10.0, (w.rows, w.cols))
    elif w.key == "dam_attention_115200x50":
        x = _dam_scores(rng)
    elif w.key == "classifier_4096x1000":
        x = 3.0 * rng.standard_normal((w.rows, w.cols))
        t = rng.integers(0, w.cols, w.rows)
        x[np.arange(w.rows), t] += 8.0
    elif w.key == "vocab_512x32768":
        x = 2.0 * rng.standard_normal((w.rows, w.cols))
        base = x.copy()
        mask = rng.random(x.shape) < 0.05
        x[mask] = -1.0e4
        rows = rng.choice(w.rows, 5, replace=False)
        cols = rng.integers(0, w.cols, 5)
        x[rows, cols] = base[rows, cols] + 80.0
    elif w.key == "longrow_64x262144":
        off = rng.uniform(-50.0, 50.0, (w.rows, 1))
        x = rng.standard_normal((w.rows, w.cols)) + off
    else:  # pragma: no cover
        raise KeyError(w.key)
    out = np.ascontiguousarray(x.astype(np.float32))
    assert out.shape == (w.rows, w.cols)
    return out


def sha256_f32(x: np.ndarray) -> str:
    """SHA-256 of the little-endian float32 bytes of a C-contiguous array."""
    a = np.ascontiguousarray(x, dtype="<f4")
    return hashlib.sha256(a.tobytes()).hexdigest()


def generate_labels(key, seed_offset: int = 1000) -> np.ndarray:
    """int64 [rows] class labels for a workload, uniform over [0, cols), from
    their own seeded stream (the workload's seed + seed_offset), so that the
    logits are the same with or without labels."""
    w = _resolve(key)
    rng = np.random.default_rng(w.seed + seed_offset)
    return np.ascontiguousarray(rng.integers(0, w.cols, size=w.rows, dtype=np.int64))


def random_logits(rows: int, cols: int, seed: int, kind: str = "normal",
                  scale: float = 4.0) -> np.ndarray:
    """Seeded float32 logits for edge-shape tests.

    kinds: ``normal`` (N(0, scale^2)), ``uniform`` (U(-scale, scale)),
    ``clip_heavy`` (a few large values over a wide negative spread, so that
    many shifted logits fall below -64), ``offset`` (N(0,1) plus a per-row
    offset in U(-50, 50)), ``dyadic`` (multiples of 1/64 in [-8, 8]).
    """
    rng = np.random.default_rng(seed)
    shape = (rows, cols)
    if kind == "normal":
        x = scale * rng.standard_normal(shape)
    elif kind == "uniform":
        x = rng.uniform(-scale, scale, shape)
    elif kind == "clip_heavy":
        x = rng.uniform(-150.0, 0.0, shape)
        if rows and cols:
            hot = rng.integers(0, cols, rows)
            x[np.arange(rows), hot] = 20.0
    elif kind == "offset":
        off = rng.uniform(-50.0, 50.0, (rows, 1))
        x = rng.standard_normal(shape) + off
    elif kind == "dyadic":
        x = rng.integers(-512, 513, shape) / 64.0
    else:
        raise ValueError(kind)
    return np.ascontiguousarray(x.astype(np.float32))


# ---------------------------------------------------------------------------
# Attention inputs (Q, K, V) for the fused attention path: softmax over the
# keys of scale * Q.K^T, then the product with V, per batch element.

@dataclass(frozen=True)
class AttentionWorkload:
    key: str
    batch: int
    lq: int
    lk: int
    d: int
    dv: int
    seed: int
    description: str

    @property
    def scale(self) -> float:
        """1/sqrt(d) rounded to fp32, the scale applied to Q.K^T."""
        return float(np.float32(1.0 / np.sqrt(self.d)))

    @property
    def algorithmic_bytes(self) -> int:
        """One fp32 read of Q, K and V and one fp32 write of the output."""
        return 4 * self.batch * (self.lq * self.d + self.lk * self.d
                                 + self.lk * self.dv + self.lq * self.dv)

    @property
    def flops(self) -> int:
        """Multiply-adds of Q.K^T and P.V, two flops each."""
        return 2 * self.batch * self.lq * self.lk * (self.d + self.dv)


ATTENTION_WORKLOADS: dict[str, AttentionWorkload] = {
    w.key: w
    for w in (
        AttentionWorkload("dam_fused_attention_2304x50x50x200", 2304, 50, 50, 200, 200, 1,
                          "DAM attention, 256 batch x 9 turns: 50 queries over 50 keys "
                          "of dimension 200; Q and K are the vectors behind "
                          "dam_attention_115200x50, V is drawn after them"),
    )
}


def generate_qkv(key: str) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """float32 Q [batch, lq, d], K [batch, lk, d], V [batch, lk, dv].

    Q and K are the same draws as the DAM scores workload (seed 1), so the
    scores of this workload are that workload's logits before rounding; V is
    drawn next, standard normal rounded to multiples of 2^-10."""
    w = ATTENTION_WORKLOADS[key]
    rng = np.random.default_rng(w.seed)
    qv, kv = _dam_qk(rng)
    vv = np.round(rng.standard_normal((w.batch, w.lk, w.dv)) * 1024.0) / 1024.0
    return tuple(np.ascontiguousarray(a.astype(np.float32)) for a in (qv, kv, vv))


def random_qkv(batch: int, lq: int, lk: int, d: int, dv: int, seed: int,
               scale: float = 1.0) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Seeded float32 Q, K, V of N(0, scale^2) entries for edge-shape tests."""
    rng = np.random.default_rng(seed)
    q = scale * rng.standard_normal((batch, lq, d))
    k = scale * rng.standard_normal((batch, lk, d))
    v = rng.standard_normal((batch, lk, dv))
    return tuple(np.ascontiguousarray(a.astype(np.float32)) for a in (q, k, v))
