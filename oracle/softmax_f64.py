"""float64 oracle: row-wise softmax of max-shifted, lower-clipped logits.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed (for each row i of a [rows, classes] matrix x):

    M_i    = max_j x_ij                               (row max)
    d_ij   = x_ij - M_i                               (shifted logit)
    c_ij   = CLIP_LO if d_ij < CLIP_LO else d_ij      (lower clip)
    y_ij   = exp(c_ij) / sum_k exp(c_ik)

Sources in the paper:
  * Sec. 1.1, Eq. (1): softmax(z_j) = e^{z_j} / sum_i e^{z_i}.  Subtracting
    the row max does not change this value; it only keeps exp from
    overflowing.
  * Sec. 1.2, Fig. 1 (the reference Eigen functor): row max along the class
    dimension, broadcast subtract, a ValueClip applied to the shifted logits,
    exp, then multiplication by the inverse of the row sum.
  * Sec. 2.1: the clip exists so that softmax never returns 0 (a log follows
    in training); the paper prints no constant for it.
  * Sec. 2.3, Fig. 4: the same computation without the clip, in the order
    max, subtract, exp, sum, scale by 1/sum, over a row-major
    [batch_size, num_classes] buffer indexed n*num_classes + c.

Readings where the paper is silent:
  * The clip bound is CLIP_LO = -64 applied to the shifted logit before exp
    (the prose's 1e-60 is not an fp32 value and describes the effect, not the
    code).  Other bounds are a parameter, ``clip_lo``; ``clip_lo = -inf``
    is no clip at all, the optimised functor of Sec. 2.3 Fig. 4 (Sec. 2.1
    describes dropping the clip as the first optimisation).  Without a clip
    an output can be 0 (exp underflows below about -745 in float64).
  * The clip is a compare-select ``d < L ? L : d`` so a NaN stays NaN; a NaN
    anywhere in a row, a +inf element or an all -inf row makes the whole row
    NaN; a -inf element among finite ones clips to e^-64.
  * fp32 inputs are widened exactly to float64; every step is float64.
"""
from __future__ import annotations

import numpy as np

CLIP_LO = -64.0


def row_max(x: np.ndarray) -> np.ndarray:
    """Row maxima M_i as a float64 column [rows, 1] (Fig. 1: maximum along
    the class dimension; Fig. 4: the first per-row loop).  NaN propagates."""
    x64 = np.asarray(x, dtype=np.float64)
    return np.max(x64, axis=1, keepdims=True)


def exp_clipped(d: np.ndarray, clip_lo: float = CLIP_LO) -> np.ndarray:
    """exp of the lower-clipped shifted logit, float64 (Fig. 1: ValueClip
    then exp; clip_lo = -inf: exp alone, as in Fig. 4).  ``d`` is already
    x - M; a NaN stays NaN."""
    d64 = np.asarray(d, dtype=np.float64)
    c = np.where(d64 < clip_lo, clip_lo, d64)
    return np.exp(c)


def softmax_clipped(x: np.ndarray, clip_lo: float = CLIP_LO) -> np.ndarray:
    """Row-wise clipped softmax of a 2-D array, returned as float64.

    Sec. 1.1 Eq. (1) with the max shift and the clip of Sec. 1.2 Fig. 1 at
    ``clip_lo`` (-inf: no clip, Sec. 2.3 Fig. 4).
    """
    x64 = np.asarray(x, dtype=np.float64)
    if x64.ndim != 2:
        raise ValueError("expected a 2-D [rows, classes] array")
    rows, cols = x64.shape
    if rows == 0 or cols == 0:
        return np.zeros((rows, cols), dtype=np.float64)
    m = row_max(x64)
    with np.errstate(invalid="ignore", over="ignore"):
        d = x64 - m
        e = exp_clipped(d, clip_lo)
        s = np.sum(e, axis=1, keepdims=True)
        return e / s


def log_softmax_clipped(x: np.ndarray, clip_lo: float = CLIP_LO) -> np.ndarray:
    """Row-wise log of the clipped softmax, float64:

        y_ij = c_ij - log(sum_k exp(c_ik)),   c_ij = max(x_ij - M_i, clip_lo)

    which is log(softmax_clipped(x, clip_lo)) written so that it stays exact
    where the probability underflows.  The log after softmax is why the
    reference functor clips at all (Sec. 2.1: softmax must not return 0 for
    the log that follows in training); with clip_lo = -inf this is the plain
    log-softmax of the shifted logits (Sec. 1.1 Eq. (1), logarithm taken).
    A -inf entry gives -inf when there is no clip.
    """
    x64 = np.asarray(x, dtype=np.float64)
    if x64.ndim != 2:
        raise ValueError("expected a 2-D [rows, classes] array")
    rows, cols = x64.shape
    if rows == 0 or cols == 0:
        return np.zeros((rows, cols), dtype=np.float64)
    m = row_max(x64)
    with np.errstate(invalid="ignore", over="ignore", divide="ignore"):
        d = x64 - m
        c = np.where(d < clip_lo, clip_lo, d)
        s = np.sum(np.exp(c), axis=1, keepdims=True)
        return c - np.log(s)


def nll_clipped(x: np.ndarray, labels: np.ndarray, clip_lo: float = CLIP_LO) -> np.ndarray:
    """Per-row negative log-likelihood of a label under the clipped softmax,
    float64 [rows]:

        loss_i = log(sum_k exp(c_ik)) - c_{i, t_i},   c_ij = max(x_ij - M_i, clip_lo)

    that is -log_softmax_clipped(x, clip_lo)[i, t_i] for the label t_i of
    row i: the training loss that the log after softmax feeds, and the
    reason the reference functor clips (Sec. 2.1).  ``labels`` holds one
    integer per row; a label outside [0, cols) gives NaN.  Rows of zero
    columns have no valid label and are rejected.
    """
    x64 = np.asarray(x, dtype=np.float64)
    if x64.ndim != 2:
        raise ValueError("expected a 2-D [rows, classes] array")
    rows, cols = x64.shape
    t = np.asarray(labels)
    if t.shape != (rows,) or not np.issubdtype(t.dtype, np.integer):
        raise ValueError("expected one integer label per row")
    if rows == 0:
        return np.zeros(0, dtype=np.float64)
    if cols == 0:
        raise ValueError("rows of zero classes have no label")
    logp = log_softmax_clipped(x64, clip_lo)
    t64 = t.astype(np.int64)
    valid = (t64 >= 0) & (t64 < cols)
    picked = logp[np.arange(rows), np.where(valid, t64, 0)]
    return np.where(valid, -picked, np.nan)
