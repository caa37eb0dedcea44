"""float64 oracle for softmax attention over small tiles, as in DAM.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed, for every batch element b (Q: [lq, d], K: [lk, d],
V: [lk, dv], one fp32 scale):

    S_b = scale * Q_b K_b^T                 [lq, lk]   (scores)
    P_b = softmax_clipped(S_b, clip_lo)     row-wise over the keys
    O_b = P_b V_b                           [lq, dv]

Sources: the paper optimises softmax for inference of the Deep Attention
Matching model (Sec. 1; the model's profile, Sec. 1.2 Fig. 2, puts softmax
at 18.5% of its time, next to the matrix multiplications around it).  The attention
formula itself belongs to that model, not to this paper: its attentive
module is scaled dot-product attention, scale = 1/sqrt(d).  The softmax
step is ``softmax_clipped`` of this package (Sec. 1.1 Eq. (1) with the clip
of Sec. 1.2 Fig. 1), applied to the float64 scores; the two products are
plain matrix products (numpy matmul as a library step).
"""
from __future__ import annotations

import numpy as np

from .softmax_f64 import CLIP_LO, softmax_clipped


def attention_clipped(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                      clip_lo: float = CLIP_LO) -> np.ndarray:
    """O = softmax_clipped(scale * Q K^T) V per batch element, float64."""
    q64 = np.asarray(q, dtype=np.float64)
    k64 = np.asarray(k, dtype=np.float64)
    v64 = np.asarray(v, dtype=np.float64)
    if q64.ndim != 3 or k64.ndim != 3 or v64.ndim != 3:
        raise ValueError("expected [batch, len, dim] arrays")
    b, lq, d = q64.shape
    if k64.shape[0] != b or k64.shape[2] != d or v64.shape[:2] != k64.shape[:2]:
        raise ValueError("shapes of q, k, v do not match")
    lk, dv = k64.shape[1], v64.shape[2]
    if lk == 0 and b * lq > 0:
        raise ValueError("softmax over zero keys is undefined")
    if b == 0 or lq == 0 or dv == 0:
        return np.zeros((b, lq, dv), dtype=np.float64)
    s = np.matmul(q64, k64.transpose(0, 2, 1)) * float(scale)
    p = softmax_clipped(s.reshape(b * lq, lk), clip_lo).reshape(b, lq, lk)
    return np.matmul(p, v64)
