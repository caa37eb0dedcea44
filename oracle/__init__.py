"""CPU oracle for the clipped row softmax -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import, call, link or run anything in this directory.  The
product path (the HIP library and its Python binding) never does, and shares
no code, header, constant or helper with it.

Contents
--------
``softmax_f64``          float64 definition of the clipped row softmax, of
                          its logarithm and of the per-row negative
                          log-likelihood of a label (plain numpy; the
                          parity references).
``attention_f64``        float64 softmax attention, softmax(scale Q K^T) V
                          per batch element, built on ``softmax_f64``.
``cpu_fp32_baseline.c``  a straightforward single-thread fp32 C softmax in the
                          loop shape of the paper's MKL-era functor; it is a
                          timed CPU baseline, never a parity reference.

Every function here is pinned by ``tests/test_oracle_pins.py`` to facts that
do not come from this code: closed forms, the logistic special case, a
50-digit ``decimal`` brute force, a library cross-check and invariants.
"""
from .attention_f64 import attention_clipped
from .softmax_f64 import (CLIP_LO, exp_clipped, log_softmax_clipped, nll_clipped, row_max,
                          softmax_clipped)

__all__ = ["CLIP_LO", "row_max", "exp_clipped", "softmax_clipped", "log_softmax_clipped",
           "nll_clipped", "attention_clipped"]
