"""Planted mistakes in copies of the oracle must each fail at least one pin.

Every mutant below is a plausible slip when writing the clipped softmax
(a dropped term, a sign, the wrong axis, the clip in the wrong place, a wrong
constant, a float32 shortcut, ...).  The mistake is planted in a local copy
of the float64 oracle on the CPU; nothing here touches the GPU path.
"""
import numpy as np
import pytest

from tests import pins

L = -64.0


def _base(x, shift="max", clip_on="d", clip_lo=L, axis=1, base_e=False,
          drop_last=False, denom="sum", dtype=np.float64,
          clip_kind="lower"):
    x64 = np.asarray(x, dtype=dtype)
    if x64.size == 0:
        return np.zeros(x64.shape, dtype=np.float64)
    with np.errstate(all="ignore"):
        if shift == "max":
            m = np.max(x64, axis=axis, keepdims=True)
        elif shift == "first":
            m = np.take(x64, [0], axis=axis)
        else:
            m = np.zeros_like(np.take(x64, [0], axis=axis))
        if clip_on == "d":
            d = x64 - m
            src = d
        else:  # clip applied to the raw logits, then shifted
            src = x64
        if clip_kind == "lower":
            c = np.where(src < clip_lo, clip_lo, src)
        elif clip_kind == "fmax":
            c = np.fmax(src, clip_lo)
        elif clip_kind == "upper":
            c = np.where(src > clip_lo, clip_lo, src)
        else:
            c = src
        if clip_on == "x":
            c = c - m
        e = np.power(2.0, c) if base_e else np.exp(c)
        if drop_last:
            s = np.sum(np.take(e, np.arange(e.shape[axis] - 1), axis=axis),
                       axis=axis, keepdims=True)
        elif denom == "sum":
            s = np.sum(e, axis=axis, keepdims=True)
        elif denom == "mean":
            s = np.mean(e, axis=axis, keepdims=True)
        elif denom == "sum_plus_one":
            s = np.sum(e, axis=axis, keepdims=True) + 1.0
        y = e / s
        return np.asarray(y, dtype=np.float64)


MUTANTS = {
    "reference_copy_is_clean": None,
    "dropped_sum_term": dict(drop_last=True),
    "wrong_sign_shift": "neg",
    "transposed_axis": dict(axis=0),
    "no_clip": dict(clip_kind="none"),
    "clip_as_upper_bound": dict(clip_kind="upper"),
    "clip_constant_-63": dict(clip_lo=-63.0),
    "clip_constant_-65": dict(clip_lo=-65.0),
    "clip_on_raw_logits": dict(clip_on="x"),
    "shift_by_first_element": dict(shift="first"),
    "no_shift": dict(shift="none"),
    "base_2_instead_of_e": dict(base_e=True),
    "mean_instead_of_sum": dict(denom="mean"),
    "off_by_one_denominator": dict(denom="sum_plus_one"),
    # An IEEE max-style clip turns NaN into the bound instead of keeping it.
    # (A NaN-ignoring row max is not listed: the NaN element still poisons
    # the row through its own exp and the sum, so it is an equivalent form.)
    "fmax_clip_drops_nan": dict(clip_kind="fmax"),
    "float32_arithmetic": dict(dtype=np.float32),
}


def _impl(spec):
    if spec is None:
        return lambda x: _base(x)
    if spec == "neg":
        return lambda x: _base(-np.asarray(x, dtype=np.float64))
    return lambda x: _base(x, **spec)


def _failures(impl):
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(impl)
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    failed = _failures(_impl(MUTANTS[name]))
    if MUTANTS[name] is None:
        assert failed == [], failed
    else:
        assert failed, f"mutant {name} passed every pin"


# Mistakes specific to the clip bound as a parameter (impl(x, clip_lo));
# they must each fail at least one of pins.CLIP_PINS.  (An IEEE fmax "clip"
# at -inf is not listed: with no clip a NaN already reaches every shifted
# logit through the row max, so it is an equivalent form.)
def _clip_off_only(spec):
    """Apply the mistake only when the clip is off (clip_lo = -inf)."""
    return lambda x, lo: _base(x, **spec) if lo == -np.inf else _base(x, clip_lo=lo)


MUTANTS_CLIP = {
    "reference_copy_is_clean": lambda x, lo: _base(x, clip_lo=lo),
    "ignores_clip_param": lambda x, lo: _base(x),
    "clip_param_plus_one": lambda x, lo: _base(x, clip_lo=lo + 1.0),
    "clip_param_on_raw_logits": lambda x, lo: _base(x, clip_lo=lo, clip_on="x"),
    "clip_off_keeps_minus_64": _clip_off_only(dict(clip_lo=L)),
    "clip_off_also_drops_shift": _clip_off_only(dict(shift="none", clip_kind="none")),
    "clip_off_float32": _clip_off_only(dict(clip_lo=-np.inf, dtype=np.float32)),
}


def _clip_failures(impl):
    failed = []
    for pin in pins.CLIP_PINS:
        try:
            pin(impl)
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("name", sorted(MUTANTS_CLIP))
def test_clip_mutant_is_caught(name):
    failed = _clip_failures(MUTANTS_CLIP[name])
    if name == "reference_copy_is_clean":
        assert failed == [], failed
    else:
        assert failed, f"mutant {name} passed every clip pin"


# Mistakes in the attention oracle: each must fail at least one of
# pins_attention.ATTN_PINS.
def _attn(q, k, v, scale, lo, axis=-1, scale_pow=1, use_k_as_v=False, clip=True,
          shift=True, normalise=True, v_transposed=False):
    q64, k64, v64 = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    if q64.shape[0] * q64.shape[1] == 0 or v64.shape[2] == 0:
        return np.zeros((q64.shape[0], q64.shape[1], v64.shape[2]))
    s = np.matmul(q64, k64.transpose(0, 2, 1)) * float(scale) ** scale_pow
    with np.errstate(all="ignore"):
        m = np.max(s, axis=axis, keepdims=True) if shift else 0.0
        d = s - m
        if clip:
            d = np.where(d < lo, lo, d)
        e = np.exp(d)
        p = e / np.sum(e, axis=axis, keepdims=True) if normalise else e
        vv = k64 if use_k_as_v else v64
        if v_transposed and vv.shape[1] == vv.shape[2]:
            vv = vv.transpose(0, 2, 1)
        return np.matmul(p, vv) if p.shape[2] == vv.shape[1] else np.matmul(p, v64)


MUTANTS_ATTN = {
    "reference_copy_is_clean": {},
    "softmax_over_queries": dict(axis=1),
    "scale_not_applied": dict(scale_pow=0),
    "scale_applied_twice": dict(scale_pow=2),
    "keys_used_as_values": dict(use_k_as_v=True),
    "no_clip": dict(clip=False),
    "no_max_shift": dict(shift=False),
    "weights_not_normalised": dict(normalise=False),
    "values_transposed": dict(v_transposed=True),
}


@pytest.mark.parametrize("name", sorted(MUTANTS_ATTN))
def test_attention_mutant_is_caught(name):
    from tests import pins_attention
    impl = lambda q, k, v, s, lo: _attn(q, k, v, s, lo, **MUTANTS_ATTN[name])  # noqa: E731
    failed = []
    for pin in pins_attention.ATTN_PINS:
        try:
            pin(impl)
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed.append(pin.__name__)
    if name == "reference_copy_is_clean":
        assert failed == [], failed
    else:
        assert failed, f"mutant {name} passed every attention pin"


# Mistakes in the log of the clipped softmax; each must fail one of
# pins.LOG_PINS.
def _logsm(x, lo, shift=True, clip_sum=True, clip_out=True, base=np.e, via_prob=False,
           sign=1.0):
    x64 = np.asarray(x, dtype=np.float64)
    if x64.size == 0:
        return np.zeros(x64.shape)
    with np.errstate(all="ignore"):
        m = np.max(x64, axis=1, keepdims=True) if shift else 0.0
        d = x64 - m
        c = np.where(d < lo, lo, d)
        s = np.sum(np.exp(c if clip_sum else d), axis=1, keepdims=True)
        if via_prob:
            return np.log(np.exp(c) / s)
        out = c if clip_out else d
        return sign * (out - np.log(s) / np.log(base))


MUTANTS_LOG = {
    "reference_copy_is_clean": {},
    "no_max_shift": dict(shift=False),
    "log_base_2": dict(base=2.0),
    "log_of_underflowed_probability": dict(via_prob=True),
    "output_not_clipped": dict(clip_out=False),
    "sum_not_clipped": dict(clip_sum=False),
    "negated": dict(sign=-1.0),
}


@pytest.mark.parametrize("name", sorted(MUTANTS_LOG))
def test_log_mutant_is_caught(name):
    impl = lambda x, lo: _logsm(x, lo, **MUTANTS_LOG[name])  # noqa: E731
    failed = []
    for pin in pins.LOG_PINS:
        try:
            pin(impl)
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed.append(pin.__name__)
    if name == "reference_copy_is_clean":
        assert failed == [], failed
    else:
        assert failed, f"mutant {name} passed every log pin"


# Mistakes in the per-row negative log-likelihood; each must fail one of
# pins.NLL_PINS.
def _nll(x, labels, lo, shift=True, clip_sum=True, clip_label=True, via_prob=False,
         sign=1.0, label_shift=0, wrap_negative=False, row_mean=False, check_range=True):
    x64 = np.asarray(x, dtype=np.float64)
    t = np.asarray(labels).astype(np.int64)
    rows, cols = x64.shape
    with np.errstate(all="ignore"):
        m = np.max(x64, axis=1, keepdims=True) if shift else 0.0
        d = x64 - m
        c = np.where(d < lo, lo, d)
        s = np.sum(np.exp(c if clip_sum else d), axis=1)
        logp = (np.log(np.exp(c) / s[:, None]) if via_prob
                else (c if clip_label else d) - np.log(s)[:, None])
        if row_mean:
            return sign * -np.mean(logp, axis=1)
        tt = (t + label_shift) % cols if label_shift else t
        if wrap_negative:
            tt = np.where(tt < 0, tt % cols, tt)
        valid = (tt >= 0) & (tt < cols) if check_range else np.ones(rows, bool)
        picked = logp[np.arange(rows), np.clip(tt, 0, cols - 1)]
        return np.where(valid, sign * -picked, np.nan)


MUTANTS_NLL = {
    "reference_copy_is_clean": {},
    "no_max_shift": dict(shift=False),
    "sum_not_clipped": dict(clip_sum=False),
    "label_term_not_clipped": dict(clip_label=False),
    "log_of_underflowed_probability": dict(via_prob=True),
    "log_probability_not_negated": dict(sign=-1.0),
    "label_off_by_one": dict(label_shift=1),
    "negative_label_wraps": dict(wrap_negative=True),
    "out_of_range_label_clamped": dict(check_range=False),
    "mean_over_classes": dict(row_mean=True),
}


@pytest.mark.parametrize("name", sorted(MUTANTS_NLL))
def test_nll_mutant_is_caught(name):
    impl = lambda x, t, lo: _nll(x, t, lo, **MUTANTS_NLL[name])  # noqa: E731
    failed = []
    for pin in pins.NLL_PINS:
        try:
            pin(impl)
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            failed.append(pin.__name__)
    if name == "reference_copy_is_clean":
        assert failed == [], failed
    else:
        assert failed, f"mutant {name} passed every NLL pin"
