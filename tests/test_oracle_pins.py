"""The float64 oracle against facts fixed by the paper and by mathematics."""
import numpy as np
import pytest

import oracle
from tests import pins, pins_attention


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle.softmax_clipped)


@pytest.mark.parametrize("pin", pins.CLIP_PINS, ids=lambda p: p.__name__)
def test_oracle_clip_pin(pin):
    pin(oracle.softmax_clipped)


def test_row_max_exact_and_nan():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((9, 77)).astype(np.float32)
    m = oracle.row_max(x)
    for i in range(9):
        assert m[i, 0] == max(float(v) for v in x[i])
    x[4, 10] = np.nan
    assert np.isnan(oracle.row_max(x)[4, 0])


def test_exp_clipped_decimal():
    """exp of clipped arguments against 50-digit decimal exp."""
    from decimal import Decimal, getcontext
    getcontext().prec = 50
    rng = np.random.default_rng(4)
    d = np.concatenate([rng.uniform(-80.0, 0.0, 2000), [-64.0, -63.999, -64.001, 0.0]])
    got = oracle.exp_clipped(d)
    for di, gi in zip(d, got):
        c = max(Decimal(float(di)), Decimal(-64))
        want = float(c.exp())
        assert abs(gi - want) <= np.finfo(np.float64).eps * want  # < 1 ulp


def test_workloads_oracle_invariants():
    """The oracle on the five workloads: sums to 1, bounded below, finite."""
    import workloads
    for key in workloads.WORKLOADS:
        if workloads.WORKLOADS[key].elements > 5_000_000:
            continue
        x = workloads.generate(key)
        y = oracle.softmax_clipped(x)
        assert np.all(np.isfinite(y))
        assert np.max(np.abs(y.sum(axis=1) - 1.0)) < 1e-12
        assert np.all(y >= np.exp(-64.0) / x.shape[1] * (1 - 1e-12))


@pytest.mark.parametrize("pin", pins_attention.ATTN_PINS, ids=lambda p: p.__name__)
def test_attention_oracle_pin(pin):
    pin(oracle.attention_clipped)


def test_attention_oracle_rejects_zero_keys():
    import workloads
    q, k, v = workloads.random_qkv(2, 3, 0, 4, 5, 1)
    with pytest.raises(ValueError):
        oracle.attention_clipped(q, k, v, 1.0)


@pytest.mark.parametrize("pin", pins.LOG_PINS, ids=lambda p: p.__name__)
def test_log_oracle_pin(pin):
    pin(oracle.log_softmax_clipped)


@pytest.mark.parametrize("pin", pins.NLL_PINS, ids=lambda p: p.__name__)
def test_nll_oracle_pin(pin):
    pin(oracle.nll_clipped)


def test_nll_oracle_rejects_bad_labels():
    with pytest.raises(ValueError):
        oracle.nll_clipped(np.zeros((2, 3), np.float32), np.zeros(3, np.int64))
    with pytest.raises(ValueError):
        oracle.nll_clipped(np.zeros((2, 3), np.float32), np.zeros(2, np.float64))
    with pytest.raises(ValueError):
        oracle.nll_clipped(np.zeros((2, 0), np.float32), np.zeros(2, np.int64))
    assert oracle.nll_clipped(np.zeros((0, 3), np.float32), np.zeros(0, np.int64)).shape == (0,)
