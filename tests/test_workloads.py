"""Seeded workload generators: frozen bytes and the stated structure."""
import json
import os

import numpy as np
import pytest

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "input_sha256.json")


@pytest.mark.parametrize("key", list(workloads.WORKLOADS))
def test_generator_bytes_frozen(key):
    with open(GOLDEN) as f:
        want = json.load(f)[key]
    x = workloads.generate(key)
    w = workloads.WORKLOADS[key]
    assert x.dtype == np.float32 and x.flags.c_contiguous
    assert x.shape == (w.rows, w.cols) == (want["rows"], want["cols"])
    assert workloads.sha256_f32(x) == want["sha256"]


def test_structure_of_each_workload():
    x = workloads.generate(1)
    assert x.min() >= -10 and x.max() <= 10
    x = workloads.generate(2)                  # DAM scores ~ N(0, 1)
    assert abs(float(x.std()) - 1.0) < 0.01 and abs(float(x.mean())) < 0.01
    x = workloads.generate(3)                  # one +8 class per row
    assert x.shape == (4096, 1000)
    assert float(np.mean(x.max(axis=1))) > 9.0
    x = workloads.generate(4)
    d = x.astype(np.float64) - x.max(axis=1, keepdims=True)
    frac = float(np.mean(d < -64.0))
    assert 0.055 < frac < 0.065                # ~5% masked + outlier rows
    assert int(np.sum(x.max(axis=1) > 60)) == 5
    x = workloads.generate(5)
    means = x.mean(axis=1)
    assert means.min() < -40 and means.max() > 40


def test_random_logits_kinds():
    for kind in ("normal", "uniform", "clip_heavy", "offset", "dyadic"):
        x = workloads.random_logits(5, 33, 1, kind)
        assert x.shape == (5, 33) and x.dtype == np.float32
    assert workloads.random_logits(0, 7, 1, "clip_heavy").shape == (0, 7)
