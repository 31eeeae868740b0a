"""Seeded scene generators: determinism, uniqueness and calibrated sizes."""
import numpy as np
import pytest

from paper_2401_06145_amd import scenes

TARGETS = {0: 2000, 1: 120_000, 2: 200_000, 3: 300_000, 4: 240_000}


@pytest.mark.parametrize("i", range(5))
def test_workload_sizes_and_uniqueness(i):
    w = scenes.workload(i)
    c = w.coords
    assert c.dtype == np.int32 and c.shape[1] == 4
    assert abs(c.shape[0] - TARGETS[i]) <= 0.03 * TARGETS[i]
    assert np.unique(c, axis=0).shape[0] == c.shape[0]
    # rows are not given in sorted order
    assert not np.array_equal(c, np.unique(c, axis=0))


def test_deterministic():
    a = scenes.workload(1).coords
    b = scenes.workload(1).coords
    assert scenes.coords_sha256(a) == scenes.coords_sha256(b)
    f1 = scenes.features(10, 4, "f16", 5)
    f2 = scenes.features(10, 4, "f16", 5)
    assert f1.dtype == np.float16 and np.array_equal(f1, f2)


def test_ranges():
    c = scenes.workload(1).coords
    assert c[:, 1].min() >= -1000 and c[:, 1].max() <= 999
    assert c[:, 3].min() >= 0 and c[:, 3].max() <= 159
    c = scenes.workload(3).coords
    assert c[:, 1].max() <= 499 and c[:, 2].max() <= 399 and c[:, 3].max() <= 149
    c = scenes.workload(4).coords
    assert set(np.unique(c[:, 0]).tolist()) == {0, 1}


def test_bf16_rounding():
    v = np.array([1.0, 1.00390625, 1.01171875, -3.0e-3, 65504.0])
    u = scenes._round_to(v, "bf16")
    back = scenes.bf16_bits_to_f64(u)
    # exact for representable values; RNE ties to even for 1 + 2^-8 -> 1.0
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.015625
    assert np.all(np.abs(back - v) <= np.abs(v) * 2.0 ** -8)


def test_weight_scale():
    w = scenes.weights(3, 64, 64, "f16", 1).astype(np.float64)
    assert w.shape == (27, 64, 64)
    assert abs(w.std() - 1 / np.sqrt(27 * 64)) < 0.05 / np.sqrt(27 * 64)
