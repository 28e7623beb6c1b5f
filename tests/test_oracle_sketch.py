"""Pins for the oracle's ROI length sketch (no GPU): CV = sigma / mu of realised lengths
(population sigma) and f_s = Pr[l < L_max / 4], checked against closed forms, boundary
cases worked by hand and numpy's own moments."""
import math

import numpy as np
import pytest

import oracle


def offsets(lens):
    return np.concatenate([[0], np.cumsum(np.asarray(lens, dtype=np.int64))])


def test_hand_worked_example():
    # l = 3, 7, 2: mu = 4, sigma^2 = (1 + 9 + 4) / 3 = 14/3; L_max = 16: l < 4 for 3 and 2
    s = oracle.length_sketch(offsets([3, 7, 2]), None, 16)
    assert (s["samples"], s["short_samples"], s["sum_len"], s["sum_sq"]) == (3, 2, 12, 62)
    assert (s["min_len"], s["max_len"], s["mean"]) == (2, 7, 4.0)
    assert abs(s["cv"] - math.sqrt(14 / 3) / 4) <= 1e-15 * s["cv"]
    assert s["short_fraction"] == 2 / 3 and s["high_roi"] == 1


@pytest.mark.parametrize("a,b,k", [(1, 3, 5), (100, 900, 1000), (512, 513, 7), (8, 16384, 2)])
def test_two_point_closed_form(a, b, k):
    # k samples of a and k of b: mu = (a+b)/2, population sigma = (b-a)/2
    s = oracle.length_sketch(offsets([a] * k + [b] * k), None, 4 * b + 4)
    want = (b - a) / (a + b)
    assert abs(s["cv"] - want) <= 2e-16 * want
    assert s["short_fraction"] == 1.0
    # a sample standard deviation (n - 1) would be larger by sqrt(2k / (2k - 1))
    assert abs(s["cv"] - want * math.sqrt(2 * k / (2 * k - 1))) > 1e-6 * want


def test_constant_lengths():
    s = oracle.length_sketch(offsets([37] * 100), None, 148)
    assert s["cv"] == 0.0 and s["short_fraction"] == 0.0 and s["high_roi"] == 0   # 37 = 148/4 is not short
    s = oracle.length_sketch(offsets([37] * 100), None, 149)
    assert s["short_fraction"] == 1.0 and s["high_roi"] == 1


def test_short_boundary():
    # L_max = 10: L/4 = 2.5, so l = 2 is short and l = 3 is not; L_max = 16: l = 4 is not
    assert oracle.length_sketch(offsets([1, 2, 3, 4]), None, 10)["short_samples"] == 2
    assert oracle.length_sketch(offsets([3, 4, 5]), None, 16)["short_samples"] == 1
    assert oracle.length_sketch(offsets([5]), None, 1)["short_samples"] == 0


def test_against_numpy_moments_and_id_subsets():
    rng = np.random.default_rng(41)
    lens = np.maximum(1, np.rint(rng.lognormal(6.0, 0.9, size=40000))).astype(np.int64)
    off = offsets(lens)
    for ids in (None, rng.choice(len(lens), size=5000, replace=False), np.array([7, 7, 7, 9]),
                np.arange(len(lens))[::3]):
        sub = lens if ids is None else lens[ids]
        s = oracle.length_sketch(off, ids, 8192)
        assert s["samples"] == len(sub) and s["sum_len"] == int(sub.sum())
        assert s["sum_sq"] == int((sub.astype(object) ** 2).sum())
        assert abs(s["cv"] - np.std(sub) / np.mean(sub)) <= 1e-12 * s["cv"]
        assert s["short_fraction"] == np.count_nonzero(4 * sub < 8192) / len(sub)
        assert (s["min_len"], s["max_len"]) == (int(sub.min()), int(sub.max()))


def test_high_roi_screen():
    # CV >= 0.8 or f_s > 0.2
    lo_cv_many_short = offsets([10] * 30 + [12] * 70)          # CV small, f_s = 1
    assert oracle.length_sketch(lo_cv_many_short, None, 100)["high_roi"] == 1
    assert oracle.length_sketch(lo_cv_many_short, None, 40)["high_roi"] == 0   # nothing below 10
    s = oracle.length_sketch(offsets([1] * 10 + [100] * 10), None, 4)        # CV = 99/101, f_s = 0
    assert s["short_fraction"] == 0.0 and s["cv"] > 0.8 and s["high_roi"] == 1
    s = oracle.length_sketch(offsets([100] * 79 + [10] * 21), None, 41)      # f_s = 0.21 > 0.2
    assert s["cv"] < 0.8 and s["high_roi"] == 1
    s = oracle.length_sketch(offsets([100] * 80 + [10] * 20), None, 41)      # f_s = 0.2 exactly
    assert s["cv"] < 0.8 and s["high_roi"] == 0


def test_empty_and_invalid():
    s = oracle.length_sketch(offsets([5, 6]), np.zeros(0, np.int64), 10)
    assert s["samples"] == 0 and s["cv"] == 0.0 and s["high_roi"] == 0
    with pytest.raises(oracle.OracleError):
        oracle.length_sketch(offsets([5, 6]), np.array([2]), 10)
    with pytest.raises(oracle.OracleError):
        oracle.length_sketch(np.array([0, 4, 4]), None, 10)
