"""Pins for the oracle's sparsity count and SNR boundary criterion (CPU only)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.detect import detect_boundary, detect_batch
from oracle.sparsity import near_zero_count, sparsity_fraction
from conftest import GOLDEN


def load_cases():
    with open(os.path.join(GOLDEN, "detector_cases.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", load_cases(), ids=lambda c: c["name"])
def test_detector_golden(case):
    got = detect_boundary(case["counts"], case["d_ff"], Fraction(*case["tau"]),
                          Fraction(*case["gamma"]), case["lookahead"])
    assert got == (case["boundary"], case["keep_len"]), case["why"]


def brute_integer_scan(counts, I, tn, td, gn, gd, w):
    """All qualifying positions, cross-multiplied in integers (no fractions)."""
    hits = []
    n = len(counts)
    for i in range(1, n):
        if i + w > n:
            break
        win = counts[i:i + w]
        dj = min(win) - counts[i - 1]
        dn = max(win) - min(win)
        if td * dj >= tn * I and gd * dn <= gn * dj:
            hits.append(i)
    return hits


def test_detector_against_integer_brute_force():
    rng = np.random.default_rng(11)
    for trial in range(400):
        n = int(rng.integers(1, 40))
        I = int(rng.integers(5, 300))
        base = rng.integers(0, I // 2 + 1)
        counts = np.clip(base + rng.integers(-I // 8 - 1, I // 8 + 2, size=n), 0, I)
        if trial % 3 == 0 and n > 4:      # plant a step
            j = int(rng.integers(1, n))
            counts[j:] = np.minimum(counts[j:] + I // 5, I)
        w = int(rng.integers(1, 5))
        tn, td = int(rng.integers(1, 10)), 100
        gn, gd = int(rng.integers(1, 5)), 5
        hits = brute_integer_scan(list(map(int, counts)), I, tn, td, gn, gd, w)
        expect = (hits[0], hits[0] + 1) if hits else (n, n)
        assert detect_boundary(counts, I, Fraction(tn, td), Fraction(gn, gd), w) == expect


def test_detector_monotone_in_tau_and_gamma():
    """Smaller tau or larger gamma never cuts later (cf. the hyper-parameter study)."""
    rng = np.random.default_rng(12)
    for _ in range(200):
        n = 30
        I = 200
        counts = rng.integers(0, 60, size=n)
        counts[int(rng.integers(3, n)):] += int(rng.integers(0, 40))
        taus = [Fraction(k, 100) for k in (1, 2, 3, 5, 8)]
        prev = -1
        for t in reversed(taus):   # decreasing tau
            b, _ = detect_boundary(counts, I, t, Fraction(3, 5), 3)
            if prev >= 0:
                assert b <= prev
            prev = b
        prev = None
        for g in [Fraction(k, 10) for k in (2, 4, 6, 8, 10)]:
            b, _ = detect_boundary(counts, I, Fraction(3, 100), g, 3)
            if prev is not None:
                assert b <= prev
            prev = b


def test_detect_batch_uses_window_slices():
    counts = np.array([99, 99, 10, 10, 40, 40, 40, 3, 3, 3, 7, 7, 20, 20, 20], np.int64)
    cu = np.array([0, 7, 15])
    win_off = np.array([2, 3])
    win_len = np.array([5, 5])
    b, k = detect_batch(counts, cu, win_off, win_len, 100)
    # seq 0 window = [10,10,40,40,40] -> i*=2; seq 1 window = [7,7,20,20,20] -> i*=2
    assert list(b) == [2, 2] and list(k) == [3, 3]


def test_count_special_cases():
    rng = np.random.default_rng(13)
    act = rng.standard_normal((4, 50))
    assert np.all(near_zero_count(act, 0.0) == 0)
    assert np.all(near_zero_count(act, np.inf) == 50)
    assert np.all(near_zero_count(np.zeros((3, 9)), 1e-30) == 9)
    row = np.array([[0.5, -0.5, 0.49, -0.49, 0.0, 1.0, -2.0]])
    assert near_zero_count(row, 0.5)[0] == 3   # strict: |0.5| is not < 0.5


def test_count_against_loops():
    rng = np.random.default_rng(14)
    act = rng.standard_normal((6, 33)) * 0.1
    eps = 0.03
    c = near_zero_count(act, eps)
    for r in range(6):
        assert c[r] == sum(1 for v in act[r] if abs(v) < eps)


def test_sparsity_fraction_hand_values():
    """The statistic is count / I (Sec. 3.2-3.3): hand values with I = 688 (the
    tiny layer's SwiGLU width, not a power of two) and I = 12288; a fraction
    divided by the model width instead (256 or 4096) fails every nonzero case."""
    f = sparsity_fraction(np.array([0, 1, 43, 344, 688]), 688)
    np.testing.assert_array_equal(f, [0.0, 1.0 / 688, 0.0625, 0.5, 1.0])
    f = sparsity_fraction(np.array([[3072, 12288], [0, 96]]), 12288)
    np.testing.assert_array_equal(f, [[0.25, 1.0], [0.0, 0.0078125]])
    # as the count's companion: an all-near-zero row is fraction 1, none is 0
    act = np.array([[0.0, 1e-9, -1e-9, 0.0], [5.0, -5.0, 6.0, -7.0]])
    np.testing.assert_array_equal(sparsity_fraction(near_zero_count(act, 1e-3), 4), [1.0, 0.0])
