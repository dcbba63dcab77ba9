"""Pins for the oracle's routing and compaction layout (CPU only)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.route import (bucket_set, bucket_of, padding_waste_ratio, coarse_class,
                          route_batch, repack_rows)
from conftest import GOLDEN


def load_cases():
    with open(os.path.join(GOLDEN, "routing_cases.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", load_cases(), ids=lambda c: c["name"])
def test_routing_golden(case):
    B = len(case["keep_len"])
    r = route_batch(case["keep_len"], [case["win_len"]] * B, case["policy"])
    assert list(r.path) == case["path"], case["why"]
    assert list(r.group) == case["group"], case["why"]
    assert list(r.alloc) == case["alloc"], case["why"]
    assert len(r.groups) == len(case["groups"])
    for g, e in zip(r.groups, case["groups"]):
        assert g["bucket"] == e["bucket"]
        assert g["pwr"] == (None if e["pwr"] is None else Fraction(*e["pwr"]))


def test_bucket_set_and_lookup():
    assert bucket_set(1024) == [8, 16, 32, 64, 128, 256, 512, 1024]
    assert bucket_set(100) == [8, 16, 32, 64, 100]
    assert bucket_set(8) == [8]
    assert bucket_set(5) == [5]
    assert bucket_of(1, 1024) == 8 and bucket_of(8, 1024) == 8 and bucket_of(9, 1024) == 16
    assert bucket_of(513, 1024) == 1024 and bucket_of(65, 100) == 100
    with pytest.raises(ValueError):
        bucket_of(101, 100)


def test_pwr_closed_forms():
    assert padding_waste_ratio([16, 16], 16) == 0
    assert padding_waste_ratio([1], 8) == Fraction(7, 8)
    assert padding_waste_ratio([10, 12, 14, 60], 64) == Fraction(5, 8)


def test_coarse_class_edges():
    assert [coarse_class(L) for L in (1, 8, 16, 17, 64, 65, 256, 257, 1024, 1025)] == \
        [2, 2, 2, 3, 3, 4, 4, 5, 5, 6]


def test_hybrid_routing_properties():
    """Every sequence gets one path; static allocations are buckets >= L*."""
    rng = np.random.default_rng(21)
    for _ in range(200):
        B = int(rng.integers(1, 40))
        N = int(rng.choice([64, 100, 1024, 2048]))
        keep = rng.integers(1, N + 1, size=B)
        r = route_batch(keep, [N] * B)
        for i in range(B):
            assert r.path[i] in (0, 1, 2)
            if r.path[i] == 0:
                assert r.alloc[i] >= keep[i] and r.alloc[i] in bucket_set(N)
            else:
                assert r.alloc[i] == keep[i]
        for g in r.groups:
            lens = [int(keep[i]) for i in g["members"]]
            assert g["pwr"] == padding_waste_ratio(lens, g["bucket"])
            if g["path"] == 0:
                assert g["pwr"] <= Fraction(1, 5) and len(lens) > 1
            if g["path"] == 1:
                assert g["pwr"] > Fraction(1, 5) and len(lens) > 1 and max(lens) > 4
        # naive pad: everybody padded to the batch-max bucket
        rn = route_batch(keep, [N] * B, policy=1)
        assert set(rn.alloc) == {bucket_of(int(keep.max()), N)}


def test_repack_layout_and_contents():
    rng = np.random.default_rng(22)
    d = 5
    pre = [3, 4, 2]
    win = [6, 6, 8]
    lens = [p + w for p, w in zip(pre, win)]
    cu_src = np.concatenate([[0], np.cumsum(lens)])
    src = rng.standard_normal((cu_src[-1], d))
    keep = [2, 6, 1]
    alloc = [4, 6, 1]
    dst, cu_dst, used, cap = repack_rows(src, cu_src, pre, keep, alloc, granule=8)
    assert list(cu_dst) == [0, 3 + 4, 3 + 4 + 4 + 6, 3 + 4 + 4 + 6 + 2 + 1]
    assert cap == 24 and dst.shape == (24, d)
    assert list(used) == [5, 10, 3]
    for b in range(3):
        n = pre[b] + keep[b]
        np.testing.assert_array_equal(dst[cu_dst[b]:cu_dst[b] + n], src[cu_src[b]:cu_src[b] + n])
        np.testing.assert_array_equal(dst[cu_dst[b] + n:cu_dst[b + 1]], 0.0)
    np.testing.assert_array_equal(dst[cu_dst[-1]:], 0.0)
