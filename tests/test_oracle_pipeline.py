"""Pins for the oracle's end-to-end step-0 pipeline (CPU only).

Planted-boundary inputs: the window holds content rows up to b and the shared
EOS vector (plus small noise) from b on, so the cut index is known: the first
EOS position b is i*, and L* = b + 1.
"""
import numpy as np
import pytest

import oracle
from oracle.layer import layer_forward
from workloads import WORKLOADS, scaled
from workloads.generate import make_workload


def run(w, **kw):
    layers, batch = make_workload(w)
    res = oracle.run_pipeline(layers, batch.x, batch.cu_seqlens, batch.win_off, batch.win_len,
                              w.shape.n_heads, w.shape.d_ff, w.rms_eps, w.act_eps, w.l_det, **kw)
    return layers, batch, res


def test_tiny_planted_boundary_detected():
    w = WORKLOADS["tiny_f32"]
    layers, batch, res = run(w)
    assert int(batch.planted[0]) == 40
    assert list(res.boundary) == [40] and list(res.keep_len) == [41]


def test_tiny_truncated_step_equals_physically_cut_window():
    w = WORKLOADS["tiny_f32"]
    layers, batch, res = run(w)
    S = w.prefix_len + int(res.keep_len[0])
    x_cut = batch.x[:S]
    y_cut, _ = layer_forward(x_cut, [0, S], layers[0], w.shape.n_heads, w.rms_eps)
    np.testing.assert_array_equal(res.y_step[:S], y_cut)
    # and step 0's output for the kept rows is the full-window output of those rows
    y_full, _ = layer_forward(batch.x, batch.cu_seqlens, layers[0], w.shape.n_heads, w.rms_eps)
    np.testing.assert_array_equal(res.y_step0[:S], y_full[:S])


def test_small_ragged_batch_planted_boundaries():
    """A small ragged batch (tiny layer shape) with planted cuts at several depths."""
    w = scaled(WORKLOADS["tiny_f32"], batch=5, boundary=("uniform", 12, 100), seed=77)
    layers, batch, res = run(w)
    np.testing.assert_array_equal(res.boundary, batch.planted)
    np.testing.assert_array_equal(res.keep_len, batch.planted + 1)
    # compacted layout: prefix + L* rows per sequence (plus static padding)
    for b in range(w.batch):
        n = int(res.cu_trunc[b + 1] - res.cu_trunc[b])
        assert n == w.prefix_len + int(res.route.alloc[b])
        assert int(res.seqused[b]) == w.prefix_len + int(res.keep_len[b])


def test_two_layer_stack_detects_after_layer_one():
    w = scaled(WORKLOADS["tiny_f32"], n_layers=2, l_det=1, batch=2,
               boundary=("uniform", 20, 90), seed=91)
    layers, batch, res = run(w)
    np.testing.assert_array_equal(res.boundary, batch.planted)


def test_no_eos_suffix_keeps_whole_window():
    """A window of pure content has no jump-plateau: nothing is cut."""
    w = scaled(WORKLOADS["tiny_f32"], boundary=("fixed", 127), seed=5)
    layers, batch, res = run(w)
    # with the EOS only at the last position there is no 3-position plateau
    assert list(res.keep_len) == [128]
