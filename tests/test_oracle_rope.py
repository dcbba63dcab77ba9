"""Pins of the oracle's rotary position embedding (CPU).

* hand values: head width 4, theta 10000, position 1 rotates the pair
  (0, 2) by 1 rad and the pair (1, 3) by 0.01 rad, with the sign convention
  x2' = x2 cos + x1 sin;
* position 0 is the identity; every rotated pair keeps its norm;
* the complex form: z_j = x_j + i x_{j+dh/2} becomes z_j e^{i pos theta_j};
* attention logits depend only on relative positions: shifting every
  position by the same amount leaves q.k unchanged, and a whole layer's
  output with it;
* with the embedding on, a layer is no longer permutation-equivariant;
* the cached step (prefix keys rotated at their positions, window rows at
  P + i) equals the full step on the window rows.
"""
import numpy as np

from oracle.kvcache import layer_forward_cached_rows, prefix_kv
from oracle.layer import layer_forward_rows
from oracle.rope import apply_rope, rope_angles


def _layer(rng, d, I):
    W = {k: rng.standard_normal(s) / np.sqrt(s[1]) for k, s in
         [("wq", (d, d)), ("wk", (d, d)), ("wv", (d, d)), ("wo", (d, d)),
          ("wg", (I, d)), ("wu", (I, d)), ("wd", (d, I))]}
    W["g1"] = 1.0 + 0.1 * rng.standard_normal(d)
    W["g2"] = 1.0 + 0.1 * rng.standard_normal(d)
    return W


def test_hand_values():
    x = np.array([[1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0]])
    y = apply_rope(x, [1, 1], 1, 10000.0)
    c1, s1 = 0.5403023058681398, 0.8414709848078965            # cos 1, sin 1
    c2, s2 = 0.9999500004166653, 0.009999833334166664          # cos 0.01, sin 0.01
    np.testing.assert_allclose(y[0], [c1, 0.0, s1, 0.0], atol=1e-15)
    np.testing.assert_allclose(y[1], [0.0, c2, 0.0, s2], atol=1e-15)
    # the second feature of a pair picks up -sin
    y = apply_rope(np.array([[0.0, 0.0, 1.0, 0.0]]), [1], 1, 10000.0)
    np.testing.assert_allclose(y[0], [-s1, 0.0, c1, 0.0], atol=1e-15)
    a = rope_angles([3], 8, 100.0)[0]
    np.testing.assert_allclose(a, [3.0, 3.0 / 100 ** 0.25, 3.0 / 100 ** 0.5, 3.0 / 100 ** 0.75], rtol=1e-15)


def test_identity_and_norms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((9, 64))
    assert np.array_equal(apply_rope(x, np.zeros(9), 4, 500000.0), x)
    pos = rng.integers(0, 5000, 9)
    y = apply_rope(x, pos, 4, 500000.0)
    for h in range(4):
        for j in range(8):
            a, b = h * 16 + j, h * 16 + j + 8
            np.testing.assert_allclose(np.hypot(y[:, a], y[:, b]), np.hypot(x[:, a], x[:, b]), rtol=1e-13)


def test_complex_form():
    rng = np.random.default_rng(1)
    n, H, dh, theta = 7, 3, 32, 10000.0
    x = rng.standard_normal((n, H * dh))
    pos = rng.integers(0, 4096, n)
    y = apply_rope(x, pos, H, theta)
    for h in range(H):
        z = x[:, h * dh:h * dh + dh // 2] + 1j * x[:, h * dh + dh // 2:(h + 1) * dh]
        freq = theta ** (-np.arange(0, dh, 2) / dh)
        zr = z * np.exp(1j * np.outer(pos, freq))
        np.testing.assert_allclose(y[:, h * dh:h * dh + dh // 2], zr.real, atol=1e-12)
        np.testing.assert_allclose(y[:, h * dh + dh // 2:(h + 1) * dh], zr.imag, atol=1e-12)


def test_logits_depend_on_relative_position():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal((5, 64)), rng.standard_normal((6, 64))
    pq, pk = rng.integers(0, 3000, 5), rng.integers(0, 3000, 6)
    s0 = apply_rope(q, pq, 2, 500000.0) @ apply_rope(k, pk, 2, 500000.0).T
    s1 = apply_rope(q, pq + 1234, 2, 500000.0) @ apply_rope(k, pk + 1234, 2, 500000.0).T
    np.testing.assert_allclose(s1, s0, rtol=1e-10, atol=1e-10)
    s2 = apply_rope(q, pq + 1, 2, 500000.0) @ apply_rope(k, pk, 2, 500000.0).T
    assert np.max(np.abs(s2 - s0)) > 1e-3


def test_layer_shift_invariance_and_order():
    rng = np.random.default_rng(3)
    d, H, I, S, used = 32, 2, 48, 11, 9
    W = _layer(rng, d, I)
    x = rng.standard_normal((S, d))
    rows = np.arange(S)
    y0 = layer_forward_rows(x, used, W, H, 1e-5, rows, rope_theta=10000.0)["y"]
    y1 = layer_forward_rows(x, used, W, H, 1e-5, rows, rope_theta=10000.0, pos_offset=517)["y"]
    np.testing.assert_allclose(y1, y0, rtol=1e-10, atol=1e-10)
    # without positions, swapping two real rows just swaps their outputs; with them it does not
    perm = np.arange(S)
    perm[[1, 4]] = perm[[4, 1]]
    yn = layer_forward_rows(x, used, W, H, 1e-5, rows)["y"]
    ynp = layer_forward_rows(x[perm], used, W, H, 1e-5, rows)["y"]
    np.testing.assert_allclose(ynp, yn[perm], rtol=1e-12, atol=1e-12)
    yrp = layer_forward_rows(x[perm], used, W, H, 1e-5, rows, rope_theta=10000.0)["y"]
    assert np.max(np.abs(yrp - y0[perm])) > 1e-4


def test_cached_step_with_rope_equals_full_step():
    rng = np.random.default_rng(4)
    d, H, I, P, Sw, used = 32, 2, 48, 13, 8, 6
    W = _layer(rng, d, I)
    x = rng.standard_normal((P + Sw, d))
    full = layer_forward_rows(x, P + used, W, H, 1e-5, np.arange(P, P + Sw), rope_theta=10000.0)["y"]
    k_pre, v_pre = prefix_kv(x, W, 1e-5, P, n_heads=H, rope_theta=10000.0)
    cached = layer_forward_cached_rows(x[P:], used, k_pre, v_pre, W, H, 1e-5, rope_theta=10000.0)["y"]
    np.testing.assert_allclose(cached, full, rtol=1e-12, atol=1e-12)
    # the cached prefix keys must carry their own positions
    k_bad, _ = prefix_kv(x, W, 1e-5, P)
    bad = layer_forward_cached_rows(x[P:], used, k_bad, v_pre, W, H, 1e-5, rope_theta=10000.0)["y"]
    assert np.max(np.abs(bad - full)) > 1e-4
