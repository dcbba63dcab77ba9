"""Pins for the oracle's layer forward (CPU only).

The oracle is checked against things other than itself:
  * torch's own CPU float64 routines (linear, scaled_dot_product_attention,
    rms_norm, silu) composed into the same pre-norm layer -- a library
    definition of every operand orientation;
  * explicit scalar loops on a tiny shape (brute force);
  * invariants: attention rows sum to one (mass conservation, Sec. 3.6),
    identical values give the value back, zero output projections give the
    identity, truncated-then-forwarded rows equal the physically cut window,
    batch-permutation equivariance.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle.layer import softmax_rows, attention_seq, layer_forward, layer_forward_rows


def rand_layer(rng, d, I, std=0.2):
    W = {
        "wq": rng.standard_normal((d, d)) * std, "wk": rng.standard_normal((d, d)) * std,
        "wv": rng.standard_normal((d, d)) * std, "wo": rng.standard_normal((d, d)) * std,
        "wg": rng.standard_normal((I, d)) * std, "wu": rng.standard_normal((I, d)) * std,
        "wd": rng.standard_normal((d, I)) * std,
        "g1": 1.0 + 0.1 * rng.standard_normal(d), "g2": 1.0 + 0.1 * rng.standard_normal(d),
    }
    return W


def torch_layer(x, W, n_heads, eps):
    """The same layer composed from torch library routines (float64, CPU)."""
    t = {k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in W.items()}
    x = torch.from_numpy(np.asarray(x, np.float64))
    S, d = x.shape
    dh = d // n_heads
    a = F.rms_norm(x, (d,), weight=t["g1"], eps=eps)
    q = F.linear(a, t["wq"]).view(S, n_heads, dh).transpose(0, 1)
    k = F.linear(a, t["wk"]).view(S, n_heads, dh).transpose(0, 1)
    v = F.linear(a, t["wv"]).view(S, n_heads, dh).transpose(0, 1)
    o = F.scaled_dot_product_attention(q, k, v, is_causal=False)
    o = o.transpose(0, 1).reshape(S, d)
    h1 = x + F.linear(o, t["wo"])
    b = F.rms_norm(h1, (d,), weight=t["g2"], eps=eps)
    act = F.silu(F.linear(b, t["wg"])) * F.linear(b, t["wu"])
    return (h1 + F.linear(act, t["wd"])).numpy(), act.numpy()


@pytest.mark.parametrize("S,d,H,I", [(7, 16, 2, 24), (33, 64, 4, 40), (1, 8, 1, 8)])
def test_layer_matches_torch_library(S, d, H, I):
    rng = np.random.default_rng(S * 100 + d)
    W = rand_layer(rng, d, I)
    x = rng.standard_normal((S, d))
    y, _ = layer_forward(x, [0, S], W, H, 1e-5)
    r = layer_forward_rows(x, S, W, H, 1e-5, np.arange(S), want_act=True)
    y_t, act_t = torch_layer(x, W, H, 1e-5)
    np.testing.assert_allclose(y, y_t, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(r["act"], act_t, rtol=1e-12, atol=1e-12)


def brute_layer(x, W, H, eps):
    """Scalar loops over every index: no matrix routine at all."""
    S, d = len(x), len(x[0])
    I = len(W["wg"])
    dh = d // H

    def rms(v, g):
        ms = sum(e * e for e in v) / d
        return [v[j] / math.sqrt(ms + eps) * g[j] for j in range(d)]

    def lin(v, w):
        return [sum(w[o][i] * v[i] for i in range(len(v))) for o in range(len(w))]

    a = [rms(x[s], W["g1"]) for s in range(S)]
    q = [lin(a[s], W["wq"]) for s in range(S)]
    k = [lin(a[s], W["wk"]) for s in range(S)]
    v = [lin(a[s], W["wv"]) for s in range(S)]
    y = []
    for s in range(S):
        o = [0.0] * d
        for h in range(H):
            logits = []
            for t in range(S):
                logits.append(sum(q[s][h * dh + j] * k[t][h * dh + j] for j in range(dh)) / math.sqrt(dh))
            m = max(logits)
            ex = [math.exp(e - m) for e in logits]
            z = sum(ex)
            for j in range(dh):
                o[h * dh + j] = sum(ex[t] / z * v[t][h * dh + j] for t in range(S))
        h1 = [x[s][j] + lin(o, W["wo"])[j] for j in range(d)]
        b = rms(h1, W["g2"])
        g = lin(b, W["wg"])
        u = lin(b, W["wu"])
        act = [g[i] / (1 + math.exp(-g[i])) * u[i] for i in range(I)]
        dn = lin(act, W["wd"])
        y.append([h1[j] + dn[j] for j in range(d)])
    return np.array(y)


def test_layer_matches_scalar_loops():
    rng = np.random.default_rng(7)
    d, H, I, S = 8, 2, 12, 5
    W = rand_layer(rng, d, I, std=0.4)
    x = rng.standard_normal((S, d))
    y, _ = layer_forward(x, [0, S], W, H, 1e-5)
    Wl = {k: np.asarray(v).tolist() for k, v in W.items()}
    np.testing.assert_allclose(y, brute_layer(x.tolist(), Wl, H, 1e-5), rtol=1e-11, atol=1e-11)


def test_attention_rows_sum_to_one():
    rng = np.random.default_rng(1)
    e = rng.standard_normal((9, 13)) * 30
    p = softmax_rows(e)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert np.all(p >= 0)


def test_identical_values_give_value_back():
    rng = np.random.default_rng(2)
    S, d, H = 11, 16, 4
    q = rng.standard_normal((S, d))
    k = rng.standard_normal((S, d))
    v = np.tile(rng.standard_normal((1, d)), (S, 1))
    np.testing.assert_allclose(attention_seq(q, k, v, H), v, rtol=1e-13, atol=1e-13)


def test_identical_keys_give_mean_value():
    rng = np.random.default_rng(3)
    S, d, H = 6, 8, 2
    q = rng.standard_normal((S, d))
    k = np.tile(rng.standard_normal((1, d)), (S, 1))
    v = rng.standard_normal((S, d))
    out = attention_seq(q, k, v, H)
    np.testing.assert_allclose(out, np.tile(v.mean(axis=0), (S, 1)), rtol=1e-13, atol=1e-13)


def test_zero_output_projections_are_identity():
    rng = np.random.default_rng(4)
    d, I, S = 16, 24, 10
    W = rand_layer(rng, d, I)
    W["wo"] = np.zeros((d, d))
    W["wd"] = np.zeros((d, I))
    x = rng.standard_normal((S, d))
    y, _ = layer_forward(x, [0, S], W, 2, 1e-5)
    np.testing.assert_array_equal(y, x)


def test_truncated_varlen_equals_physically_cut():
    """Rows past seqused are masked keys: the kept rows equal the cut window."""
    rng = np.random.default_rng(5)
    d, I, H = 32, 48, 4
    W = rand_layer(rng, d, I)
    lens = [13, 20, 7]
    used = [9, 20, 3]
    xs = [rng.standard_normal((n, d)) for n in lens]
    for i in range(3):
        xs[i][used[i]:] = 0.0
    x = np.concatenate(xs)
    cu = np.concatenate([[0], np.cumsum(lens)])
    y, cnt = layer_forward(x, cu, W, H, 1e-5, seqused=used, act_eps=0.05)
    for i in range(3):
        yi, ci = layer_forward(xs[i][:used[i]], [0, used[i]], W, H, 1e-5, act_eps=0.05)
        np.testing.assert_array_equal(y[cu[i]:cu[i] + used[i]], yi)
        np.testing.assert_array_equal(cnt[cu[i]:cu[i] + used[i]], ci)
        # zero pad rows stay zero and count as fully sparse
        np.testing.assert_array_equal(y[cu[i] + used[i]:cu[i + 1]], 0.0)
        assert np.all(cnt[cu[i] + used[i]:cu[i + 1]] == I)


def test_packed_batch_equals_separate_sequences_and_is_permutation_equivariant():
    rng = np.random.default_rng(6)
    d, I, H = 16, 20, 2
    W = rand_layer(rng, d, I)
    lens = [5, 9, 4]
    xs = [rng.standard_normal((n, d)) for n in lens]
    cu = np.concatenate([[0], np.cumsum(lens)])
    y, _ = layer_forward(np.concatenate(xs), cu, W, H, 1e-5)
    for i in range(3):
        yi, _ = layer_forward(xs[i], [0, lens[i]], W, H, 1e-5)
        np.testing.assert_array_equal(y[cu[i]:cu[i + 1]], yi)
    perm = [2, 0, 1]
    lp = [lens[p] for p in perm]
    cup = np.concatenate([[0], np.cumsum(lp)])
    yp, _ = layer_forward(np.concatenate([xs[p] for p in perm]), cup, W, H, 1e-5)
    for j, p in enumerate(perm):
        np.testing.assert_array_equal(yp[cup[j]:cup[j + 1]], y[cu[p]:cu[p + 1]])


def test_row_sampled_forward_equals_full_forward():
    rng = np.random.default_rng(8)
    d, I, H, S = 16, 24, 4, 21
    W = rand_layer(rng, d, I)
    x = rng.standard_normal((S, d))
    y, _ = layer_forward(x, [0, S], W, H, 1e-5)
    rows = np.array([0, 5, 20, 11])
    r = layer_forward_rows(x, S, W, H, 1e-5, rows)
    np.testing.assert_allclose(r["y"], y[rows], rtol=1e-13, atol=1e-13)
