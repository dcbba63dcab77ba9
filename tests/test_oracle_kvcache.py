"""Pins for the oracle's cached-prefix truncated step (CPU only).

The cached step must be the full layer restricted to the window rows when the
cache holds the prefix keys/values of a full step over the same inputs.  It
is pinned against:
  * the oracle's full layer on [prefix; window] (the definition it must
    reproduce), including padding rows and a two-layer stack with a cache per
    layer;
  * torch's own CPU float64 routines: rms_norm, linear and
    scaled_dot_product_attention with queries of the window only and keys of
    [prefix; window], composed independently of the oracle;
  * special cases: an empty prefix reduces to the plain layer on the window;
    an empty window gives an empty output.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle.kvcache import layer_forward_cached, layer_forward_cached_rows, prefix_kv
from oracle.layer import layer_forward, layer_forward_rows
from test_oracle_layer import rand_layer

EPS = 1e-5


@pytest.mark.parametrize("P,Sw,used,d,H,I", [(5, 7, 7, 16, 2, 24), (19, 11, 6, 32, 4, 40),
                                            (1, 1, 1, 8, 1, 8), (0, 9, 9, 16, 2, 12)])
def test_cached_equals_full_on_window_rows(P, Sw, used, d, H, I):
    rng = np.random.default_rng(P * 31 + Sw)
    W = rand_layer(rng, d, I)
    x = rng.standard_normal((P + Sw, d))
    full = layer_forward_rows(x, P + used, W, H, EPS, np.arange(P + Sw))["y"]
    k_pre, v_pre = prefix_kv(x, W, EPS, P)
    y = layer_forward_cached_rows(x[P:], used, k_pre, v_pre, W, H, EPS)["y"]
    np.testing.assert_allclose(y, full[P:], rtol=0, atol=1e-12)


def test_empty_prefix_is_the_plain_layer():
    rng = np.random.default_rng(3)
    W = rand_layer(rng, 16, 20)
    x = rng.standard_normal((6, 16))
    k0, v0 = prefix_kv(x, W, EPS, 0)
    assert k0.shape == (0, 16) and v0.shape == (0, 16)
    y = layer_forward_cached_rows(x, 6, k0, v0, W, 2, EPS)["y"]
    ref, _ = layer_forward(x, [0, 6], W, 2, EPS)
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)


def test_empty_window():
    rng = np.random.default_rng(4)
    W = rand_layer(rng, 8, 8)
    x = rng.standard_normal((5, 8))
    k_pre, v_pre = prefix_kv(x, W, EPS, 5)
    y = layer_forward_cached(np.zeros((0, 8)), [0, 0], [(k_pre, v_pre)], W, 1, EPS)
    assert y.shape == (0, 8)


def test_cached_attention_matches_torch_library():
    """Queries of the window rows only, keys/values of [prefix; window], from
    torch's scaled_dot_product_attention (float64, CPU)."""
    rng = np.random.default_rng(5)
    P, Sw, d, H, I = 13, 9, 32, 4, 24
    W = rand_layer(rng, d, I)
    x = rng.standard_normal((P + Sw, d))
    t = {k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in W.items()}
    xt = torch.from_numpy(x)
    dh = d // H
    a = F.rms_norm(xt, (d,), weight=t["g1"], eps=EPS)
    q = F.linear(a[P:], t["wq"]).view(Sw, H, dh).transpose(0, 1)
    k = F.linear(a, t["wk"]).view(P + Sw, H, dh).transpose(0, 1)
    v = F.linear(a, t["wv"]).view(P + Sw, H, dh).transpose(0, 1)
    o = F.scaled_dot_product_attention(q, k, v, is_causal=False).transpose(0, 1).reshape(Sw, d)
    h1 = xt[P:] + F.linear(o, t["wo"])
    b = F.rms_norm(h1, (d,), weight=t["g2"], eps=EPS)
    y_t = h1 + F.linear(F.silu(F.linear(b, t["wg"])) * F.linear(b, t["wu"]), t["wd"])
    k_pre, v_pre = prefix_kv(x, W, EPS, P)
    y = layer_forward_cached_rows(x[P:], Sw, k_pre, v_pre, W, H, EPS)["y"]
    np.testing.assert_allclose(y, y_t.numpy(), rtol=1e-12, atol=1e-12)


def test_packed_two_layer_stack():
    """Two layers, three sequences of different prefix/window lengths: caching
    each layer's prefix K/V from a full pass and running the cached pass on
    the window rows gives the full pass's window rows."""
    rng = np.random.default_rng(6)
    d, H, I = 16, 2, 20
    layers = [rand_layer(rng, d, I) for _ in range(2)]
    P = [4, 0, 7]
    Wn = [5, 3, 2]
    used = [5, 2, 2]
    x = [rng.standard_normal((P[b] + Wn[b], d)) for b in range(3)]
    # full pass, per layer, caching the prefix K/V of that layer's input
    caches = []
    cur = [xb.copy() for xb in x]
    for W in layers:
        caches.append([prefix_kv(cur[b], W, EPS, P[b]) for b in range(3)])
        cur = [layer_forward_rows(cur[b], P[b] + used[b], W, H, EPS, np.arange(P[b] + Wn[b]))["y"]
               for b in range(3)]
    # cached pass on the packed window rows
    cu = np.concatenate([[0], np.cumsum(Wn)])
    xw = np.concatenate([x[b][P[b]:] for b in range(3)])
    for l, W in enumerate(layers):
        xw = layer_forward_cached(xw, cu, caches[l], W, H, EPS, seqused=used)
    for b in range(3):
        np.testing.assert_allclose(xw[cu[b]:cu[b] + used[b]], cur[b][P[b]:P[b] + used[b]], rtol=0, atol=1e-11)


def test_selected_rows_match_all_rows():
    rng = np.random.default_rng(8)
    W = rand_layer(rng, 16, 20)
    x = rng.standard_normal((10, 16))
    k_pre, v_pre = prefix_kv(rng.standard_normal((4, 16)), W, EPS, 4)
    full = layer_forward_cached_rows(x, 7, k_pre, v_pre, W, 2, EPS)["y"]
    rows = np.array([0, 3, 6, 7, 9])
    part = layer_forward_cached_rows(x, 7, k_pre, v_pre, W, 2, EPS, rows=rows)["y"]
    np.testing.assert_allclose(part, full[rows], rtol=0, atol=1e-13)
