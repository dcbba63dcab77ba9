"""Truncated steps with the visual/prompt prefix's keys and values cached
(oracle, fp64).

The paper reports Seer combined with a KV cache of the prefix (Appendix D,
compatibility with KV caching, and its table): the prefix keys and values of
every layer are reused across denoising steps, so a step only runs the rows of
the (truncated) generation window.  Each window row still attends to every
key of its sequence: the cached prefix keys, then the window's own keys.

Reading (the appendix gives no equations): the cache holds, per layer, the
keys and values that a full step computes for the prefix rows (`prefix_kv`).
A cached step on the window rows computes the same layer as the full step
restricted to those rows (`layer_forward_cached_rows`); when the cache comes
from a full step over the same inputs, the two agree exactly (pinned by the
CPU tests).  Window rows at index >= used are padding: not keys, zero
attention output, as in `layer.layer_forward_rows`.
"""
import numpy as np

from .layer import attention_seq, rms_norm, silu
from .rope import apply_rope


def _w(W, name):
    return np.asarray(W[name], np.float64)


def prefix_kv(x_seq, W, rms_eps, n_prefix, n_heads=None, rope_theta=None):
    """Keys and values [n_prefix, d] a layer computes for the first n_prefix
    rows of a sequence (the attention sub-block's K and V projections; keys
    rotated by positions 0..n_prefix-1 when rope_theta is set)."""
    a = rms_norm(np.asarray(x_seq, np.float64)[:n_prefix], _w(W, "g1"), rms_eps)
    k = a @ _w(W, "wk").T
    if rope_theta:
        k = apply_rope(k, np.arange(n_prefix), n_heads, rope_theta)
    return k, a @ _w(W, "wv").T


def layer_forward_cached_rows(x_win, used, k_pre, v_pre, W, n_heads, rms_eps, want_act=False,
                              rows=None, rope_theta=None):
    """The layer on the window rows of one sequence with cached prefix keys.

    x_win: [Sw, d] window rows; rows [0, used) are real.  k_pre, v_pre:
    [P, d] cached keys/values of the prefix.  Every real row attends to the
    P prefix keys followed by the `used` window keys.  ``rows``: the window
    rows whose outputs are wanted (default all).  With rope_theta, window row
    i sits at position P + i (the cached keys are already rotated).  Returns
    dict y [len(rows), d] (and act, h1 when want_act)."""
    x = np.asarray(x_win, np.float64)
    rows = np.arange(x.shape[0]) if rows is None else np.asarray(rows, np.int64)
    g1, g2 = _w(W, "g1"), _w(W, "g2")
    a_keys = rms_norm(x[:used], g1, rms_eps)
    P = np.asarray(k_pre).shape[0]
    k_own = a_keys @ _w(W, "wk").T
    xr = x[rows]
    q = rms_norm(xr, g1, rms_eps) @ _w(W, "wq").T
    if rope_theta:
        k_own = apply_rope(k_own, P + np.arange(used), n_heads, rope_theta)
        q = apply_rope(q, P + rows, n_heads, rope_theta)
    k = np.concatenate([np.asarray(k_pre, np.float64), k_own], axis=0)
    v = np.concatenate([np.asarray(v_pre, np.float64), a_keys @ _w(W, "wv").T], axis=0)
    o = np.zeros_like(xr)
    real = rows < used
    if np.any(real) and k.shape[0] > 0:
        o[real] = attention_seq(q[real], k, v, n_heads)
    h1 = xr + o @ _w(W, "wo").T
    b = rms_norm(h1, g2, rms_eps)
    act = silu(b @ _w(W, "wg").T) * (b @ _w(W, "wu").T)
    y = h1 + act @ _w(W, "wd").T
    out = {"y": y}
    if want_act:
        out["act"] = act
        out["h1"] = h1
    return out


def layer_forward_cached(x_w, cu_w, kv_pre, W, n_heads, rms_eps, seqused=None, rope_theta=None):
    """Packed version: sequence b's window rows are x_w[cu_w[b]:cu_w[b+1]],
    its cache kv_pre[b] = (k [P_b, d], v [P_b, d]).  Returns y [T_w, d]."""
    x = np.asarray(x_w, np.float64)
    cu = np.asarray(cu_w, np.int64)
    y = np.array(x, copy=True)
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        if s1 == s0:
            continue
        used = s1 - s0 if seqused is None else int(seqused[b])
        k_pre, v_pre = kv_pre[b]
        y[s0:s1] = layer_forward_cached_rows(x[s0:s1], used, k_pre, v_pre, W, n_heads, rms_eps,
                                             rope_theta=rope_theta)["y"]
    return y
