"""One bidirectional transformer layer in fp64 (oracle).

The layer is what each denoising step runs over the whole sequence
(Sec. 3.1, the denoising-step equation and the complexity equation): full,
non-causal self-attention over [visual prefix; prompt; window] followed by a
SwiGLU MLP.  Attention follows the Sec. 3.6 equations: logits q.k/sqrt(d_h),
a softmax over every key of the same sequence, a weighted sum of values.

Readings where the paper is silent: pre-norm RMSNorm (gain g, eps 1e-5) before
attention and before the MLP, no biases, scale 1/sqrt(head_dim), and by default
no positional encoding; with ``rope_theta`` set, queries and keys are rotated
by their position in the sequence (``rope.apply_rope``; position = row index
plus ``pos_offset``).  Rows of a sequence at index >= ``used`` are inert padding:
they are not attention keys and receive no attention output; the rest of the
layer applies to them row by row.

Everything is computed in float64 from the given (bf16- or fp32-valued) inputs,
directly from the definitions: softmax is evaluated on the full logit row,
not online.  (``dtype`` exists only so that the benchmark can also time the
same definitions in float32; every check uses the float64 default.)
"""
import numpy as np

from .rope import apply_rope


def silu(z):
    return z / (1.0 + np.exp(-z))


def rms_norm(x, gain, eps, dtype=np.float64):
    x = np.asarray(x, dtype)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype)


def softmax_rows(e):
    m = np.max(e, axis=-1, keepdims=True)
    p = np.exp(e - m)
    return p / np.sum(p, axis=-1, keepdims=True)


def attention_seq(q, k, v, n_heads, q_rows=None, dtype=np.float64):
    """Bidirectional multi-head attention of one sequence.

    q: [Sq, d] (the query rows wanted), k, v: [Sk, d] (every key of the
    sequence).  Returns [Sq, d] = concat_h softmax(q_h k_h^T / sqrt(d_h)) v_h.
    """
    q = np.asarray(q, dtype)
    k = np.asarray(k, dtype)
    v = np.asarray(v, dtype)
    d = q.shape[1]
    dh = d // n_heads
    out = np.empty((q.shape[0], d), dtype)
    for h in range(n_heads):
        sl = slice(h * dh, (h + 1) * dh)
        e = q[:, sl] @ k[:, sl].T / np.sqrt(dh)
        out[:, sl] = softmax_rows(e) @ v[:, sl]
    return out


def _w(W, name, dtype=np.float64):
    return np.asarray(W[name], dtype)


def layer_forward_rows(x_seq, used, W, n_heads, rms_eps, rows, want_act=False, rope_theta=None,
                       pos_offset=0, dtype=np.float64):
    """Layer outputs for selected rows of one sequence.

    x_seq: [S, d] rows of one sequence; ``used``: rows [0, used) are real,
    the rest padding.  ``rows``: indices whose outputs are wanted.  Keys and
    values come from all ``used`` rows.  Returns dict with y [len(rows), d],
    and when want_act the SwiGLU activation act [len(rows), I] and the
    intermediates h1.
    """
    x_seq = np.asarray(x_seq, dtype)
    rows = np.asarray(rows, np.int64)
    g1, g2 = _w(W, "g1", dtype), _w(W, "g2", dtype)
    # attention sub-block
    a_keys = rms_norm(x_seq[:used], g1, rms_eps, dtype)
    k = a_keys @ _w(W, "wk", dtype).T
    v = a_keys @ _w(W, "wv", dtype).T
    xr = x_seq[rows]
    ar = rms_norm(xr, g1, rms_eps, dtype)
    q = ar @ _w(W, "wq", dtype).T
    if rope_theta:
        k = apply_rope(k, pos_offset + np.arange(used), n_heads, rope_theta)
        q = apply_rope(q, pos_offset + rows, n_heads, rope_theta)
    o = np.zeros_like(xr)
    real = rows < used
    if used > 0 and np.any(real):
        o[real] = attention_seq(q[real], k, v, n_heads, dtype=dtype)
    h1 = xr + o @ _w(W, "wo", dtype).T
    # SwiGLU MLP sub-block
    b = rms_norm(h1, g2, rms_eps, dtype)
    gate = b @ _w(W, "wg", dtype).T
    up = b @ _w(W, "wu", dtype).T
    act = silu(gate) * up
    y = h1 + act @ _w(W, "wd", dtype).T
    out = {"y": y}
    if want_act:
        out["act"] = act
        out["h1"] = h1
    return out


def layer_forward(x, cu_seqlens, W, n_heads, rms_eps, seqused=None, act_eps=None, rope_theta=None,
                  dtype=np.float64):
    """One layer over packed sequences (rows of sequence b are cu[b]..cu[b+1]).

    Returns (y [T, d] float64, counts [T] int64 or None).  ``counts`` is the
    per-row number of SwiGLU activations with |act| < act_eps, for every row.
    """
    from .sparsity import near_zero_count
    x = np.asarray(x, dtype)
    cu = np.asarray(cu_seqlens, np.int64)
    B = len(cu) - 1
    y = np.array(x, copy=True)
    counts = None if act_eps is None else np.zeros(x.shape[0], np.int64)
    for b in range(B):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        S = s1 - s0
        used = S if seqused is None else int(seqused[b])
        if S == 0:
            continue
        r = layer_forward_rows(x[s0:s1], used, W, n_heads, rms_eps, np.arange(S),
                               want_act=act_eps is not None, rope_theta=rope_theta, dtype=dtype)
        y[s0:s1] = r["y"]
        if act_eps is not None:
            counts[s0:s1] = near_zero_count(r["act"], act_eps)
    return y, counts
