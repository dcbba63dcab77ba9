"""Rotary position embedding of queries and keys (oracle, fp64).

TEST INFRASTRUCTURE ONLY (part of the oracle package).

The paper says nothing about positional encoding (its layer equations in
Sec. 3.1 and Sec. 3.6 have none); the diffusion LLM backbones it runs on use
rotary embeddings.  Reading: rotary embedding as defined for RoFormer (Su et
al., 2021) in the "rotate half" pairing -- within each head of width dh,
feature j is paired with feature j + dh/2 (j < dh/2), and the pair is rotated
by the angle pos * theta^(-2 j / dh), where pos is the row's position in its
sequence (0 for the first visual token).  Queries and keys are rotated after
their projections; values are not.  theta is a parameter.
"""
import numpy as np


def rope_angles(positions, head_dim, theta):
    """[n, head_dim/2] angles pos * theta^(-2 j / head_dim)."""
    pos = np.asarray(positions, np.float64).reshape(-1, 1)
    j = np.arange(head_dim // 2, dtype=np.float64).reshape(1, -1)
    return pos * np.power(float(theta), -2.0 * j / head_dim)


def apply_rope(x, positions, n_heads, theta):
    """Rotate every head of x [n, d] by its row's position.

    For head h, feature pairs (j, j + dh/2) of columns h*dh + ... become
    (x1 cos a - x2 sin a, x2 cos a + x1 sin a) with a = rope_angles()[j]."""
    x = np.asarray(x, np.float64)
    n, d = x.shape
    dh = d // n_heads
    half = dh // 2
    a = rope_angles(positions, dh, theta)
    c, s = np.cos(a), np.sin(a)
    out = np.empty_like(x)
    for h in range(n_heads):
        x1 = x[:, h * dh:h * dh + half]
        x2 = x[:, h * dh + half:(h + 1) * dh]
        out[:, h * dh:h * dh + half] = x1 * c - x2 * s
        out[:, h * dh + half:(h + 1) * dh] = x2 * c + x1 * s
    return out
