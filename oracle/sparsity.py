"""Per-position MLP activation sparsity (oracle).

The statistic the method reads at step 0 (Sec. 3.2 and 3.3): for each text
position, the fraction of MLP activations whose magnitude is below an absolute
near-zero threshold (the introduction states that an absolute threshold
separates the boundary best).  Readings: the activation is the SwiGLU product
silu(gate) * up, the tensor the down projection consumes; "near zero" is the
strict inequality |a| < eps.  The count is kept as an integer; the sparsity
fraction is count / I.
"""
import numpy as np


def near_zero_count(act, eps):
    """Number of entries per row with |act| < eps (strict)."""
    a = np.asarray(act, np.float64)
    return np.sum(np.abs(a) < eps, axis=-1).astype(np.int64)


def sparsity_fraction(counts, d_ff):
    return np.asarray(counts, np.float64) / float(d_ff)
