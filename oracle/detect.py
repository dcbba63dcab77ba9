"""SNR-aware semantic boundary detection (oracle), Sec. 3.3.

Given the sparsity array S = [s_1 .. s_N] of the generation window, position i
is a boundary when the look-ahead window W_i = {s_i, .., s_{i+w-1}} (w = 3 by
default) satisfies
    jump  = min(W_i) - s_{i-1}  >= tau_jump          (significant signal)
    noise = max(W_i) - min(W_i) <= gamma * jump      (stable plateau)
and the sequence is cut to L* = i* + 1 positions.

Readings: positions are 0-based, so i runs over [1, N-w] and i* is the first
plateau position (the first EOS); keeping i*+1 positions keeps the content and
that first EOS.  The first (leftmost) qualifying i is taken.  When no i
qualifies the window is kept whole (i* = N, L* = N).  s_i = count_i / I is
evaluated in exact rational arithmetic, so the decision carries no rounding.
"""
from fractions import Fraction

import numpy as np


def detect_boundary(counts, d_ff, tau=Fraction(3, 100), gamma=Fraction(3, 5), lookahead=3):
    """Return (i_star, keep_len) for one window's per-position counts."""
    tau = Fraction(tau)
    gamma = Fraction(gamma)
    n = len(counts)
    s = [Fraction(int(c), int(d_ff)) for c in counts]
    for i in range(1, n - lookahead + 1):
        win = s[i:i + lookahead]
        jump = min(win) - s[i - 1]
        noise = max(win) - min(win)
        if jump >= tau and noise <= gamma * jump:
            return i, i + 1
    return n, n


def detect_batch(counts, cu_seqlens, win_off, win_len, d_ff, tau=Fraction(3, 100),
                 gamma=Fraction(3, 5), lookahead=3):
    """Per-sequence (boundary, keep_len) from packed per-row counts."""
    cu = np.asarray(cu_seqlens, np.int64)
    B = len(cu) - 1
    boundary = np.zeros(B, np.int64)
    keep = np.zeros(B, np.int64)
    for b in range(B):
        s0 = int(cu[b]) + int(win_off[b])
        win = counts[s0:s0 + int(win_len[b])]
        boundary[b], keep[b] = detect_boundary(win, d_ff, tau, gamma, lookahead)
    return boundary, keep
