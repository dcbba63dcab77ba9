"""Step-0 detection, one-shot truncation and truncated steps (oracle).

Order of the method (Sec. 3.2-3.5 and the pipeline figure): at step 0 the
layers up to the detection layer run on the full window; the MLP sparsity of
the detection layer gives one count per window position; the SNR criterion
gives each sequence's boundary; the batch is routed and compacted; the suffix
is then absent from every later layer of step 0 and from every later denoising
step.

Reading for the later steps: no sampler or LM head is involved, so each
truncated step re-feeds the truncated step-input embeddings through all
layers (the compute of a denoising step, Sec. 3.1).
"""
from dataclasses import dataclass
from fractions import Fraction
from typing import List, Optional

import numpy as np

from .layer import layer_forward
from .detect import detect_batch
from .route import route_batch, repack_rows, POLICY_HYBRID, RouteResult


@dataclass
class PipelineResult:
    counts: np.ndarray          # [T_full] near-zero counts at the detection layer
    boundary: np.ndarray        # [B]
    keep_len: np.ndarray        # [B]
    route: RouteResult
    cu_trunc: np.ndarray        # [B+1]
    seqused: np.ndarray         # [B]
    capacity: int
    x_trunc: np.ndarray         # compacted step-input embeddings [capacity, d]
    y_step0: np.ndarray         # step-0 output after the last layer, compacted
    y_step: Optional[np.ndarray]  # one truncated denoising step's output


def run_pipeline(layers: List[dict], x, cu_seqlens, win_off, win_len, n_heads, d_ff,
                 rms_eps, act_eps, l_det, policy=POLICY_HYBRID, tau_pad=Fraction(1, 5),
                 granule=1, tau=Fraction(3, 100), gamma=Fraction(3, 5), lookahead=3,
                 run_trunc_step=True, dtype=np.float64):
    x = np.asarray(x, dtype)
    h = x
    counts = None
    for l in range(l_det + 1):
        h, c = layer_forward(h, cu_seqlens, layers[l], n_heads, rms_eps,
                             act_eps=act_eps if l == l_det else None, dtype=dtype)
        if l == l_det:
            counts = c
    boundary, keep = detect_batch(counts, cu_seqlens, win_off, win_len, d_ff,
                                  tau, gamma, lookahead)
    route = route_batch(keep, win_len, policy, tau_pad)
    h_t, cu_t, used, cap = repack_rows(h, cu_seqlens, win_off, keep, route.alloc, granule)
    x_t, _, _, _ = repack_rows(x, cu_seqlens, win_off, keep, route.alloc, granule)
    for l in range(l_det + 1, len(layers)):
        h_t, _ = layer_forward(h_t, cu_t, layers[l], n_heads, rms_eps, seqused=used, dtype=dtype)
    y_step = None
    if run_trunc_step:
        y_step = x_t
        for l in range(len(layers)):
            y_step, _ = layer_forward(y_step, cu_t, layers[l], n_heads, rms_eps, seqused=used, dtype=dtype)
    return PipelineResult(counts=counts, boundary=boundary, keep_len=keep, route=route,
                          cu_trunc=cu_t, seqused=used, capacity=cap, x_trunc=x_t,
                          y_step0=h_t, y_step=y_step)
