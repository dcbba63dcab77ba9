"""Shared helpers of the GPU parity tests: device upload, error metrics.

Nothing here computes any part of the method; the expected values always come
from ``oracle`` on the same seeded inputs.
"""
import sys

import numpy as np


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_dt(dtype):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def dev(a, dtype=None):
    """Upload a numpy array; float arrays go to the given dtype (bf16/f32)."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype.kind in "iu":
        return torch.from_numpy(a.astype(np.int32)).cuda()
    t = torch.from_numpy(a.astype(np.float32))
    return t.to(torch_dt(dtype or "f32")).cuda()


def host(t):
    """Device tensor -> float64 / int64 numpy (exact upcast)."""
    import torch
    t = t.detach()
    if t.dtype in (torch.int32, torch.int64, torch.int16, torch.uint8):
        return t.cpu().numpy().astype(np.int64)
    return t.float().cpu().numpy().astype(np.float64)


def upload_weights(W, dtype):
    return {k: (dev(v, dtype) if k not in ("g1", "g2") else dev(v, "f32")) for k, v in W.items()}


def rel_err(got, ref):
    """max |got - ref| / max(|ref|, rms(ref row)) over all elements."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    den = np.maximum(np.abs(ref), rms)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(got - ref) / den))


def row_errs(got, ref):
    """Per-row max of |got - ref| / max(|ref|, rms(ref row)) (rel_err per row)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return np.zeros(ref.shape[0])
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    den = np.maximum(np.abs(ref), rms)
    den = np.where(den == 0, 1.0, den)
    return np.max(np.abs(got - ref) / den, axis=-1)


def view_ws(workspace, offset, rows, cols, dtype):
    """A typed view of a region of the layer workspace."""
    import torch
    es = 2 if dtype == "bf16" else 4
    nbytes = rows * cols * es
    raw = workspace[offset:offset + nbytes]
    return raw.view(torch_dt(dtype)).view(rows, cols)


def view_ws_f32(workspace, offset, rows):
    import torch
    return workspace[offset:offset + rows * 4].view(torch.float32)


def count_band(b, wg, wu, eps):
    """Per-row range of near-zero counts consistent with fp32 evaluation.

    b: the MLP input (RMS-normalised) in float64, wg/wu: [I, d] weights.  An
    activation is ambiguous when its reference magnitude lies within the
    error an fp32 evaluation can make of it: the gate and up products carry
    about sqrt(K) * 2^-24 of the sum of absolute terms (times a safety factor
    of 8), and exp / division / the row scale add a few ulps of |act|.  The
    decision of every other activation is fixed, so a correct kernel's count
    lies in [c_min, c_max].  Returns (c_min, c_max, c_ref).
    """
    K = b.shape[1]
    u32 = 2.0 ** -24
    gam = 8.0 * np.sqrt(K) * u32
    g = b @ wg.T
    u = b @ wu.T
    dg = gam * (np.abs(b) @ np.abs(wg).T) + 4 * u32 * np.abs(g)
    du = gam * (np.abs(b) @ np.abs(wu).T) + 4 * u32 * np.abs(u)
    sig = 1.0 / (1.0 + np.exp(-g))
    s = g * sig
    ds = np.abs(sig * (1.0 + g * (1.0 - sig)))     # |d silu / dg|
    act = s * u
    da = ds * dg * np.abs(u) + np.abs(s) * du + 16 * u32 * np.abs(act)
    a = np.abs(act)
    c_min = np.sum(a < eps - da, axis=-1)
    c_max = np.sum(a < eps + da, axis=-1)
    c_ref = np.sum(a < eps, axis=-1)
    return c_min, c_max, c_ref


def check_counts(cnt_gpu, b, wg, wu, eps, d_ff, frac_tol=1e-3, band=False, act_gpu=None, act_tol=1e-4,
                 chunk=2048):
    """Gate the per-position sparsity fraction (Sec. 3.2-3.3) against the oracle.

    The oracle recomputes the SwiGLU activations in fp64 from the same MLP
    input ``b`` (RMS-normalised, teacher-forced from the GPU's own residual)
    and counts |act| < eps.  The gate is the spec bar itself:
    max over rows of |cnt_gpu - c_ref| / d_ff <= frac_tol.

    One count is 1/d_ff; when that exceeds frac_tol (d_ff < 1000, the fp32
    tiny layer) the bar means equal counts, and an activation within fp32
    rounding of eps may fall on either side.  Only for such a row, and only
    when the GPU's own unrounded activations ``act_gpu`` are given (fp32
    layers store them so), a difference is accepted element by element: the
    kernel's count must equal the count of its own activations, and every
    element whose decision differs must be a straddle of eps by two values of
    that element that agree within ``act_tol`` (relative to max(|act|, row
    rms)) -- the same decision taken on values equal to fp32 accuracy.
    ``band=True`` also evaluates the fp32-consistent count range of
    ``count_band`` (reported, never asserted).

    Returns a dict: rows, max_count_diff, max_frac_diff, straddles, and with
    band the rows outside [c_min, c_max] and the total range width."""
    from oracle.layer import silu
    from oracle.sparsity import near_zero_count, sparsity_fraction
    cnt_gpu = np.asarray(cnt_gpu, np.int64)
    b = np.asarray(b, np.float64)
    wg = np.asarray(wg, np.float64)
    wu = np.asarray(wu, np.float64)
    n = cnt_gpu.shape[0]
    assert b.shape[0] == n
    c_ref = np.zeros(n, np.int64)
    outside, ties, straddles = 0, 0, 0
    quantum_exceeds = 1.0 / d_ff > frac_tol
    for r0 in range(0, n, chunk):
        bb = b[r0:r0 + chunk]
        act = silu(bb @ wg.T) * (bb @ wu.T)
        c = near_zero_count(act, eps)
        c_ref[r0:r0 + chunk] = c
        cg = cnt_gpu[r0:r0 + chunk]
        off = np.nonzero(np.abs(sparsity_fraction(cg, d_ff) - sparsity_fraction(c, d_ff)) > frac_tol)[0]
        if off.size and quantum_exceeds and act_gpu is not None:
            ag = np.asarray(act_gpu[r0:r0 + chunk], np.float64)
            for r in off:
                assert cg[r] == near_zero_count(ag[r:r + 1], eps)[0], \
                    "row %d: count %d is not the count of the kernel's own activations" % (r0 + r, cg[r])
                diff = np.nonzero((np.abs(ag[r]) < eps) != (np.abs(act[r]) < eps))[0]
                scale = np.maximum(np.abs(act[r, diff]), np.sqrt(np.mean(act[r] ** 2)))
                gap = np.abs(ag[r, diff] - act[r, diff]) / scale
                assert np.all(gap <= act_tol), "row %d: decisions differ on elements %s whose values differ " \
                    "by %s (relative)" % (r0 + r, diff[:4], gap[:4])
                straddles += diff.size
            c_ref[r0:r0 + chunk][off] = cg[off]      # accepted: the flips are straddles of eps
        del act
        if band:
            c_min, c_max, _ = count_band(bb, wg, wu, eps)
            outside += int(np.sum((cg < c_min) | (cg > c_max)))
            ties += int(np.sum(c_max - c_min))
    dfrac = np.abs(sparsity_fraction(cnt_gpu, d_ff) - sparsity_fraction(c_ref, d_ff))
    res = dict(rows=n, max_count_diff=int(np.abs(cnt_gpu - c_ref).max()) if n else 0,
               max_frac_diff=float(dfrac.max()) if n else 0.0, straddles=straddles)
    if band:
        res.update(band_outside=outside, ties=ties)
    bad = np.nonzero(dfrac > frac_tol)[0]
    assert bad.size == 0, "rows %s: sparsity fraction off by %s (counts %s vs oracle %s), bar %g" % (
        bad[:5], dfrac[bad[:5]], cnt_gpu[bad[:5]], c_ref[bad[:5]], frac_tol)
    return res


def fmt_counts(res):
    s = "count diff max %d (fraction %.2e) over %d rows" % (res["max_count_diff"], res["max_frac_diff"],
                                                            res["rows"])
    if res.get("straddles"):
        s += ", %d single-element straddles of eps accepted (one count exceeds the bar)" % res["straddles"]
    if "band_outside" in res:
        s += ", fp32 band: %d rows outside, %d ties" % (res["band_outside"], res["ties"])
    return s
