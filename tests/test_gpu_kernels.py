"""GPU parity of each C-ABI entry point against the oracle, at small sizes.

Sizes span several GEMM tiles (256 rows) and attention tiles (128 queries,
64 keys) with ragged tails.  Tolerances: boundary indices, offsets, routes
and copied rows bit-exact; sparsity fractions within 1e-3 (teacher-forced at
the MLP input); hidden states within 2e-2 max relative error for bf16
(error / max(|ref|, rms of the reference row)) and 1e-4 for fp32.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from conftest import GOLDEN
from gpu_util import check_counts, dev, fmt_counts, host, log, rel_err, upload_weights, view_ws, view_ws_f32
from oracle.detect import detect_batch, detect_boundary
from oracle.layer import attention_seq, layer_forward, rms_norm, silu
from oracle.route import repack_rows, route_batch
from oracle.sparsity import near_zero_count

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4
FRAC_TOL = 1e-3


@pytest.fixture(scope="module")
def S():
    import torch
    from paper_2607_14557_amd import seer
    seer.load_library()
    torch.cuda.init()
    return seer


def _i32(n):
    import torch
    return torch.empty(n, dtype=torch.int32, device="cuda")


# ---------------------------------------------------------------------------
# SNR boundary scan

def test_detect_golden_cases(S):
    import torch
    with open(os.path.join(GOLDEN, "detector_cases.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        log("detect golden: %s" % c["name"])
        n = len(c["counts"])
        cnt = dev(np.array(c["counts"], np.int32))
        bnd, keep = _i32(1), _i32(1)
        prm = S.seer_snr_params(c["tau"][0], c["tau"][1], c["gamma"][0], c["gamma"][1], c["lookahead"])
        S.seer_step0_detect(cnt, dev(np.array([0, n])), dev(np.array([0])), dev(np.array([n])), 1,
                            c["d_ff"], prm, bnd, keep)
        torch.cuda.synchronize()
        assert (int(bnd[0]), int(keep[0])) == (c["boundary"], c["keep_len"]), c["name"]


@pytest.mark.parametrize("lookahead,tau,gamma", [(3, (3, 100), (3, 5)), (2, (1, 50), (1, 2)),
                                                 (5, (7, 100), (4, 5)), (1, (3, 100), (3, 5))])
def test_detect_random_batch_vs_oracle(S, lookahead, tau, gamma):
    import torch
    rng = np.random.default_rng(100 + lookahead)
    B, I = 64, 997
    pre = rng.integers(0, 40, size=B)
    win = rng.integers(1, 300, size=B)
    win[:3] = [1, 2, lookahead]                    # windows too short for any candidate
    lens = pre + win + rng.integers(0, 5, size=B)  # a little slack after the window
    cu = np.concatenate([[0], np.cumsum(lens)])
    counts = rng.integers(0, 120, size=int(cu[-1]))
    for b in range(B):                             # plant steps in most windows
        if b % 4:
            j = int(cu[b] + pre[b] + rng.integers(0, max(1, win[b])))
            counts[j:cu[b + 1]] += int(rng.integers(0, 80))
    counts = np.minimum(counts, I)
    bnd, keep = _i32(B), _i32(B)
    log("detect random lookahead=%d" % lookahead)
    S.seer_step0_detect(dev(counts.astype(np.int32)), dev(cu), dev(pre), dev(win), B, I,
                        S.seer_snr_params(tau[0], tau[1], gamma[0], gamma[1], lookahead), bnd, keep)
    torch.cuda.synchronize()
    eb, ek = detect_batch(counts, cu, pre, win, I, Fraction(*tau), Fraction(*gamma), lookahead)
    np.testing.assert_array_equal(host(bnd), eb)
    np.testing.assert_array_equal(host(keep), ek)


# ---------------------------------------------------------------------------
# routing + compaction

def _repack_case(S, policy, granule, B=13, d=64, seed=0, capacity=None):
    import torch
    rng = np.random.default_rng(seed)
    win_off = rng.integers(5, 41, size=B)
    win_len = np.full(B, 200)
    keep = rng.integers(1, 201, size=B)
    keep[:3] = [2, 3, 4]
    keep[3:6] = [60, 61, 63]
    lens = win_off + win_len
    cu_src = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu_src[-1])
    src1 = rng.standard_normal((T, d)).astype(np.float32)
    src2 = rng.standard_normal((T, d)).astype(np.float32)
    full_cap = int(np.sum(win_off + win_len.max()))
    if capacity is None:
        capacity = ((full_cap + granule - 1) // granule) * granule + granule
    s1, s2 = dev(src1, "bf16"), dev(src2, "bf16")
    sentinel = -7.0
    d1 = torch.full((capacity, d), sentinel, dtype=torch.bfloat16, device="cuda")
    d2 = torch.full((capacity, d), sentinel, dtype=torch.bfloat16, device="cuda")
    cu_dst, used = _i32(B + 1), _i32(B)
    route = torch.empty(B, 3, dtype=torch.int32, device="cuda")
    ctrl = torch.zeros(16, dtype=torch.int32, device="cuda")
    ctrl_h = torch.zeros(16, dtype=torch.int32).pin_memory()
    desc = S.seer_repack_desc(policy, 1, 5, granule, d * 2, capacity, 0, 0)
    S.seer_batch_repack(desc, [s1, s2], [d1, d2], dev(cu_src), dev(win_off), dev(win_len),
                        dev(keep), B, cu_dst, used, route, ctrl, ctrl_h)
    torch.cuda.synchronize()
    return dict(win_off=win_off, win_len=win_len, keep=keep, cu_src=cu_src, s=[s1, s2], d=[d1, d2],
                cu_dst=cu_dst, used=used, route=route, ctrl=ctrl, ctrl_h=ctrl_h, capacity=capacity)


@pytest.mark.parametrize("policy", [0, 1, 2])
@pytest.mark.parametrize("granule", [1, 256])
def test_repack_vs_oracle(S, policy, granule):
    import torch
    log("repack policy=%d granule=%d" % (policy, granule))
    r = _repack_case(S, policy, granule, seed=policy * 10 + granule)
    rt = route_batch(r["keep"], r["win_len"], policy, Fraction(1, 5))
    route = host(r["route"])
    np.testing.assert_array_equal(route[:, 0], rt.path)
    np.testing.assert_array_equal(route[:, 1], rt.group)
    np.testing.assert_array_equal(route[:, 2], rt.alloc)
    for bi in range(2):
        src = host(r["s"][bi])
        exp, cu_e, used_e, cap = repack_rows(src, r["cu_src"], r["win_off"], r["keep"], rt.alloc, granule)
        np.testing.assert_array_equal(host(r["cu_dst"]), cu_e)
        np.testing.assert_array_equal(host(r["used"]), used_e)
        got = host(r["d"][bi])
        np.testing.assert_array_equal(got[:cap], exp)
        assert np.all(got[cap:] == -7.0), "rows past the routed capacity must be untouched"
    ctrl = host(r["ctrl"])
    assert list(ctrl[:9]) == [cu_e[-1], cap, int(np.sum(rt.path == 0)), int(np.sum(rt.path == 1)),
                              int(np.sum(rt.path == 2)), len(rt.groups), int(rt.alloc.max()), 0, 1]
    np.testing.assert_array_equal(host(r["ctrl_h"]), ctrl)


def test_repack_overflow_reports_status(S):
    log("repack overflow")
    r = _repack_case(S, 0, 1, seed=3, capacity=50)
    ctrl = host(r["ctrl"])
    assert ctrl[7] == S.SEER_EWORKSPACE and ctrl[8] == 1
    assert np.all(host(r["cu_dst"]) == 0)
    assert np.all(host(r["d"][0]) == -7.0), "nothing may be written on overflow"


# ---------------------------------------------------------------------------
# one layer, bf16 and fp32

def _rand_layer(rng, d, I, std):
    return {"wq": rng.standard_normal((d, d)) * std, "wk": rng.standard_normal((d, d)) * std,
            "wv": rng.standard_normal((d, d)) * std, "wo": rng.standard_normal((d, d)) * std,
            "wg": rng.standard_normal((I, d)) * std, "wu": rng.standard_normal((I, d)) * std,
            "wd": rng.standard_normal((d, I)) * std,
            "g1": np.ones(d), "g2": np.ones(d)}


def _round(W, dtype):
    from workloads.generate import round_to_dtype
    return {k: (round_to_dtype(v, dtype).astype(np.float64) if k not in ("g1", "g2") else v)
            for k, v in W.items()}


class _Layer:
    """One prepacked layer + workspace driven through the C ABI."""

    def __init__(self, S, d, H, dh, I, dtype, rows_ub, W):
        import torch
        from paper_2607_14557_amd.runner import dims_for
        self.S = S
        self.dims = dims_for(d, H, dh, I, dtype)
        self.dtype = dtype
        self.rows_ub = rows_ub
        self.packed = torch.empty(S.seer_prepacked_bytes(self.dims), dtype=torch.uint8, device="cuda")
        S.seer_prepack_weights(self.dims, upload_weights(W, dtype), self.packed)
        self.ws = torch.empty(S.seer_layer_workspace_bytes(self.dims, rows_ub), dtype=torch.uint8,
                              device="cuda")
        self.off = S.seer_layer_workspace_offsets(self.dims, rows_ub)

    def run(self, x, cu, batch, seqused=None, eps=None):
        import torch
        out = torch.zeros_like(x)
        cnt = _i32(self.rows_ub) if eps is not None else None
        self.S.seer_layer_forward_varlen(self.dims, self.packed, x, out, self.rows_ub, cu, seqused,
                                         batch, 0.0 if eps is None else eps, cnt, self.ws)
        torch.cuda.synchronize()
        return out, cnt

    def inter(self, name, rows, cols=None):
        idx = {"qkv": 0, "o": 1, "h1": 2, "act": 3, "inv1": 4, "inv2": 5, "h1f": 6}[name]
        if name.startswith("inv"):
            return view_ws_f32(self.ws, self.off[idx], rows)
        if name == "h1f":
            # h1 as the final residual add reads it: bf16 high part + bf16 low part
            if self.dtype == "f32":
                return view_ws(self.ws, self.off[idx], rows, cols, "f32")
            return (view_ws(self.ws, self.off[2], rows, cols, "bf16").float() +
                    view_ws(self.ws, self.off[idx], rows, cols, "bf16").float())
        t = view_ws(self.ws, self.off[idx], rows, cols, self.dtype)
        if name == "qkv" and self.dtype == "bf16":
            # bf16 layers store the v third in fp16 (the type of the P V product)
            import torch
            d = cols // 3
            t = torch.cat([t[:, :2 * d].float(), t[:, 2 * d:].contiguous().view(torch.float16).float()], dim=1)
        return t


# bf16_k640: d_ff = 640 gives the down projection K / 64 = 10 tiles, so the
# GEMM's four-stage ring ends on its two-tile tail
@pytest.mark.parametrize("case", ["bf16", "bf16_k640", "f32"])
def test_layer_vs_oracle_ragged(S, case):
    dtype = "f32" if case == "f32" else "bf16"
    d, H, dh, I = {"bf16": (512, 4, 128, 1024), "bf16_k640": (256, 2, 128, 640), "f32": (256, 4, 64, 688)}[case]
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    rng = np.random.default_rng(42)
    W = _round(_rand_layer(rng, d, I, 0.02), dtype)
    lens = [300, 77, 513, 1, 129]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    rows_ub = T + 5
    x = np.zeros((rows_ub, d))
    x[:T] = rng.standard_normal((T, d))
    xd = dev(x, dtype)
    x = host(xd)                                    # exact values the GPU sees
    eps = 0.01 * 0.0004 * d
    log("layer %s ragged lens=%s (d %d, d_ff %d)" % (dtype, lens, d, I))
    L = _Layer(S, d, H, dh, I, dtype, rows_ub, W)
    y, cnt = L.run(xd, dev(cu), len(lens), eps=eps)
    y = host(y)
    y_ref, cnt_ref = layer_forward(x[:T], cu, W, H, 1e-5, act_eps=eps)
    e = rel_err(y[:T], y_ref)
    log("  y rel err %.3e" % e)
    assert e <= tol
    assert np.all(y[T:] == 0.0), "rows past cu[B] must not be written"
    # teacher-forced stages
    qkv = host(L.inter("qkv", T, 3 * d))
    a = rms_norm(x[:T], W["g1"], 1e-5)
    qkv_ref = np.concatenate([a @ W["wq"].T, a @ W["wk"].T, a @ W["wv"].T], axis=1)
    assert rel_err(qkv, qkv_ref) <= tol
    o = host(L.inter("o", T, d))
    for b in range(len(lens)):
        s = slice(cu[b], cu[b + 1])
        o_ref = attention_seq(qkv[s, :d], qkv[s, d:2 * d], qkv[s, 2 * d:], H)
        eo = rel_err(o[s], o_ref)
        assert eo <= tol, "attention seq %d err %.3e" % (b, eo)
    h1 = host(L.inter("h1", T, d))
    assert rel_err(h1, x[:T] + o @ W["wo"].T) <= tol
    bnorm = rms_norm(h1, W["g2"], 1e-5)
    act_ref = silu(bnorm @ W["wg"].T) * (bnorm @ W["wu"].T)
    act = host(L.inter("act", T, I))
    assert rel_err(act, act_ref) <= tol
    cr = check_counts(host(cnt)[:T], bnorm, W["wg"], W["wu"], eps, I, FRAC_TOL, band=True,
                      act_gpu=act if dtype == "f32" else None)
    log("  teacher-forced %s; untethered count diff max %d of %d" %
        (fmt_counts(cr), np.abs(host(cnt)[:T] - cnt_ref).max(), I))
    if dtype == "f32":
        # the fp32 activations are stored unrounded: the kernel's count must be
        # exactly the count of its own activations
        np.testing.assert_array_equal(host(cnt)[:T], near_zero_count(act, eps))
    # the final residual add uses h1 to ~2^-17 (bf16 high + low part)
    h1f = host(L.inter("h1f", T, d))
    assert rel_err(h1f, x[:T] + o @ W["wo"].T) <= (1e-5 if dtype == "bf16" else tol)
    e_dn = rel_err(y[:T], h1f + act @ W["wd"].T)
    log("  stage errors (teacher-forced): qkv %.2e attn %.2e act %.2e down %.2e" %
        (rel_err(qkv, qkv_ref), max(rel_err(o[cu[b]:cu[b + 1]], attention_seq(
            qkv[cu[b]:cu[b + 1], :d], qkv[cu[b]:cu[b + 1], d:2 * d], qkv[cu[b]:cu[b + 1], 2 * d:], H))
            for b in range(len(lens))), rel_err(act, act_ref), e_dn))
    assert e_dn <= tol


def test_attention_peaked_softmax(S):
    """Scores spread over hundreds of log2 units (q and k projections 12x the
    usual scale): for most queries a later key tile holds a score far above
    the first tile's maximum, so the softmax's reference maximum has to move
    mid-sequence, past the range fp16 probabilities can hold.  The attention
    stage, teacher-forced from the kernel's own q, k and v, must match the
    oracle's softmax within the bf16 bar."""
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(4242)
    W = _rand_layer(rng, d, I, 0.02)
    W["wq"] = W["wq"] * 12.0
    W["wk"] = W["wk"] * 12.0
    W = _round(W, "bf16")
    lens = [700, 64, 1, 333, 129]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    x = rng.standard_normal((T, d))
    xd = dev(x, "bf16")
    log("peaked softmax: lens=%s, q/k projections x12" % lens)
    L = _Layer(S, d, H, dh, I, "bf16", T, W)
    L.run(xd, dev(cu), len(lens))
    qkv = host(L.inter("qkv", T, 3 * d))
    o = host(L.inter("o", T, d))
    c = np.log2(np.e) / np.sqrt(dh)
    jumps = []
    for b in range(len(lens)):
        s = slice(cu[b], cu[b + 1])
        q, k = qkv[s, :d], qkv[s, d:2 * d]
        for h in range(H):
            hs = slice(h * dh, (h + 1) * dh)
            e = (q[:, hs] @ k[:, hs].T) * c               # log2 units
            jumps.append(e.max(axis=1) - e[:, :64].max(axis=1))
        o_ref = attention_seq(q, k, qkv[s, 2 * d:], H)
        eo = rel_err(o[s], o_ref)
        assert eo <= BF16_TOL, "attention seq %d err %.3e" % (b, eo)
    jumps = np.concatenate(jumps)
    log("  max over later key tiles above the first tile's: >8 for %.0f%%, >16 for %.0f%% of query heads "
        "(largest %.0f log2 units)" % (100 * np.mean(jumps > 8), 100 * np.mean(jumps > 16), jumps.max()))
    assert np.mean(jumps > 16) > 0.2, "the case does not move the reference maximum far enough"


def test_layer_static_padding_equals_cut_layout_bitwise(S):
    """Pad rows masked by seqused leave the kept rows bit-identical."""
    import torch
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(7)
    W = _round(_rand_layer(rng, d, I, 0.02), "bf16")
    used = [200, 65, 130]
    alloc = [256, 128, 130]
    cu_pad = np.concatenate([[0], np.cumsum(alloc)])
    cu_cut = np.concatenate([[0], np.cumsum(used)])
    xs = [rng.standard_normal((u, d)) for u in used]
    x_pad = np.zeros((int(cu_pad[-1]), d))
    for b in range(3):
        x_pad[cu_pad[b]:cu_pad[b] + used[b]] = xs[b]
    x_cut = np.concatenate(xs)
    rows_ub = int(cu_pad[-1])
    L = _Layer(S, d, H, dh, I, "bf16", rows_ub, W)
    log("layer static padding vs cut")
    y_pad, c_pad = L.run(dev(x_pad, "bf16"), dev(cu_pad), 3, seqused=dev(np.array(used)), eps=0.002)
    y_cut, c_cut = L.run(dev(np.concatenate([x_cut, np.zeros((rows_ub - len(x_cut), d))]), "bf16"),
                         dev(cu_cut), 3, eps=0.002)
    yp, yc = host(y_pad), host(y_cut)
    cp, cc = host(c_pad), host(c_cut)
    for b in range(3):
        np.testing.assert_array_equal(yp[cu_pad[b]:cu_pad[b] + used[b]], yc[cu_cut[b]:cu_cut[b + 1]])
        np.testing.assert_array_equal(cp[cu_pad[b]:cu_pad[b] + used[b]], cc[cu_cut[b]:cu_cut[b + 1]])
        assert np.all(yp[cu_pad[b] + used[b]:cu_pad[b + 1]] == 0.0)
        assert np.all(cp[cu_pad[b] + used[b]:cu_pad[b + 1]] == I)


def test_layer_deterministic(S):
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(9)
    W = _round(_rand_layer(rng, d, I, 0.02), "bf16")
    lens = [333, 190]
    cu = np.concatenate([[0], np.cumsum(lens)])
    x = dev(rng.standard_normal((int(cu[-1]), d)), "bf16")
    L = _Layer(S, d, H, dh, I, "bf16", int(cu[-1]), W)
    log("layer determinism")
    y1, c1 = L.run(x, dev(cu), 2, eps=0.002)
    y2, c2 = L.run(x, dev(cu), 2, eps=0.002)
    np.testing.assert_array_equal(host(y1), host(y2))
    np.testing.assert_array_equal(host(c1), host(c2))


def test_timed_layer_with_one_kernel_timed(S):
    """The timed entry point with only the two events around the gate/up GEMM
    set (the others NULL, skipped): the output is bit-identical to the untimed
    call, and the two recorded events bound a positive kernel time."""
    import ctypes
    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")
    hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(19)
    W = _round(_rand_layer(rng, d, I, 0.02), "bf16")
    lens = [300, 1, 517]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    x = dev(rng.standard_normal((T, d)), "bf16")
    L = _Layer(S, d, H, dh, I, "bf16", T, W)
    log("timed layer, gate/up events only")
    y_ref, _ = L.run(x, dev(cu), len(lens))
    ev = []
    for _ in range(2):
        e = ctypes.c_void_p()
        assert hip.hipEventCreate(ctypes.byref(e)) == 0
        ev.append(e.value)
    y = torch.zeros_like(x)
    S.seer_layer_forward_varlen_timed(L.dims, L.packed, x, y, T, dev(cu), None, len(lens), 0.0, None, L.ws,
                                      [None] * 5 + ev + [None])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(y), host(y_ref))
    ms = ctypes.c_float()
    assert hip.hipEventElapsedTime(ctypes.byref(ms), ev[0], ev[1]) == 0
    log("  gate/up GEMM %.4f ms" % ms.value)
    assert ms.value > 0.0
    for e in ev:
        hip.hipEventDestroy(e)


def test_layer_batch_permutation_bitwise(S):
    """Reordering the sequences of a packed batch reorders the results and
    changes nothing else, bit for bit: every row's projections, its
    sequence's attention and its count are independent of where the sequence
    sits (rows move between and inside GEMM tiles and query tiles)."""
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(21)
    W = _round(_rand_layer(rng, d, I, 0.02), "bf16")
    lens = [333, 1, 190, 0, 257, 64]
    perm = [4, 2, 0, 5, 1, 3]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    xs = [rng.standard_normal((n, d)) for n in lens]
    lens_p = [lens[b] for b in perm]
    cu_p = np.concatenate([[0], np.cumsum(lens_p)])
    L = _Layer(S, d, H, dh, I, "bf16", T, W)
    log("layer batch permutation %s" % perm)
    y, c = L.run(dev(np.concatenate(xs), "bf16"), dev(cu), len(lens), eps=0.002)
    yp, cp = L.run(dev(np.concatenate([xs[b] for b in perm]), "bf16"), dev(cu_p), len(lens), eps=0.002)
    y, c, yp, cp = host(y), host(c), host(yp), host(cp)
    for j, b in enumerate(perm):
        np.testing.assert_array_equal(yp[cu_p[j]:cu_p[j + 1]], y[cu[b]:cu[b + 1]])
        np.testing.assert_array_equal(cp[cu_p[j]:cu_p[j + 1]], c[cu[b]:cu[b + 1]])


# ---------------------------------------------------------------------------
# degenerate inputs: empty sequences and windows, the largest repack batch

def test_layer_with_empty_sequences(S):
    """Zero-length sequences between real ones, and a batch with no rows at all."""
    import torch
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(7)
    W = _round(_rand_layer(rng, d, I, 0.02), "bf16")
    lens = [0, 130, 0, 1, 257, 0]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    rows_ub = T + 3
    xd = dev(np.concatenate([rng.standard_normal((T, d)), np.zeros((3, d))]), "bf16")
    x = host(xd)
    eps = 0.01 * 0.0004 * d
    log("layer with empty sequences lens=%s" % lens)
    L = _Layer(S, d, H, dh, I, "bf16", rows_ub, W)
    y, cnt = L.run(xd, dev(cu), len(lens), eps=eps)
    y = host(y)
    y_ref, _ = layer_forward(x[:T], cu, W, H, 1e-5, act_eps=eps)
    assert rel_err(y[:T], y_ref) <= BF16_TOL
    assert np.all(y[T:] == 0.0)
    bnorm = rms_norm(host(L.inter("h1", T, d)), W["g2"], 1e-5)
    check_counts(host(cnt)[:T], bnorm, W["wg"], W["wu"], eps, I, FRAC_TOL)
    # no rows: nothing is written, the counts stay zero
    L0 = _Layer(S, d, H, dh, I, "bf16", 8, W)
    x0 = torch.zeros(8, d, dtype=torch.bfloat16, device="cuda")
    y0, c0 = L0.run(x0, dev(np.array([0, 0, 0])), 2, eps=eps)
    assert torch.count_nonzero(y0).item() == 0
    assert torch.count_nonzero(c0).item() == 0


@pytest.mark.parametrize("policy", [0, 1])
def test_detect_and_repack_largest_batch(S, policy):
    """1024 sequences (the largest batch one repack launch plans), with empty
    windows, empty prefixes and windows too short for any candidate; hybrid
    routing (all varlen here) and naive padding (all static)."""
    import torch
    rng = np.random.default_rng(2024)
    B, I, d = 1024, 257, 64
    pre = rng.integers(0, 9, size=B)
    win = rng.integers(0, 40, size=B)
    win[:6] = [0, 0, 1, 2, 3, 4]
    pre[6:9] = 0
    lens = pre + win
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    counts = rng.integers(0, 60, size=T)
    for b in range(B):
        if win[b] > 4 and b % 3:
            j = int(cu[b] + pre[b] + rng.integers(0, win[b]))
            counts[j:cu[b + 1]] += 100
    counts = np.minimum(counts, I).astype(np.int32)
    bnd, keep = _i32(B), _i32(B)
    log("detect + repack, B=%d, %d rows, policy %d" % (B, T, policy))
    S.seer_step0_detect(dev(counts), dev(cu), dev(pre), dev(win), B, I, S.seer_snr_params(3, 100, 3, 5, 3),
                        bnd, keep)
    torch.cuda.synchronize()
    eb, ek = detect_batch(counts, cu, pre, win, I, Fraction(3, 100), Fraction(3, 5), 3)
    np.testing.assert_array_equal(host(bnd), eb)
    np.testing.assert_array_equal(host(keep), ek)
    src = rng.standard_normal((T, d)).astype(np.float32)
    s1 = dev(src, "bf16")
    cap = int(np.sum(pre)) + B * (int(win.max()) + 8) + 256
    d1 = torch.full((cap, d), -7.0, dtype=torch.bfloat16, device="cuda")
    cu_dst, used = _i32(B + 1), _i32(B)
    route = torch.empty(B, 3, dtype=torch.int32, device="cuda")
    ctrl = torch.zeros(16, dtype=torch.int32, device="cuda")
    desc = S.seer_repack_desc(policy, 1, 5, 1, d * 2, cap, 0, 0)
    S.seer_batch_repack(desc, [s1], [d1], dev(cu), dev(pre), dev(win), keep, B, cu_dst, used, route, ctrl)
    torch.cuda.synchronize()
    rt = route_batch(ek, win, policy, Fraction(1, 5))
    rh = host(route)
    np.testing.assert_array_equal(rh[:, 0], rt.path)
    np.testing.assert_array_equal(rh[:, 1], rt.group)
    np.testing.assert_array_equal(rh[:, 2], rt.alloc)
    exp, cu_e, used_e, cap_e = repack_rows(host(s1), cu, pre, ek, rt.alloc, 1)
    np.testing.assert_array_equal(host(cu_dst), cu_e)
    np.testing.assert_array_equal(host(used), used_e)
    got = host(d1)
    np.testing.assert_array_equal(got[:cap_e], exp)
    assert np.all(got[cap_e:] == -7.0)
    assert host(ctrl)[7] == 0 and host(ctrl)[0] == cu_e[-1]


def test_v_fp16_range_status(S):
    """V is kept in fp16 for the attention's P V product.  Large but finite
    values (|v| up to ~2.5e4) still match the oracle and leave the workspace
    status word clear; values beyond fp16's largest finite value (65504) set
    SEER_STATUS_V_RANGE, which accumulates until seer_layer_status_reset."""
    import torch
    d, H, dh, I = 512, 4, 128, 1024
    rng = np.random.default_rng(77)
    lens = [130, 200, 5]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    x = rng.standard_normal((T, d))
    xd = dev(x, "bf16")
    x = host(xd)

    def layer(v_std):
        W = _rand_layer(rng, d, I, 0.02)
        W["wv"] = rng.standard_normal((d, d)) * (v_std / np.sqrt(d))
        return _round(W, "bf16")

    def status(L):
        torch.cuda.synchronize()
        return int(L.ws[:4].view(torch.int32).item())

    W_in = layer(5000.0)
    L = _Layer(S, d, H, dh, I, "bf16", T, W_in)
    S.seer_layer_status_reset(L.ws)
    y, _ = L.run(xd, dev(cu), len(lens))
    vmax = float(np.abs(host(L.inter("qkv", T, 3 * d))[:, 2 * d:]).max())
    y_ref, _ = layer_forward(x, cu, W_in, H, 1e-5)
    e = rel_err(host(y), y_ref)
    log("  in range: max |v| %.0f, rel err %.3e, status %d" % (vmax, e, status(L)))
    assert 8000 < vmax < 65504 and e <= BF16_TOL and status(L) == 0

    W_out = layer(60000.0)
    L2 = _Layer(S, d, H, dh, I, "bf16", T, W_out)
    L2.ws = L.ws                                   # same workspace: the word accumulates
    L2.run(xd, dev(cu), len(lens))
    log("  out of range: status %d" % status(L2))
    assert status(L2) == S.SEER_STATUS_V_RANGE
    L.run(xd, dev(cu), len(lens))                  # an in-range call does not clear it
    assert status(L) == S.SEER_STATUS_V_RANGE
    S.seer_layer_status_reset(L.ws)
    assert status(L) == 0
    L.run(xd, dev(cu), len(lens))
    assert status(L) == 0


def test_layer_many_rows_unsplit_k_tail(S):
    """A bf16 layer with d_ff = 640 over 33280 rows (130 sequences of 256): every
    projection has more 256x256 tiles than half the CUs, so none splits K, and
    the down projection (K / 64 = 10) ends its four-stage ring on the two-tile
    tail.  (Small layers like the other cases split K instead.)"""
    d, H, dh, I = 256, 2, 128, 640
    rng = np.random.default_rng(43)
    W = _round(_rand_layer(rng, d, I, 0.02), "bf16")
    lens = [256] * 130
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    xd = dev(rng.standard_normal((T, d)), "bf16")
    x = host(xd)
    log("layer bf16 %d rows (d %d, d_ff %d)" % (T, d, I))
    L = _Layer(S, d, H, dh, I, "bf16", T, W)
    y, _ = L.run(xd, dev(cu), len(lens))
    y_ref, _ = layer_forward(x, cu, W, H, 1e-5)
    e = rel_err(host(y), y_ref)
    log("  y rel err %.3e" % e)
    assert e <= BF16_TOL
