"""GPU parity on the two 32-layer stacks (LLaDA-8B layer shape, bf16):
the multi-crop batch (B=8, 3645-token visual prefix, 64-token prompt,
512-position window, boundaries uniform in [32, 256]) and the video batch
(B=4, 3136-token prefix, 128-token prompt, 2048-position window, boundaries
uniform in [64, 1024]); detection after the fourth layer.

The product path (SeerStack.step0, then truncated steps with
SeerStack.forward) is run and then replayed call by call to capture the
intermediates the oracle needs; the replay must reproduce it bit for bit.
Against the oracle:
  * boundaries: equal to the planted ones, and the oracle's SNR criterion on
    the GPU counts of the whole window gives b; on every window row the
    sparsity fraction is within 1e-3 of the oracle's, recomputed from the
    GPU's own detection-layer residual (teacher-forced);
  * routes, offsets and compacted rows: bit-exact against the oracle router;
  * hidden states: sampled rows of the first and last sequence, teacher-forced
    at sampled layers of step 0 (full window) and of the truncated step, with
    keys and values over the whole sequence.  The 32-layer end-to-end drift is
    reported, not gated (each layer rounds to bf16).
"""
import numpy as np
import pytest

from gpu_util import check_counts, dev, fmt_counts, host, log, rel_err, view_ws
from oracle.detect import detect_boundary
from oracle.layer import layer_forward_rows, rms_norm
from oracle.route import repack_rows, route_batch
from workloads import WORKLOADS
from workloads.generate import layer_weights_torch, make_stack_batch

pytestmark = pytest.mark.gpu
TOL = 2e-2
GRANULE = 256


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    seer.load_library()
    return seer


def _w64(Wdev):
    return {k: host(v) for k, v in Wdev.items()}


def _rows(rng, n, cut, k=3):
    r = {0, n - 1, max(cut - 1, 0), min(cut, n - 1)}
    r |= set(int(i) for i in rng.integers(0, n, size=k))
    return np.array(sorted(r))


def _check_rows(tag, W, x_seq, used, y_seq, rows, n_heads, eps):
    ref = layer_forward_rows(x_seq, used, W, n_heads, eps, rows)["y"]
    e = rel_err(y_seq[rows], ref)
    log("  %s: rel err %.3e over %d rows" % (tag, e, len(rows)))
    assert e <= TOL, tag


@pytest.mark.parametrize("name", ["llada32_multicrop_b8", "llada32_video_b4"])
def test_stack_parity(S, name):
    import torch
    from paper_2607_14557_amd.runner import SeerStack, dims_for
    w = WORKLOADS[name]
    sh = w.shape
    d, I, B, L, P = sh.d_model, sh.d_ff, w.batch, w.n_layers, w.prefix_len
    T = w.rows_full
    cap = ((T + GRANULE - 1) // GRANULE) * GRANULE + GRANULE
    step0_layers = sorted({0, w.l_det})
    trunc_layers = sorted({0, L // 2, L - 1})
    seqs = sorted({0, B - 1})
    rng = np.random.default_rng(11)

    log("stack %s: inputs (%d rows, %d layers)" % (name, T, L))
    batch = make_stack_batch(w, "cuda")
    st = SeerStack(dims_for(d, sh.n_heads, sh.head_dim, I, "bf16", w.rms_eps), L, cap)
    for l in range(L):
        Wl = layer_weights_torch(w, l, "cuda")
        st.set_layer(l, Wl)
        del Wl
    x = dev(batch.x, "bf16")
    cu, off, wl = dev(batch.cu_seqlens), dev(batch.win_off), dev(batch.win_len)

    # -- the product path
    log("stack %s: step 0 and one truncated step through the runner" % name)
    r = st.step0(x, cu, off, wl, B, T, w.l_det, w.act_eps, granule=GRANULE, trunc_capacity=cap)
    y_step = st.forward(r.x_trunc, r.cu_trunc, r.seqused, B, cap, out=torch.empty_like(r.x_trunc))
    y_step2 = st.forward(r.x_trunc, r.cu_trunc, r.seqused, B, cap, out=torch.empty_like(r.x_trunc))
    torch.cuda.synchronize()
    bnd, keep = host(r.boundary), host(r.keep_len)
    np.testing.assert_array_equal(bnd, batch.planted)
    np.testing.assert_array_equal(keep, batch.planted + 1)
    tot = int(host(r.cu_trunc)[-1])
    assert torch.equal(y_step[:tot], y_step2[:tot]), "truncated step is not deterministic"

    # -- replay of the same calls, keeping what the oracle needs
    log("stack %s: replay" % name)
    cnt = torch.empty(T, dtype=torch.int32, device="cuda")
    ins = {}
    cur = x
    for l in range(w.l_det + 1):
        ins[l] = cur
        nxt = torch.empty_like(x)
        st.layer(l, cur, nxt, cu, None, B, T, act_eps=w.act_eps,
                 act_count=cnt if l == w.l_det else None)
        cur = nxt
    torch.cuda.synchronize()
    assert torch.equal(cnt, r.counts)
    off_ws = S.seer_layer_workspace_offsets(st.dims, T)     # layout of calls with rows_ub = T
    h1_dev = view_ws(st.workspace, off_ws[2], T, d, "bf16")
    win_rows = {}
    for b in range(B):
        r0 = int(batch.cu_seqlens[b]) + P
        win_rows[b] = (host(h1_dev[r0:r0 + w.window]), host(cnt[r0:r0 + w.window]))
    y_det = cur
    bnd2 = torch.empty(B, dtype=torch.int32, device="cuda")
    keep2 = torch.empty(B, dtype=torch.int32, device="cuda")
    S.seer_step0_detect(cnt, cu, off, wl, B, I, S.seer_snr_params(3, 100, 3, 5, 3), bnd2, keep2)
    x_t = torch.zeros(cap, d, dtype=torch.bfloat16, device="cuda")
    h_t = torch.zeros(cap, d, dtype=torch.bfloat16, device="cuda")
    cu_t = torch.empty(B + 1, dtype=torch.int32, device="cuda")
    used = torch.empty(B, dtype=torch.int32, device="cuda")
    route = torch.empty(B, 3, dtype=torch.int32, device="cuda")
    ctrl = torch.zeros(16, dtype=torch.int32, device="cuda")
    desc = S.seer_repack_desc(0, 1, 5, GRANULE, d * 2, cap, 0, 0)
    S.seer_batch_repack(desc, [x, y_det], [x_t, h_t], cu, off, wl, keep2, B, cu_t, used, route, ctrl)
    torch.cuda.synchronize()
    assert torch.equal(bnd2, r.boundary) and torch.equal(cu_t, r.cu_trunc)
    assert torch.equal(x_t[:tot], r.x_trunc[:tot])

    # -- routing and compaction against the oracle router
    rt = route_batch(keep, batch.win_len)
    rh = host(route)
    np.testing.assert_array_equal(rh[:, 0], rt.path)
    np.testing.assert_array_equal(rh[:, 1], rt.group)
    np.testing.assert_array_equal(rh[:, 2], rt.alloc)
    exp_x, cu_e, used_e, cap_e = repack_rows(batch.x, batch.cu_seqlens, batch.win_off, keep, rt.alloc,
                                             GRANULE)
    np.testing.assert_array_equal(host(cu_t), cu_e)
    np.testing.assert_array_equal(host(used), used_e)
    assert tot == cu_e[-1] and cap_e <= cap
    np.testing.assert_array_equal(x_t[:cap_e].float().cpu().numpy(), exp_x)
    del exp_x
    y_det_h = y_det.float().cpu().numpy()
    exp_h, _, _, _ = repack_rows(y_det_h, batch.cu_seqlens, batch.win_off, keep, rt.alloc, GRANULE)
    np.testing.assert_array_equal(h_t[:cap_e].float().cpu().numpy(), exp_h)
    del exp_h, y_det_h
    h_cur = h_t
    for l in range(w.l_det + 1, L):
        nxt = torch.empty_like(h_t)
        st.layer(l, h_cur, nxt, cu_t, used, B, cap)
        h_cur = nxt
    torch.cuda.synchronize()
    assert torch.equal(h_cur[:tot], r.h_trunc[:tot])

    # truncated step replay, keeping the inputs and outputs of sampled layers (checked sequences)
    t_io = {}
    cur = x_t
    used_h, cu_th = host(used), host(cu_t)
    for l in range(L):
        nxt = torch.empty_like(x_t)
        st.layer(l, cur, nxt, cu_t, used, B, cap)
        if l in trunc_layers:
            torch.cuda.synchronize()
            t_io[l] = {b: (host(cur[cu_th[b]:cu_th[b] + used_h[b]]), host(nxt[cu_th[b]:cu_th[b] + used_h[b]]))
                       for b in seqs}
        cur = nxt
    torch.cuda.synchronize()
    assert torch.equal(cur[:tot], y_step[:tot])

    # -- boundaries and counts against the oracle (teacher-forced)
    log("stack %s: oracle checks" % name)
    W_det = _w64(layer_weights_torch(w, w.l_det, "cuda"))
    worst = 0.0
    for b in range(B):
        h1, cg = win_rows[b]
        cr = check_counts(cg, rms_norm(h1, W_det["g2"], w.rms_eps), W_det["wg"], W_det["wu"],
                          w.act_eps, I)
        ib, _ = detect_boundary(cg, I)
        assert ib == bnd[b], "seq %d: oracle criterion on the GPU counts gives %d" % (b, ib)
        log("  seq %d: boundary %d, teacher-forced %s (whole window)" % (b, ib, fmt_counts(cr)))
        worst = max(worst, cr["max_frac_diff"])
    log("  %s teacher-forced sparsity fraction diff max %.2e over all %d window rows" %
        (name, worst, B * w.window))

    # -- hidden states, teacher-forced at sampled layers
    for l in sorted(set(step0_layers) | set(trunc_layers)):
        W = W_det if l == w.l_det else _w64(layer_weights_torch(w, l, "cuda"))
        for b in seqs:
            cut = P + int(bnd[b])
            if l in step0_layers:
                s0, n = int(batch.cu_seqlens[b]), w.seq_len_full
                y_l = ins[l + 1] if l + 1 in ins else y_det
                rows = _rows(rng, n, cut)
                _check_rows("step 0 layer %d seq %d" % (l, b), W, host(ins[l][s0:s0 + n]), n,
                            host(y_l[s0:s0 + n]), rows, sh.n_heads, w.rms_eps)
            if l in trunc_layers:
                xin, yout = t_io[l][b]
                rows = _rows(rng, len(xin), cut)
                _check_rows("truncated layer %d seq %d" % (l, b), W, xin, len(xin), yout, rows,
                            sh.n_heads, w.rms_eps)
        del W
