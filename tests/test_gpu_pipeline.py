"""GPU parity of the whole step-0 pipeline against the oracle, small workloads.

Step 0 (layers up to the detection layer on the full window, fused count),
the SNR scan, routing + compaction and the truncated denoising step, all
through the C ABI, compared with oracle.run_pipeline on the same seeded
inputs.  Boundaries, offsets, routes and compacted embeddings are bit-exact;
counts are gated teacher-forced (the oracle recomputes the detection layer's
MLP from the GPU's own post-attention residual); hidden states are gated per
layer, teacher-forced, and the end-to-end error of stacks is reported.
"""
import numpy as np
import pytest

import oracle
from gpu_util import check_counts, dev, fmt_counts, host, log, rel_err, upload_weights, view_ws
from oracle.layer import layer_forward, rms_norm
from oracle.route import repack_rows
from workloads import WORKLOADS
from workloads.generate import make_workload

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-4}


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    seer.load_library()
    return seer


def build_stack(w, layers, max_rows):
    from paper_2607_14557_amd.runner import SeerStack, dims_for
    sh = w.shape
    st = SeerStack(dims_for(sh.d_model, sh.n_heads, sh.head_dim, sh.d_ff, w.dtype, w.rms_eps),
                   w.n_layers, max_rows)
    for l in range(w.n_layers):
        st.set_layer(l, upload_weights(layers[l], w.dtype))
    return st


@pytest.mark.parametrize("name", ["tiny_f32", "small_bf16_ragged", "small_bf16_stack"])
def test_pipeline_vs_oracle(S, name):
    import torch
    w = WORKLOADS[name]
    sh = w.shape
    tol = TOL[w.dtype]
    log("pipeline %s: generating inputs" % name)
    layers, batch = make_workload(w)
    W64 = [{k: np.asarray(v, np.float64) for k, v in L.items()} for L in layers]
    T = w.rows_full
    granule = 256
    cap = T + granule
    st = build_stack(w, layers, cap)
    x = dev(batch.x, w.dtype)
    cu, off, wl = dev(batch.cu_seqlens), dev(batch.win_off), dev(batch.win_len)

    # -- teacher-forced count at the detection layer (layer by layer through the ABI)
    log("pipeline %s: step-0 layers 0..%d" % (name, w.l_det))
    cur = x
    cnt = torch.empty(T, dtype=torch.int32, device="cuda")
    for l in range(w.l_det + 1):
        nxt = torch.empty_like(x)
        st.layer(l, cur, nxt, cu, None, w.batch, T, act_eps=w.act_eps,
                 act_count=cnt if l == w.l_det else None)
        cur = nxt
    torch.cuda.synchronize()
    off6 = S.seer_layer_workspace_offsets(st.dims, T)   # layout of calls made with rows_ub = T
    h1 = host(view_ws(st.workspace, off6[2], T, sh.d_model, w.dtype))
    b = rms_norm(h1, W64[w.l_det]["g2"], w.rms_eps)
    # fp32 layers store the activations unrounded: the kernel's own values
    act_gpu = host(view_ws(st.workspace, off6[3], T, sh.d_ff, w.dtype)) if w.dtype == "f32" else None
    cr = check_counts(host(cnt), b, W64[w.l_det]["wg"], W64[w.l_det]["wu"], w.act_eps, sh.d_ff,
                      band=True, act_gpu=act_gpu)
    log("  teacher-forced %s (I=%d)" % (fmt_counts(cr), sh.d_ff))

    # -- the product path: step0 = layers + count + detect + repack + remaining layers
    log("pipeline %s: step0 through the runner" % name)
    r = st.step0(x, cu, off, wl, w.batch, T, w.l_det, w.act_eps, granule=granule, trunc_capacity=cap)
    torch.cuda.synchronize()
    log("pipeline %s: oracle" % name)
    res = oracle.run_pipeline(layers, batch.x, batch.cu_seqlens, batch.win_off, batch.win_len,
                              sh.n_heads, sh.d_ff, w.rms_eps, w.act_eps, w.l_det, granule=granule)
    np.testing.assert_array_equal(res.boundary, batch.planted)
    np.testing.assert_array_equal(host(r.boundary), res.boundary)
    np.testing.assert_array_equal(host(r.keep_len), res.keep_len)
    cdiff = np.abs(host(r.counts) - res.counts).max()
    log("  untethered count diff max %d (fraction %.2e, reported)" % (cdiff, cdiff / sh.d_ff))
    np.testing.assert_array_equal(host(r.cu_trunc), res.cu_trunc)
    np.testing.assert_array_equal(host(r.seqused), res.seqused)
    route = host(r.route)
    np.testing.assert_array_equal(route[:, 0], res.route.path)
    np.testing.assert_array_equal(route[:, 1], res.route.group)
    np.testing.assert_array_equal(route[:, 2], res.route.alloc)
    ctrl = host(r.ctrl)
    assert ctrl[0] == res.cu_trunc[-1] and ctrl[1] == res.capacity and ctrl[7] == 0 and ctrl[8] == 1
    np.testing.assert_array_equal(host(r.x_trunc[:res.capacity]), res.x_trunc)

    # -- step-0 output (compacted) and the truncated step, gated per layer
    cu_t = r.cu_trunc
    used = r.seqused
    if w.n_layers == 1:
        e0 = rel_err(host(r.h_trunc[:int(res.cu_trunc[-1])]), res.y_step0[:int(res.cu_trunc[-1])])
        log("  step-0 output rel err %.3e" % e0)
        assert e0 <= tol
    else:
        log("  step-0 end-to-end rel err %.3e (reported)" %
            rel_err(host(r.h_trunc[:int(res.cu_trunc[-1])]), res.y_step0[:int(res.cu_trunc[-1])]))
    tot = int(res.cu_trunc[-1])          # the layer writes rows [0, cu[B]) only
    cur = r.x_trunc
    for l in range(w.n_layers):
        nxt = torch.zeros_like(cur)
        st.layer(l, cur, nxt, cu_t, used, w.batch, cap)
        torch.cuda.synchronize()
        xin = host(cur[:tot])
        y_ref, _ = layer_forward(xin, res.cu_trunc, W64[l], sh.n_heads, w.rms_eps, seqused=res.seqused)
        y = host(nxt)
        e = rel_err(y[:tot], y_ref)
        log("  truncated step layer %d rel err %.3e (teacher-forced)" % (l, e))
        assert e <= tol
        assert np.all(y[tot:] == 0.0)
        cur = nxt
    e_end = rel_err(host(cur)[:tot], res.y_step[:tot])
    log("  truncated step end-to-end rel err %.3e" % e_end)
    if w.n_layers == 1:
        assert e_end <= tol


def test_step0_capacity_and_overflow(S):
    """The runner's default compacted capacity holds the routing's worst case
    (every window padded to the longest); a capacity the routed batch does not
    fit raises SeerError (the repack kernel's status) before any later layer."""
    import torch
    w = WORKLOADS["small_bf16_stack"]
    layers, batch = make_workload(w)
    T = w.rows_full
    st = build_stack(w, layers, T + 256)
    x = dev(batch.x, w.dtype)
    cu, off, wl = dev(batch.cu_seqlens), dev(batch.win_off), dev(batch.win_len)
    log("step0: default capacity")
    r = st.step0(x, cu, off, wl, w.batch, T, w.l_det, w.act_eps, granule=256)
    torch.cuda.synchronize()
    worst = int(np.sum(batch.win_off)) + w.batch * int(np.max(batch.win_len))
    assert r.x_trunc.shape[0] == -(-worst // 256) * 256
    ctrl = host(r.ctrl)
    assert ctrl[7] == 0 and ctrl[8] == 1 and ctrl[1] <= r.x_trunc.shape[0]
    np.testing.assert_array_equal(host(r.boundary), batch.planted)
    log("step0: a 256-row capacity (the compacted batch needs %d rows)" % int(ctrl[0]))
    assert ctrl[0] > 256
    with pytest.raises(S.SeerError) as ei:
        st.step0(x, cu, off, wl, w.batch, T, w.l_det, w.act_eps, granule=256, trunc_capacity=256)
    assert ei.value.code == S.SEER_EWORKSPACE
