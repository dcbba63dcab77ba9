"""GPU parity at full size: the LLaDA-8B-shaped layer, B=1 and the B=16 ragged batch.

These run the exact launch sequence bench.py times (step-0 layer with the
fused count, SNR scan, routing + compaction, truncated step) and compare every
output with the oracle:
  * boundaries: equal to the planted ones; the oracle's SNR criterion on the
    GPU's counts of the whole window gives the same index; the oracle's own
    step-0 counts (fp64 from the inputs) give it too;
  * counts: every window row of every sequence, teacher-forced (the oracle
    recomputes the MLP activations from the GPU's post-attention residual),
    sparsity fraction within 1e-3; the untethered fraction difference (the
    oracle's own step 0 from the inputs) is reported;
  * offsets / routes / compacted rows: bit-exact against the oracle router;
  * hidden states: every row of the step-0 layer and of the truncated step
    against the oracle's layer on the same inputs (the layer input of both is
    an input of the path: the bf16 embeddings, and their compacted rows), max
    relative error within 2e-2; the 99.9th percentile of the per-row error is
    reported.
"""
import numpy as np
import pytest

from gpu_util import check_counts, dev, fmt_counts, host, log, row_errs, view_ws
from oracle.detect import detect_boundary
from oracle.layer import layer_forward, rms_norm
from oracle.route import repack_rows, route_batch
from oracle.sparsity import sparsity_fraction
from workloads import WORKLOADS
from workloads.generate import make_workload

pytestmark = pytest.mark.gpu
TOL = 2e-2
NAMES = ["llada_b1", "llada_b16_ragged"]
_CACHE = {}


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    seer.load_library()
    return seer


def _run_bench_path(S, w, layers, batch):
    """The bench.py launch sequence; returns host arrays."""
    import torch
    from paper_2607_14557_amd.runner import dims_for
    sh = w.shape
    d, I = sh.d_model, sh.d_ff
    dims = dims_for(d, sh.n_heads, sh.head_dim, I, "bf16", w.rms_eps)
    T = w.rows_full
    cap = ((T + 255) // 256) * 256
    wdev = {k: dev(v, "bf16" if k not in ("g1", "g2") else "f32") for k, v in layers[0].items()}
    packed = torch.empty(S.seer_prepacked_bytes(dims), dtype=torch.uint8, device="cuda")
    S.seer_prepack_weights(dims, wdev, packed)
    del wdev
    ws = torch.empty(S.seer_layer_workspace_bytes(dims, cap), dtype=torch.uint8, device="cuda")
    x = dev(batch.x, "bf16")
    cu, off, wl = dev(batch.cu_seqlens), dev(batch.win_off), dev(batch.win_len)
    y = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    cnt = torch.empty(T, dtype=torch.int32, device="cuda")
    S.seer_layer_forward_varlen(dims, packed, x, y, T, cu, None, w.batch, w.act_eps, cnt, ws)
    torch.cuda.synchronize()
    h1 = host(view_ws(ws, S.seer_layer_workspace_offsets(dims, T)[2], T, d, "bf16"))
    bnd = torch.empty(w.batch, dtype=torch.int32, device="cuda")
    keep = torch.empty(w.batch, dtype=torch.int32, device="cuda")
    S.seer_step0_detect(cnt, cu, off, wl, w.batch, I, S.seer_snr_params(3, 100, 3, 5, 3), bnd, keep)
    x_t = torch.zeros(cap, d, dtype=torch.bfloat16, device="cuda")
    h_t = torch.zeros(cap, d, dtype=torch.bfloat16, device="cuda")
    y_t = torch.zeros(cap, d, dtype=torch.bfloat16, device="cuda")
    cu_t = torch.empty(w.batch + 1, dtype=torch.int32, device="cuda")
    used = torch.empty(w.batch, dtype=torch.int32, device="cuda")
    route = torch.empty(w.batch, 3, dtype=torch.int32, device="cuda")
    ctrl = torch.zeros(16, dtype=torch.int32, device="cuda")
    desc = S.seer_repack_desc(0, 1, 5, 256, d * 2, cap, 0, 0)
    S.seer_batch_repack(desc, [x, y], [x_t, h_t], cu, off, wl, keep, w.batch, cu_t, used, route, ctrl)
    S.seer_layer_forward_varlen(dims, packed, x_t, y_t, cap, cu_t, used, w.batch, 0.0, None, ws)
    torch.cuda.synchronize()
    out = dict(y=host(y), cnt=host(cnt), h1=h1, bnd=host(bnd), keep=host(keep), x_t=host(x_t),
               h_t=host(h_t), y_t=host(y_t), cu_t=host(cu_t), used=host(used), route=host(route),
               ctrl=host(ctrl))
    del packed, ws, x, y, cnt, x_t, h_t, y_t
    torch.cuda.empty_cache()
    return out


def _get(S, name):
    if name not in _CACHE:
        _CACHE.clear()
        w = WORKLOADS[name]
        log("full %s: inputs" % name)
        layers, batch = make_workload(w)
        W = {k: np.asarray(v, np.float64) for k, v in layers[0].items()}
        log("full %s: GPU path" % name)
        g = _run_bench_path(S, w, layers, batch)
        _CACHE[name] = (w, W, batch, g)
    return _CACHE[name]


def _report_rows(tag, e):
    q = float(np.quantile(e, 0.999)) if e.size else 0.0
    log("  %s: %d rows, max rel err %.3e (row %d), 99.9th percentile %.3e, median %.3e" %
        (tag, e.size, e.max(), int(e.argmax()), q, float(np.median(e))))
    return q


@pytest.mark.parametrize("name", NAMES)
def test_full_boundaries_and_counts(S, name):
    w, W, batch, g = _get(S, name)
    I = w.shape.d_ff
    S_full, P = w.seq_len_full, w.prefix_len
    np.testing.assert_array_equal(g["bnd"], batch.planted)
    np.testing.assert_array_equal(g["keep"], batch.planted + 1)
    worst = dict(max_count_diff=0, max_frac_diff=0.0)
    for b in range(w.batch):
        r0 = b * S_full + P
        bn = rms_norm(g["h1"][r0:r0 + w.window], W["g2"], w.rms_eps)
        cg = g["cnt"][r0:r0 + w.window]
        cr = check_counts(cg, bn, W["wg"], W["wu"], w.act_eps, I)
        ib, kb = detect_boundary(cg, I)
        assert ib == g["bnd"][b], "seq %d: oracle criterion on the GPU counts gives %d" % (b, ib)
        log("  seq %d: boundary %d, teacher-forced %s" % (b, ib, fmt_counts(cr)))
        worst = {k: max(worst[k], cr[k]) for k in worst}
    log("  %s teacher-forced counts, all %d window rows: max diff %d, max fraction diff %.2e" %
        (name, w.batch * w.window, worst["max_count_diff"], worst["max_frac_diff"]))


@pytest.mark.parametrize("name", NAMES)
def test_full_routing_and_compaction(S, name):
    w, W, batch, g = _get(S, name)
    rt = route_batch(g["keep"], batch.win_len)
    np.testing.assert_array_equal(g["route"][:, 0], rt.path)
    np.testing.assert_array_equal(g["route"][:, 1], rt.group)
    np.testing.assert_array_equal(g["route"][:, 2], rt.alloc)
    x_bf = host(dev(batch.x, "bf16"))
    exp_x, cu_e, used_e, cap_e = repack_rows(x_bf, batch.cu_seqlens, batch.win_off, g["keep"], rt.alloc, 256)
    np.testing.assert_array_equal(g["cu_t"], cu_e)
    np.testing.assert_array_equal(g["used"], used_e)
    np.testing.assert_array_equal(g["x_t"][:cap_e], exp_x)
    exp_h, _, _, _ = repack_rows(g["y"], batch.cu_seqlens, batch.win_off, g["keep"], rt.alloc, 256)
    np.testing.assert_array_equal(g["h_t"][:cap_e], exp_h)
    assert g["ctrl"][0] == cu_e[-1] and g["ctrl"][7] == 0 and g["ctrl"][8] == 1


@pytest.mark.parametrize("name", NAMES)
def test_full_step0_every_row(S, name):
    """The step-0 layer over the full window, every row of every sequence; its
    input is the path's input, so this is also the untethered comparison: the
    oracle's own counts must give the planted boundaries."""
    w, W, batch, g = _get(S, name)
    sh = w.shape
    I = sh.d_ff
    S_full, P = w.seq_len_full, w.prefix_len
    x_bf = host(dev(batch.x, "bf16"))
    errs, dfr = [], 0.0
    for b in range(w.batch):
        s0 = b * S_full
        sl = slice(s0, s0 + S_full)
        y_ref, c_ref = layer_forward(x_bf[sl], [0, S_full], W, sh.n_heads, w.rms_eps, act_eps=w.act_eps)
        e = row_errs(g["y"][sl], y_ref)
        errs.append(e)
        ib, _ = detect_boundary(c_ref[P:], I)
        assert ib == batch.planted[b], "seq %d: the oracle's own counts give %d" % (b, ib)
        d_un = np.abs(sparsity_fraction(g["cnt"][sl][P:], I) - sparsity_fraction(c_ref[P:], I)).max()
        dfr = max(dfr, float(d_un))
        log("  seq %d: step-0 rows max rel err %.3e; untethered window fraction diff %.2e" %
            (b, e.max(), d_un))
        assert e.max() <= TOL, "seq %d row %d: %.3e" % (b, int(e.argmax()), e.max())
    _report_rows("%s step-0 layer" % name, np.concatenate(errs))
    log("  %s untethered sparsity fraction diff max %.2e (reported)" % (name, dfr))


@pytest.mark.parametrize("name", NAMES)
def test_full_truncated_step_every_row(S, name):
    """One truncated denoising step over the compacted batch, every kept row."""
    w, W, batch, g = _get(S, name)
    sh = w.shape
    tot = int(g["cu_t"][-1])
    y_ref, _ = layer_forward(g["x_t"][:tot], g["cu_t"], W, sh.n_heads, w.rms_eps, seqused=g["used"])
    errs = []
    for b in range(w.batch):
        t0 = int(g["cu_t"][b])
        sl = slice(t0, t0 + int(g["used"][b]))
        errs.append(row_errs(g["y_t"][sl], y_ref[sl]))
        pad = slice(t0 + int(g["used"][b]), int(g["cu_t"][b + 1]))
        assert np.all(g["y_t"][pad] == 0.0), "seq %d: padding rows must stay zero" % b
    e = np.concatenate(errs)
    _report_rows("%s truncated step" % name, e)
    assert e.max() <= TOL, "row %d: %.3e" % (int(e.argmax()), e.max())
