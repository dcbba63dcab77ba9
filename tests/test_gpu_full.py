"""GPU parity at full size: the LLaDA-8B-shaped layer, B=1 and the B=16 ragged batch.

These run the exact launch sequence bench.py times (step-0 layer with the
fused count, SNR scan, routing + compaction, truncated step) and compare with
the oracle where it finishes in seconds:
  * boundaries: the oracle's SNR criterion on counts it recomputes from the
    GPU's own detection-layer residual (teacher-forced) over window positions
    [0, b_gpu + lookahead) -- exactly the positions that decide whether b_gpu
    is the first qualifying one -- must give b_gpu; b_gpu must also equal the
    planted boundary; the untethered oracle pipeline on the first sequences
    must agree too;
  * counts: within the fp32-consistent band of the teacher-forced count;
  * offsets / routes / compacted rows: bit-exact against the oracle router;
  * hidden states: sampled rows (first, last, around the cut, random) of the
    step-0 output and of the truncated step against the oracle's layer
    evaluated for those rows with keys/values over the whole sequence.
"""
import numpy as np
import pytest

import oracle
from gpu_util import check_counts, dev, host, log, rel_err, view_ws
from oracle.detect import detect_boundary
from oracle.layer import layer_forward_rows, rms_norm
from oracle.route import repack_rows, route_batch
from workloads import WORKLOADS
from workloads.generate import make_workload

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    seer.load_library()
    return seer


def _run_bench_path(S, w, layers, batch):
    """The bench.py launch sequence; returns device tensors."""
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
    return dict(y=host(y), cnt=host(cnt), h1=h1, bnd=host(bnd), keep=host(keep), x_t=host(x_t),
                h_t=host(h_t), y_t=host(y_t), cu_t=host(cu_t), used=host(used), route=host(route),
                ctrl=host(ctrl))


def _sample_rows(rng, S_len, cut, k=4):
    rows = {0, S_len - 1, max(cut - 1, 0), min(cut, S_len - 1)}
    rows |= set(int(r) for r in rng.integers(0, S_len, size=k))
    return np.array(sorted(rows))


@pytest.mark.parametrize("name,n_seq_check,n_untethered", [("llada_b1", 1, 1),
                                                           ("llada_b16_ragged", 5, 2)])
def test_full_size_parity(S, name, n_seq_check, n_untethered):
    w = WORKLOADS[name]
    sh = w.shape
    I = sh.d_ff
    log("full %s: inputs" % name)
    layers, batch = make_workload(w)
    W = {k: np.asarray(v, np.float64) for k, v in layers[0].items()}
    log("full %s: GPU path" % name)
    g = _run_bench_path(S, w, layers, batch)
    S_full = w.seq_len_full
    P = w.prefix_len
    rng = np.random.default_rng(5)

    # -- boundaries: planted, and the oracle's criterion on teacher-forced counts
    np.testing.assert_array_equal(g["bnd"], batch.planted)
    np.testing.assert_array_equal(g["keep"], batch.planted + 1)
    Wg, Wu = W["wg"], W["wu"]
    for b in range(w.batch):
        hi = min(int(g["bnd"][b]) + 3, w.window)
        r0 = b * S_full + P
        bn = rms_norm(g["h1"][r0:r0 + hi], W["g2"], w.rms_eps)
        cg = g["cnt"][r0:r0 + hi]
        dmax, ties = check_counts(cg, bn, Wg, Wu, w.act_eps, I)
        ib, kb = detect_boundary(cg, I)
        assert ib == g["bnd"][b], "seq %d: oracle criterion on the GPU counts gives %d" % (b, ib)
        log("  seq %d: boundary %d, count diff %d (ties %d) over %d positions" %
            (b, ib, dmax, ties, hi))

    # -- routing and compaction against the oracle router
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

    # -- hidden states on sampled rows (keys/values over whole sequences)
    for b in range(n_seq_check):
        s0 = b * S_full
        xs = x_bf[s0:s0 + S_full]
        rows = _sample_rows(rng, S_full, P + int(batch.planted[b]))
        ref = layer_forward_rows(xs, S_full, W, sh.n_heads, w.rms_eps, rows)["y"]
        e0 = rel_err(g["y"][s0 + rows], ref)
        t0 = int(g["cu_t"][b])
        St = int(g["used"][b])
        rows_t = _sample_rows(rng, St, P + int(batch.planted[b]))
        ref_t = layer_forward_rows(g["x_t"][t0:t0 + St], St, W, sh.n_heads, w.rms_eps, rows_t)["y"]
        e1 = rel_err(g["y_t"][t0 + rows_t], ref_t)
        log("  seq %d: full-window rows err %.3e, truncated-step rows err %.3e" % (b, e0, e1))
        assert e0 <= TOL and e1 <= TOL

    # -- untethered oracle pipeline on the first sequences
    for b in range(n_untethered):
        s0 = b * S_full
        res = oracle.run_pipeline(layers, batch.x[s0:s0 + S_full], [0, S_full], batch.win_off[b:b + 1],
                                  batch.win_len[b:b + 1], sh.n_heads, I, w.rms_eps, w.act_eps, w.l_det)
        assert int(res.boundary[0]) == int(g["bnd"][b])
        diff = np.abs(res.counts[P:] - g["cnt"][s0 + P:s0 + S_full])
        t0 = int(g["cu_t"][b])
        St = int(g["used"][b])
        e = rel_err(g["y_t"][t0:t0 + St], res.y_step[:St])
        e0 = rel_err(g["h_t"][t0:t0 + St], res.y_step0[:St])
        log("  untethered seq %d: boundary %d, window count diff max %d (fraction %.2e), "
            "step-0 err %.3e, truncated step err %.3e" %
            (b, res.boundary[0], diff.max(), diff.max() / I, e0, e))
        assert e <= TOL and e0 <= TOL
