"""GPU parity of the synthetic LM head and the remasking sampler.

* seer_lm_head_predict against oracle.sampler.lm_head_predict on the GPU's
  own bf16 rows (teacher-forced): confidence within 1e-3 relative (fp32
  logits and sums); the prediction equal to the oracle's argmax wherever the
  oracle's top two logits are more than 2e-3 (1 + |l_max|) apart, and
  otherwise a token within 1e-3 (1 + |l_max|) of the maximum (the argmax is a
  decision taken on fp32 logits, whose error is ~1e-6 relative) -- small layer (vocab 4096, ragged rows) and the
  LLaDA shape (vocab 126464, sampled rows);
* seer_remask_step against oracle.sampler.remask_step / next_inputs on the
  same predictions and confidences (many ties), bit for bit, for several
  steps-left values, padding rows and partly committed states;
* a sampled denoising loop on the 3-layer stack with the prefix cached:
  every step's committed set and next inputs follow the oracle from the
  GPU's confidences, the inputs change from step to step, and after the last
  step every real window position is committed.
"""
import numpy as np
import pytest

from gpu_util import dev, host, log, upload_weights
from oracle.sampler import MASKED, lm_head_predict, next_inputs, remask_step
from workloads import WORKLOADS
from workloads.generate import lm_head_torch, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    seer.load_library()
    return seer


def _bf(t):
    return t.float().cpu().numpy().astype(np.float64)


def _check_predictions(tag, pred, conf, h, W, eps):
    """The GPU's fp32 logits differ from the oracle's fp64 ones by ~1e-6
    relative (bf16 products are exact in fp32; K-term fp32 accumulation);
    TIE = 1e-3 (1 + |l_max|) bounds that with a wide margin.  Rows whose top
    two logits are further apart than 2 TIE must match the oracle's argmax;
    in the others the GPU's token must be within TIE of the maximum."""
    tok_ref, conf_ref = lm_head_predict(h, W, eps)
    a = h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps)
    logits = a @ W.T
    lmax = logits.max(axis=1)
    tie = 1e-3 * (1.0 + np.abs(lmax))
    second = np.partition(logits, -2, axis=1)[:, -2]
    clear = (lmax - second) > 2 * tie
    for r in range(len(pred)):
        if clear[r]:
            assert pred[r] == tok_ref[r], (tag, r)
        else:
            assert lmax[r] - logits[r, pred[r]] <= tie[r], (tag, r)
    e = np.max(np.abs(conf - conf_ref) / conf_ref)
    log("  %s: %d rows, %d with a clear argmax, confidence rel err %.2e" % (tag, len(pred), int(clear.sum()), e))
    assert e <= 1e-3


@pytest.mark.parametrize("case", ["small", "llada"])
def test_lm_head_predict(S, case):
    import torch
    from paper_2607_14557_amd.runner import dims_for
    if case == "small":
        w = WORKLOADS["small_bf16_ragged"]
        vocab, B, lens = 4096, 5, [1, 130, 257, 0, 300]
    else:
        w = WORKLOADS["llada_b16_ragged"]
        vocab, B, lens = 126464, 4, [97, 260, 3, 300]
    sh = w.shape
    dims = dims_for(sh.d_model, sh.n_heads, sh.head_dim, sh.d_ff, "bf16", w.rms_eps)
    w_lm, _ = lm_head_torch(w, vocab, "cuda")
    cu_h = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    R = int(cu_h[-1])
    rows_ub = R + 37
    gen = torch.Generator(device="cuda")
    gen.manual_seed(42)
    x = torch.randn(rows_ub, sh.d_model, device="cuda", generator=gen).to(torch.bfloat16)
    pred = torch.full((rows_ub,), -7, dtype=torch.int32, device="cuda")
    conf = torch.zeros(rows_ub, dtype=torch.float32, device="cuda")
    ws = torch.empty(S.seer_lm_head_workspace_bytes(dims, vocab, rows_ub), dtype=torch.uint8, device="cuda")
    packed = torch.empty(vocab * sh.d_model * 2, dtype=torch.uint8, device="cuda")
    S.seer_lm_head_prepack(dims, w_lm, vocab, packed)
    S.seer_lm_head_predict(dims, packed, vocab, x, rows_ub, dev(cu_h), B, pred, conf, ws)
    torch.cuda.synchronize()
    if case == "small":
        # the operand order, bit for bit: (32-row block, 16-column block, column half, row, 8 columns)
        w16 = w_lm.view(torch.int16).cpu().numpy()
        want = w16.reshape(vocab // 32, 32, sh.d_model // 16, 2, 8).transpose(0, 2, 3, 1, 4).reshape(-1)
        assert np.array_equal(packed.view(torch.int16).cpu().numpy(), want)
    ph, ch = host(pred), host(conf)
    assert np.all(ph[R:] == -7), "rows past cu[B] must not be written"
    rng = np.random.default_rng(3)
    rows = np.arange(R) if case == "small" else np.array(sorted(set(rng.integers(0, R, 40).tolist()) | {0, R - 1}))
    W = _bf(w_lm)
    _check_predictions(case, ph[rows], ch[rows], _bf(x[torch.from_numpy(rows).cuda()]), W, w.rms_eps)


def test_remask_step(S):
    import torch
    from paper_2607_14557_amd.runner import dims_for
    w = WORKLOADS["small_bf16_ragged"]
    sh = w.shape
    d = sh.d_model
    dims = dims_for(d, sh.n_heads, sh.head_dim, sh.d_ff, "bf16", w.rms_eps)
    rng = np.random.default_rng(7)
    lens = [0, 5, 300, 64, 1, 129]
    used = [0, 3, 290, 64, 1, 100]
    B = len(lens)
    cu_h = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    R = int(cu_h[-1])
    vocab = 50
    emb = torch.randn(vocab, d, device="cuda").to(torch.bfloat16)
    x0 = torch.randn(R, d, device="cuda").to(torch.bfloat16)
    for steps_left in (1, 2, 3, 7, 500):
        tokens_h = np.where(rng.random(R) < 0.3, rng.integers(0, vocab, R), MASKED).astype(np.int32)
        pred_h = rng.integers(0, vocab, R).astype(np.int32)
        conf_h = rng.choice(np.array([0.25, 0.5, 0.125, 1e-3], np.float32), R)
        tokens = dev(tokens_h)
        x_next = torch.full((R, d), 3.0, device="cuda").to(torch.bfloat16)
        S.seer_remask_step(dims, dev(cu_h), dev(np.array(used)), B, 400, steps_left, dev(pred_h), dev(conf_h),
                           tokens, x0, emb, vocab, x_next)
        torch.cuda.synchronize()
        tg, xg = host(tokens), _bf(x_next)
        x0h, embh = _bf(x0), _bf(emb)
        for b in range(B):
            s0, s1 = int(cu_h[b]), int(cu_h[b + 1])
            ref = remask_step(tokens_h[s0:s1], pred_h[s0:s1], conf_h[s0:s1].astype(np.float64), used[b], steps_left)
            np.testing.assert_array_equal(tg[s0:s1], ref)
            np.testing.assert_array_equal(xg[s0:s1], next_inputs(ref, x0h[s0:s1], embh, used[b]))
        log("  steps_left %d: %d committed" % (steps_left, int(np.sum((tokens_h < 0) & (tg >= 0)))))


def test_sampled_denoising_loop(S):
    import torch
    from paper_2607_14557_amd.runner import SeerStack, SyntheticSampler, dims_for
    w = WORKLOADS["small_bf16_stack"]
    sh = w.shape
    d, B, L = sh.d_model, w.batch, w.n_layers
    layers, batch = make_workload(w)
    granule = 256
    T = w.rows_full
    cap = ((T + granule - 1) // granule) * granule + granule
    dims = dims_for(d, sh.n_heads, sh.head_dim, sh.d_ff, "bf16", w.rms_eps)
    st = SeerStack(dims, L, cap)
    for l in range(L):
        st.set_layer(l, upload_weights(layers[l], "bf16"))
    x = dev(batch.x, "bf16")
    cu, off, wl = dev(batch.cu_seqlens), dev(batch.win_off), dev(batch.win_len)
    r = st.step0(x, cu, off, wl, B, T, w.l_det, w.act_eps, granule=granule, trunc_capacity=cap)
    P = np.asarray(batch.win_off, np.int64)
    cu_kv_h = np.concatenate([[0], np.cumsum(P)]).astype(np.int64)
    kv_rows = int(cu_kv_h[-1])
    cu_kv = dev(cu_kv_h)
    caches = st.alloc_kv_caches(kv_rows)
    x_w, cu_w, used_w, _ = st.window_rows(x, cu, off, wl, r.keep_len, B, cap, granule=granule)
    st.forward_export(r.x_trunc, r.cu_trunc, r.seqused, B, cap, caches, cu_kv, kv_rows)
    vocab = 2048
    w_lm, emb = lm_head_torch(w, vocab, "cuda")
    smp = SyntheticSampler(dims, w_lm, emb, cap)
    x0 = x_w.clone()
    bufs = [torch.zeros_like(x_w), torch.zeros_like(x_w)]
    cu_h, used_h = host(cu_w), host(used_w)
    max_used = int(used_h.max())
    # only rows [0, cu_w[B]) of the window buffer are written by the library
    W, embh, x0h = _bf(w_lm), _bf(emb), _bf(x0[:int(cu_h[-1])])
    steps = 4
    x_in = x0
    prev = None
    for s in range(steps):
        steps_left = steps - s
        h = st.forward_cached(x_in, cu_w, used_w, B, cap, caches, cu_kv, kv_rows)
        tok_before = host(smp.tokens).copy()
        x_next = bufs[s % 2]
        smp.step(h, cu_w, used_w, B, cap, x0, x_next, steps_left, max_used)
        torch.cuda.synchronize()
        tg, ph, chf = host(smp.tokens), host(smp.pred), host(smp.conf)
        R = int(cu_h[-1])
        _check_predictions("step %d" % s, ph[:R], chf[:R], _bf(h[:R]), W, w.rms_eps)
        xg = _bf(x_next[:R])
        for b in range(B):
            s0, s1 = int(cu_h[b]), int(cu_h[b + 1])
            ref = remask_step(tok_before[s0:s1], ph[s0:s1], chf[s0:s1].astype(np.float64), int(used_h[b]),
                              steps_left)
            np.testing.assert_array_equal(tg[s0:s1], ref)
            np.testing.assert_array_equal(xg[s0:s1], next_inputs(ref, x0h[s0:s1], embh, int(used_h[b])))
        if prev is not None:
            assert not np.array_equal(prev, xg), "step inputs did not change"
        prev = xg
        x_in = x_next
    tg = host(smp.tokens)
    for b in range(B):
        s0 = int(cu_h[b])
        assert np.all(tg[s0:s0 + int(used_h[b])] >= 0)
    log("  %d steps: every real window position committed" % steps)
