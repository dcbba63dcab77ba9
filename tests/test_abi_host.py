"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function include/seer.h declares, and rejects bad arguments with the
documented status codes before launching anything."""
import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "seer.h")


@pytest.fixture(scope="module")
def S():
    from paper_2607_14557_amd import seer
    if not os.path.exists(seer.LIB_PATH):
        pytest.skip("libseer.so not built")
    seer.load_library()
    return seer


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(seer_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(S):
    names = declared_functions()
    assert len(names) >= 9
    lib = ctypes.CDLL(S.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(S.EXPORTED)
    assert S.seer_abi_version() == 104


def dims(S, d=4096, h=32, dh=128, i=12288, dtype=1):
    return S.seer_dims(d, h, dh, i, dtype, 1e-5)


def test_dims_validation(S):
    assert S.seer_prepacked_bytes(dims(S)) == 436207616
    assert S.seer_prepacked_bytes(dims(S, dh=64)) == 0
    assert "head_dim" in S.seer_last_error()
    assert S.seer_prepacked_bytes(dims(S, d=4000, h=32, dh=125)) == 0     # bf16 needs d % 256
    assert S.seer_prepacked_bytes(dims(S, d=256, h=4, dh=64, i=688, dtype=2)) > 0
    assert S.seer_prepacked_bytes(dims(S, dtype=7)) == 0
    d = dims(S)
    d.rope_theta = 500000.0
    assert S.seer_prepacked_bytes(d) == 436207616
    for bad in (0.5, 1.0, -1.0, float("inf"), float("nan")):
        d.rope_theta = bad
        assert S.seer_prepacked_bytes(d) == 0, bad
        assert "rope_theta" in S.seer_last_error()
    d = dims(S, d=260, h=4, dh=65, i=688, dtype=2)
    assert S.seer_prepacked_bytes(d) > 0
    d.rope_theta = 10000.0
    assert S.seer_prepacked_bytes(d) == 0 and "even head_dim" in S.seer_last_error()


def test_workspace_layout_is_consistent(S):
    d = dims(S)
    a = S.seer_layer_workspace_bytes(d, 1000)
    b = S.seer_layer_workspace_bytes(d, 2000)
    assert 0 < a < b
    off = S.seer_layer_workspace_offsets(d, 2000)
    assert off == sorted(off) and off[7] == b and all(o % 256 == 0 for o in off)
    # bytes [0, 256) are the header holding the status word, for every rows bound
    assert off[0] == 256 and S.seer_layer_workspace_offsets(d, 0)[0] == 256
    # bf16: qkv, o, h1 (bf16), act, two fp32 statistics, low part of h1 (bf16)
    assert b >= 2000 * (3 * 4096 * 2 + 4096 * 2 * 2 + 12288 * 2 + 8 + 4096 * 2)


FAKE = 1 << 20   # a non-null, aligned address that is never dereferenced


def call_layer(S, d, **kw):
    a = dict(w=FAKE, x_in=FAKE, x_out=FAKE + 4096, rows=100, cu=FAKE, used=None, batch=1,
             eps=0.0, cnt=None, ws=FAKE, ws_bytes=1 << 40)
    a.update(kw)
    L = S.load_library()
    return L.seer_layer_forward_varlen(ctypes.byref(d), a["w"], a["x_in"], a["x_out"], a["rows"],
                                       a["cu"], a["used"], a["batch"], a["eps"], a["cnt"], a["ws"],
                                       a["ws_bytes"], 0)


def test_layer_forward_argument_errors(S):
    d = dims(S)
    assert call_layer(S, d, w=None) == S.SEER_EINVAL
    assert call_layer(S, d, rows=174763) == S.SEER_EUNSUPPORTED      # 174763 x 12288 x 2 B >= 4 GiB
    assert "4 GiB" in S.seer_last_error()
    assert call_layer(S, d, cu=None) == S.SEER_EINVAL
    assert call_layer(S, d, batch=0) == S.SEER_EINVAL
    assert call_layer(S, d, rows=0) == S.SEER_EINVAL
    assert call_layer(S, d, x_out=FAKE) == S.SEER_EINVAL          # aliasing
    assert call_layer(S, d, ws=FAKE + 8) == S.SEER_EINVAL         # misaligned workspace
    assert call_layer(S, d, ws_bytes=1024) == S.SEER_EWORKSPACE
    assert "workspace" in S.seer_last_error()
    assert call_layer(S, d, cnt=FAKE, eps=-1.0) == S.SEER_EINVAL
    assert call_layer(S, dims(S, dh=64)) == S.SEER_EINVAL              # 32 x 64 != 4096
    assert call_layer(S, dims(S, h=64, dh=64)) == S.SEER_EUNSUPPORTED  # bf16 needs head_dim 128
    L = S.load_library()
    rc = L.seer_layer_forward_varlen_timed(ctypes.byref(d), FAKE, FAKE, FAKE + 4096, 100, FAKE, None,
                                           1, 0.0, None, FAKE, 1 << 40, 0, None)
    assert rc == S.SEER_EINVAL and "events" in S.seer_last_error()
    # NULL entries are skipped, not rejected: the call goes on to the next check
    ev = (ctypes.c_void_p * 8)(*([None] * 5 + [FAKE, FAKE, None]))
    rc = L.seer_layer_forward_varlen_timed(ctypes.byref(d), FAKE, FAKE, FAKE + 4096, 100, FAKE, None,
                                           0, 0.0, None, FAKE, 1 << 40, 0, ev)
    assert rc == S.SEER_EINVAL and "batch" in S.seer_last_error()


def test_detect_argument_errors(S):
    L = S.load_library()
    good = S.seer_snr_params(3, 100, 3, 5, 3)

    def call(p=good, batch=1, dff=100, cnt=FAKE):
        return L.seer_step0_detect(cnt, FAKE, FAKE, FAKE, batch, dff, ctypes.byref(p), FAKE, FAKE, 0)

    assert call(cnt=None) == S.SEER_EINVAL
    assert call(batch=0) == S.SEER_EINVAL
    assert call(dff=0) == S.SEER_EINVAL
    assert call(p=S.seer_snr_params(3, 0, 3, 5, 3)) == S.SEER_EINVAL
    assert call(p=S.seer_snr_params(-1, 100, 3, 5, 3)) == S.SEER_EINVAL
    assert call(p=S.seer_snr_params(3, 100, 3, 5, 0)) == S.SEER_EINVAL


def test_detection_layer_argument_errors(S):
    L = S.load_library()
    d = dims(S)
    good = S.seer_snr_params(3, 100, 3, 5, 3)

    def call(cnt=FAKE, off=FAKE, wl=FAKE, p=good, bnd=FAKE, keep=FAKE, ws_bytes=1 << 40, batch=1, eps=0.01,
             events=None):
        args = (ctypes.byref(d), FAKE, FAKE, FAKE + 4096, 100, FAKE, batch, eps, cnt, off, wl, ctypes.byref(p),
                bnd, keep, FAKE, ws_bytes, 0)
        if events is None:
            return L.seer_layer_forward_detect(*args)
        return L.seer_layer_forward_detect_timed(*args, events)

    assert call(cnt=None) == S.SEER_EINVAL                       # the count is required
    assert call(off=None) == S.SEER_EINVAL
    assert call(wl=None) == S.SEER_EINVAL
    assert call(bnd=None) == S.SEER_EINVAL
    assert call(keep=None) == S.SEER_EINVAL
    assert call(p=S.seer_snr_params(3, 0, 3, 5, 3)) == S.SEER_EINVAL
    assert call(p=S.seer_snr_params(3, 100, 3, 5, 0)) == S.SEER_EINVAL
    assert call(batch=0) == S.SEER_EINVAL
    assert call(eps=-1.0) == S.SEER_EINVAL
    assert call(ws_bytes=S.seer_layer_workspace_bytes(d, 100) - 1) == S.SEER_EWORKSPACE
    ev = (ctypes.c_void_p * 9)(*([FAKE] * 8 + [None]))
    assert call(events=ev, batch=0) == S.SEER_EINVAL and "batch" in S.seer_last_error()   # NULL entry skipped


def test_repack_argument_errors(S):
    L = S.load_library()
    P = ctypes.c_void_p

    def call(desc, batch=4, n=1, src=FAKE, dst=FAKE * 2):
        sa = (P * max(n, 1))(*([src] * max(n, 1)))
        da = (P * max(n, 1))(*([dst] * max(n, 1)))
        return L.seer_batch_repack(ctypes.byref(desc), sa, da, n, FAKE, FAKE, FAKE, FAKE, batch, FAKE,
                                   FAKE, FAKE, None, None, 0)

    ok = dict(policy=0, tau_pad_num=1, tau_pad_den=5, granule=256, row_bytes=8192,
              dst_capacity_rows=100, max_batch_hint=0, flags=0)

    def desc(**kw):
        a = dict(ok)
        a.update(kw)
        return S.seer_repack_desc(*[a[k] for k in ("policy", "tau_pad_num", "tau_pad_den", "granule",
                                                   "row_bytes", "dst_capacity_rows", "max_batch_hint",
                                                   "flags")])

    assert call(desc(policy=3)) == S.SEER_EINVAL
    assert call(desc(tau_pad_den=0)) == S.SEER_EINVAL
    assert call(desc(granule=0)) == S.SEER_EINVAL
    assert call(desc(row_bytes=100)) == S.SEER_EINVAL
    assert call(desc(), batch=0) == S.SEER_EINVAL
    assert call(desc(), batch=5000) == S.SEER_EUNSUPPORTED
    assert call(desc(), n=0) == S.SEER_EINVAL
    assert call(desc(), n=5) == S.SEER_EINVAL
    assert call(desc(), dst=FAKE) == S.SEER_EINVAL              # src aliases dst
    assert call(desc(), src=FAKE + 8) == S.SEER_EINVAL          # misaligned


def test_cached_forward_argument_errors(S):
    L = S.load_library()
    d = dims(S)

    def call(kv=FAKE, cu_kv=FAKE, kv_rows=1000, ws_bytes=1 << 40, w=FAKE):
        return L.seer_layer_forward_cached(ctypes.byref(d), w, FAKE, FAKE + 4096, 100, FAKE, None, 1,
                                           kv, cu_kv, kv_rows, FAKE, ws_bytes, 0)

    assert call(kv=None) == S.SEER_EINVAL
    assert call(cu_kv=None) == S.SEER_EINVAL
    assert call(kv_rows=-1) == S.SEER_EINVAL
    assert call(kv=FAKE + 8) == S.SEER_EINVAL                    # misaligned cache
    assert call(kv_rows=1 << 20) == S.SEER_EUNSUPPORTED          # 2^20 * 8192 elements >= 2^32
    assert call(ws_bytes=1024) == S.SEER_EWORKSPACE
    assert call(w=None) == S.SEER_EINVAL


def test_kv_export_argument_errors(S):
    L = S.load_library()
    d = dims(S)

    def call(ws=FAKE, ws_bytes=1 << 40, rows=100, cu=FAKE, batch=1, cu_kv=FAKE, kv_rows=10, dst=FAKE):
        return L.seer_kv_export(ctypes.byref(d), ws, ws_bytes, rows, cu, batch, cu_kv, kv_rows, dst, 0)

    assert call(ws=None) == S.SEER_EINVAL
    assert call(cu=None) == S.SEER_EINVAL
    assert call(cu_kv=None) == S.SEER_EINVAL
    assert call(dst=None) == S.SEER_EINVAL
    assert call(batch=0) == S.SEER_EINVAL
    assert call(rows=0) == S.SEER_EINVAL
    assert call(kv_rows=-1) == S.SEER_EINVAL
    assert call(dst=FAKE + 4) == S.SEER_EINVAL                    # misaligned destination
    assert call(ws_bytes=1024) == S.SEER_EWORKSPACE
    assert call(ws=FAKE + 16) == S.SEER_EINVAL                    # misaligned workspace


def test_graph_argument_errors(S):
    L = S.load_library()
    g = ctypes.c_void_p(123)
    assert L.seer_graph_begin(None) == S.SEER_EINVAL
    assert "stream" in S.seer_last_error()
    assert L.seer_graph_end(FAKE, None) == S.SEER_EINVAL
    assert L.seer_graph_end(None, ctypes.byref(g)) == S.SEER_EINVAL
    assert g.value is None                      # cleared on error
    assert L.seer_graph_launch(None, FAKE) == S.SEER_EINVAL
    assert L.seer_graph_destroy(None) == S.SEER_OK


def test_graph_shapes():
    from paper_2607_14557_amd.runner import graph_shape
    g = 256
    shapes = [graph_shape(r, g) for r in range(0, 200 * g, 37)]
    assert shapes == sorted(shapes)
    assert sorted(set(s // g for s in shapes))[:9] == [1, 2, 3, 4, 6, 8, 12, 16, 24]
    for r in range(1, 200 * g, 53):
        s = graph_shape(r, g)
        assert s % g == 0 and s >= r
        assert s <= max(2 * g, 1.5 * (-(-r // g) * g))


def test_sampler_argument_errors(S):
    L = S.load_library()
    d = dims(S)
    assert S.seer_lm_head_workspace_bytes(d, 126464, 1000) >= 1000 * (126464 // 64) * 16
    pargs = lambda **kw: [kw.get(k, v) for k, v in [
        ("dims", ctypes.byref(d)), ("w", FAKE), ("vocab", 126464), ("dst", FAKE), ("dst_bytes", 1 << 40),
        ("stream", None)]]
    assert L.seer_lm_head_prepack(*pargs(w=None)) == S.SEER_EINVAL
    assert L.seer_lm_head_prepack(*pargs(dst=None)) == S.SEER_EINVAL
    assert L.seer_lm_head_prepack(*pargs(dst_bytes=126464 * 4096 * 2 - 1)) == S.SEER_EINVAL
    assert L.seer_lm_head_prepack(*pargs(vocab=1000)) == S.SEER_EUNSUPPORTED
    assert L.seer_lm_head_prepack(*pargs(vocab=524288)) == S.SEER_EUNSUPPORTED     # 4 GiB
    assert L.seer_lm_head_prepack(*pargs(dims=ctypes.byref(dims(S, d=256, h=4, dh=64, i=688, dtype=2)))) \
        == S.SEER_EUNSUPPORTED
    args = lambda **kw: [kw.get(k, v) for k, v in [
        ("dims", ctypes.byref(d)), ("w", FAKE), ("vocab", 126464), ("x", FAKE), ("rows", 100), ("cu", FAKE),
        ("batch", 1), ("pred", FAKE), ("conf", FAKE), ("ws", FAKE), ("ws_bytes", 1 << 40), ("stream", None)]]
    assert L.seer_lm_head_predict(*args(w=None)) == S.SEER_EINVAL
    assert L.seer_lm_head_predict(*args(vocab=1000)) == S.SEER_EUNSUPPORTED
    assert L.seer_lm_head_predict(*args(rows=0)) == S.SEER_EINVAL
    assert L.seer_lm_head_predict(*args(ws_bytes=16)) == S.SEER_EWORKSPACE
    assert L.seer_lm_head_predict(*args(vocab=524288)) == S.SEER_EUNSUPPORTED     # 4 GiB of head weights
    d32 = dims(S, d=256, h=4, dh=64, i=688, dtype=2)
    assert L.seer_lm_head_predict(*args(dims=ctypes.byref(d32))) == S.SEER_EUNSUPPORTED
    rargs = lambda **kw: [kw.get(k, v) for k, v in [
        ("dims", ctypes.byref(d)), ("cu", FAKE), ("used", None), ("batch", 2), ("max_used", 100), ("steps", 3),
        ("pred", FAKE), ("conf", FAKE), ("tokens", FAKE), ("x0", FAKE), ("emb", FAKE), ("vocab", 10),
        ("x_next", FAKE), ("stream", None)]]
    assert L.seer_remask_step(*rargs(tokens=None)) == S.SEER_EINVAL
    assert L.seer_remask_step(*rargs(steps=0)) == S.SEER_EINVAL
    assert L.seer_remask_step(*rargs(max_used=8193)) == S.SEER_EUNSUPPORTED
    assert L.seer_remask_step(*rargs(x0=FAKE + 8)) == S.SEER_EINVAL


def test_status_reset_argument_errors(S):
    L = S.load_library()
    assert L.seer_layer_status_reset(None, 256, 0) == S.SEER_EINVAL
    assert L.seer_layer_status_reset(FAKE + 4, 256, 0) == S.SEER_EINVAL
    assert L.seer_layer_status_reset(FAKE, 255, 0) == S.SEER_EWORKSPACE


def test_noalloc_refuses_rows_beyond_its_array(S):
    """The no-allocation layer call checks its rows bound against the 256 MiB
    in-library workspace before touching the device (the LLaDA-8B bf16 layer
    fits 2730 rows)."""
    d = dims(S)
    L = S.load_library()
    assert S.seer_layer_workspace_bytes(d, 2730) <= (256 << 20) < S.seer_layer_workspace_bytes(d, 2731)
    rc = L.seer_layer_forward_varlen_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE + 4096, 2731, FAKE, None, 1,
                                             0.0, None, None, 0)
    assert rc == S.SEER_EWORKSPACE and "2731" in S.seer_last_error()
    assert L.seer_layer_forward_varlen_noalloc(ctypes.byref(d), FAKE, FAKE, FAKE + 4096, 0, FAKE, None, 1,
                                               0.0, None, None, 0) == S.SEER_EINVAL
