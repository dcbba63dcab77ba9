"""ctypes binding of libseer.so (include/seer.h), argument marshalling only.

Every function keeps the C name and argument order.  Pointer arguments accept
a torch tensor (its data_ptr), a plain integer address or None (NULL);
``stream`` defaults to torch's current HIP stream.  A non-zero status raises
SeerError carrying the library's message.  All arithmetic of the hot path
runs inside the library's HIP kernels; nothing here computes.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libseer.so")

SEER_OK, SEER_EINVAL, SEER_EUNSUPPORTED, SEER_EWORKSPACE, SEER_EHIP = 0, -1, -2, -3, -4
SEER_DTYPE_BF16, SEER_DTYPE_F32 = 1, 2
SEER_ROUTE_HYBRID, SEER_ROUTE_NAIVE_PAD, SEER_ROUTE_VARLEN_ONLY = 0, 1, 2
SEER_PATH_STATIC, SEER_PATH_VARLEN, SEER_PATH_EAGER = 0, 1, 2
SEER_REPACK_WINDOW_ONLY = 1
SEER_STATUS_V_RANGE = 1

EXPORTED = ("seer_prepacked_bytes", "seer_prepack_weights", "seer_layer_workspace_bytes",
            "seer_layer_status_reset", "seer_layer_workspace_offsets", "seer_layer_forward_varlen",
            "seer_layer_forward_varlen_noalloc",
            "seer_layer_forward_varlen_timed", "seer_step0_detect", "seer_layer_forward_detect",
            "seer_layer_forward_detect_timed", "seer_batch_repack",
            "seer_layer_forward_cached", "seer_kv_export", "seer_graph_begin", "seer_graph_end",
            "seer_graph_launch", "seer_graph_destroy", "seer_lm_head_workspace_bytes", "seer_lm_head_prepack",
            "seer_lm_head_predict", "seer_remask_step", "seer_last_error", "seer_abi_version")


class SeerError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("seer error %d: %s" % (code, msg))
        self.code = code


class seer_dims(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float)]


class seer_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "g1", "g2")]


class seer_snr_params(ctypes.Structure):
    _fields_ = [("tau_num", ctypes.c_int32), ("tau_den", ctypes.c_int32),
                ("gamma_num", ctypes.c_int32), ("gamma_den", ctypes.c_int32),
                ("lookahead", ctypes.c_int32)]


class seer_repack_desc(ctypes.Structure):
    _fields_ = [("policy", ctypes.c_int32), ("tau_pad_num", ctypes.c_int32),
                ("tau_pad_den", ctypes.c_int32), ("granule", ctypes.c_int32),
                ("row_bytes", ctypes.c_int32), ("dst_capacity_rows", ctypes.c_int32),
                ("max_batch_hint", ctypes.c_int32), ("flags", ctypes.c_int32)]


class seer_route_ctrl(ctypes.Structure):
    _fields_ = [("total_rows", ctypes.c_int32), ("capacity_rows", ctypes.c_int32),
                ("n_static", ctypes.c_int32), ("n_varlen", ctypes.c_int32),
                ("n_eager", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("max_alloc", ctypes.c_int32), ("status", ctypes.c_int32),
                ("ready", ctypes.c_int32), ("reserved", ctypes.c_int32 * 7)]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int32


def load_library():
    """Load libseer.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    # torch first: its HIP runtime carries the same soname, so the library binds
    # to the runtime that owns torch's streams and allocations.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libseer.so is not built (%s); run `python -m paper_2607_14557_amd.build`"
                           % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    L.seer_prepacked_bytes.argtypes = [ctypes.POINTER(seer_dims)]
    L.seer_prepacked_bytes.restype = ctypes.c_size_t
    L.seer_prepack_weights.argtypes = [ctypes.POINTER(seer_dims), ctypes.POINTER(seer_layer_weights),
                                       _P, ctypes.c_size_t, _P]
    L.seer_prepack_weights.restype = ctypes.c_int
    L.seer_layer_workspace_bytes.argtypes = [ctypes.POINTER(seer_dims), _I]
    L.seer_layer_workspace_bytes.restype = ctypes.c_size_t
    L.seer_layer_status_reset.argtypes = [_P, ctypes.c_size_t, _P]
    L.seer_layer_status_reset.restype = ctypes.c_int
    L.seer_layer_workspace_offsets.argtypes = [ctypes.POINTER(seer_dims), _I,
                                               ctypes.POINTER(ctypes.c_size_t)]
    L.seer_layer_workspace_offsets.restype = ctypes.c_int
    L.seer_layer_forward_varlen.argtypes = [ctypes.POINTER(seer_dims), _P, _P, _P, _I, _P, _P, _I,
                                            ctypes.c_float, _P, _P, ctypes.c_size_t, _P]
    L.seer_layer_forward_varlen.restype = ctypes.c_int
    L.seer_layer_forward_varlen_noalloc.argtypes = [ctypes.POINTER(seer_dims), _P, _P, _P, _I, _P, _P, _I,
                                                    ctypes.c_float, _P, _P, _P]
    L.seer_layer_forward_varlen_noalloc.restype = ctypes.c_int
    L.seer_layer_forward_varlen_timed.argtypes = L.seer_layer_forward_varlen.argtypes + [
        ctypes.POINTER(_P)]
    L.seer_layer_forward_varlen_timed.restype = ctypes.c_int
    L.seer_step0_detect.argtypes = [_P, _P, _P, _P, _I, _I, ctypes.POINTER(seer_snr_params), _P, _P, _P]
    L.seer_step0_detect.restype = ctypes.c_int
    L.seer_layer_forward_detect.argtypes = [ctypes.POINTER(seer_dims), _P, _P, _P, _I, _P, _I, ctypes.c_float,
                                            _P, _P, _P, ctypes.POINTER(seer_snr_params), _P, _P, _P,
                                            ctypes.c_size_t, _P]
    L.seer_layer_forward_detect.restype = ctypes.c_int
    L.seer_layer_forward_detect_timed.argtypes = L.seer_layer_forward_detect.argtypes + [ctypes.POINTER(_P)]
    L.seer_layer_forward_detect_timed.restype = ctypes.c_int
    L.seer_batch_repack.argtypes = [ctypes.POINTER(seer_repack_desc), ctypes.POINTER(_P),
                                    ctypes.POINTER(_P), _I, _P, _P, _P, _P, _I, _P, _P, _P, _P, _P, _P]
    L.seer_batch_repack.restype = ctypes.c_int
    L.seer_layer_forward_cached.argtypes = [ctypes.POINTER(seer_dims), _P, _P, _P, _I, _P, _P, _I,
                                            _P, _P, _I, _P, ctypes.c_size_t, _P]
    L.seer_layer_forward_cached.restype = ctypes.c_int
    L.seer_kv_export.argtypes = [ctypes.POINTER(seer_dims), _P, ctypes.c_size_t, _I, _P, _I, _P, _I, _P, _P]
    L.seer_kv_export.restype = ctypes.c_int
    L.seer_lm_head_workspace_bytes.argtypes = [ctypes.POINTER(seer_dims), _I, _I]
    L.seer_lm_head_workspace_bytes.restype = ctypes.c_size_t
    L.seer_lm_head_prepack.argtypes = [ctypes.POINTER(seer_dims), _P, _I, _P, ctypes.c_size_t, _P]
    L.seer_lm_head_prepack.restype = ctypes.c_int
    L.seer_lm_head_predict.argtypes = [ctypes.POINTER(seer_dims), _P, _I, _P, _I, _P, _I, _P, _P, _P,
                                       ctypes.c_size_t, _P]
    L.seer_lm_head_predict.restype = ctypes.c_int
    L.seer_remask_step.argtypes = [ctypes.POINTER(seer_dims), _P, _P, _I, _I, _I, _P, _P, _P, _P, _P, _I, _P, _P]
    L.seer_remask_step.restype = ctypes.c_int
    L.seer_graph_begin.argtypes = [_P]
    L.seer_graph_begin.restype = ctypes.c_int
    L.seer_graph_end.argtypes = [_P, ctypes.POINTER(_P)]
    L.seer_graph_end.restype = ctypes.c_int
    L.seer_graph_launch.argtypes = [_P, _P]
    L.seer_graph_launch.restype = ctypes.c_int
    L.seer_graph_destroy.argtypes = [_P]
    L.seer_graph_destroy.restype = ctypes.c_int
    L.seer_last_error.argtypes = []
    L.seer_last_error.restype = ctypes.c_char_p
    L.seer_abi_version.argtypes = []
    L.seer_abi_version.restype = ctypes.c_int32
    _lib = L
    return L


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(rc):
    if rc != 0:
        raise SeerError(rc, load_library().seer_last_error().decode())


def seer_last_error():
    return load_library().seer_last_error().decode()


def seer_abi_version():
    return load_library().seer_abi_version()


def seer_prepacked_bytes(dims):
    return load_library().seer_prepacked_bytes(ctypes.byref(dims))


def seer_prepack_weights(dims, weights, dst, dst_bytes=None, stream=None):
    """weights: dict with wq wk wv wo wg wu wd (device tensors) and optional g1 g2."""
    w = seer_layer_weights(*[_ptr(weights.get(n)) for n in
                             ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "g1", "g2")])
    nbytes = dst_bytes if dst_bytes is not None else dst.numel() * dst.element_size()
    _check(load_library().seer_prepack_weights(ctypes.byref(dims), ctypes.byref(w), _ptr(dst),
                                               nbytes, _stream(stream)))


def seer_layer_workspace_bytes(dims, max_rows):
    return load_library().seer_layer_workspace_bytes(ctypes.byref(dims), int(max_rows))


def seer_layer_status_reset(workspace, workspace_bytes=None, stream=None):
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    _check(load_library().seer_layer_status_reset(_ptr(workspace), nbytes, _stream(stream)))


def seer_layer_workspace_offsets(dims, max_rows):
    """Returns the eight byte offsets as a list."""
    off = (ctypes.c_size_t * 8)()
    _check(load_library().seer_layer_workspace_offsets(ctypes.byref(dims), int(max_rows), off))
    return list(off)


def seer_layer_forward_varlen_noalloc(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused,
                                      batch, act_eps, act_count, status=None, stream=None):
    _check(load_library().seer_layer_forward_varlen_noalloc(
        ctypes.byref(dims), _ptr(w_packed), _ptr(x_in), _ptr(x_out), int(total_rows_ub), _ptr(cu_seqlens),
        _ptr(seqused), int(batch), float(act_eps), _ptr(act_count), _ptr(status), _stream(stream)))


def seer_layer_forward_varlen(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused,
                              batch, act_eps, act_count, workspace, workspace_bytes=None,
                              stream=None):
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    _check(load_library().seer_layer_forward_varlen(
        ctypes.byref(dims), _ptr(w_packed), _ptr(x_in), _ptr(x_out), int(total_rows_ub),
        _ptr(cu_seqlens), _ptr(seqused), int(batch), float(act_eps), _ptr(act_count),
        _ptr(workspace), nbytes, _stream(stream)))


def seer_layer_forward_varlen_timed(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens,
                                    seqused, batch, act_eps, act_count, workspace, events,
                                    workspace_bytes=None, stream=None):
    """events: sequence of 8 raw hipEvent_t handles (ints); a None entry
    skips that point."""
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    ev = (_P * 8)(*events)
    _check(load_library().seer_layer_forward_varlen_timed(
        ctypes.byref(dims), _ptr(w_packed), _ptr(x_in), _ptr(x_out), int(total_rows_ub),
        _ptr(cu_seqlens), _ptr(seqused), int(batch), float(act_eps), _ptr(act_count),
        _ptr(workspace), nbytes, _stream(stream), ev))


def seer_layer_forward_cached(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, seqused, batch,
                              kv_cache, cu_kv, kv_rows_ub, workspace, workspace_bytes=None, stream=None):
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    _check(load_library().seer_layer_forward_cached(
        ctypes.byref(dims), _ptr(w_packed), _ptr(x_in), _ptr(x_out), int(total_rows_ub),
        _ptr(cu_seqlens), _ptr(seqused), int(batch), _ptr(kv_cache), _ptr(cu_kv), int(kv_rows_ub),
        _ptr(workspace), nbytes, _stream(stream)))


def seer_kv_export(dims, workspace, total_rows_ub, cu_seqlens, batch, cu_kv, kv_rows_ub, kv_dst,
                   workspace_bytes=None, stream=None):
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    _check(load_library().seer_kv_export(
        ctypes.byref(dims), _ptr(workspace), nbytes, int(total_rows_ub), _ptr(cu_seqlens), int(batch),
        _ptr(cu_kv), int(kv_rows_ub), _ptr(kv_dst), _stream(stream)))


def seer_step0_detect(act_count, cu_seqlens, win_off, win_len, batch, d_ff, params, boundary,
                      keep_len, stream=None):
    _check(load_library().seer_step0_detect(
        _ptr(act_count), _ptr(cu_seqlens), _ptr(win_off), _ptr(win_len), int(batch), int(d_ff),
        ctypes.byref(params), _ptr(boundary), _ptr(keep_len), _stream(stream)))


def seer_layer_forward_detect(dims, w_packed, x_in, x_out, total_rows_ub, cu_seqlens, batch, act_eps,
                              act_count, win_off, win_len, params, boundary, keep_len, workspace,
                              workspace_bytes=None, stream=None, events=None):
    """The detection layer; with events (9 raw hipEvent_t handles) the timed
    variant."""
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    args = [ctypes.byref(dims), _ptr(w_packed), _ptr(x_in), _ptr(x_out), int(total_rows_ub), _ptr(cu_seqlens),
            int(batch), float(act_eps), _ptr(act_count), _ptr(win_off), _ptr(win_len), ctypes.byref(params),
            _ptr(boundary), _ptr(keep_len), _ptr(workspace), nbytes, _stream(stream)]
    L = load_library()
    if events is None:
        _check(L.seer_layer_forward_detect(*args))
    else:
        _check(L.seer_layer_forward_detect_timed(*args, (_P * 9)(*events)))


def seer_batch_repack(desc, srcs, dsts, cu_src, win_off, win_len, keep_len, batch, cu_dst,
                      seqused, route, ctrl_dev=None, ctrl_host=None, stream=None):
    n = len(srcs)
    src_arr = (_P * n)(*[_ptr(s) for s in srcs])
    dst_arr = (_P * n)(*[_ptr(d) for d in dsts])
    _check(load_library().seer_batch_repack(
        ctypes.byref(desc), src_arr, dst_arr, n, _ptr(cu_src), _ptr(win_off), _ptr(win_len),
        _ptr(keep_len), int(batch), _ptr(cu_dst), _ptr(seqused), _ptr(route), _ptr(ctrl_dev),
        _ptr(ctrl_host), _stream(stream)))


def seer_graph_begin(stream):
    """Start recording the seer calls issued on `stream` (a created stream)."""
    _check(load_library().seer_graph_begin(_stream(stream)))


def seer_graph_end(stream):
    """End the recording; returns the graph handle (an int)."""
    g = _P()
    _check(load_library().seer_graph_end(_stream(stream), ctypes.byref(g)))
    return g.value


def seer_graph_launch(graph, stream=None):
    _check(load_library().seer_graph_launch(graph, _stream(stream)))


def seer_graph_destroy(graph):
    _check(load_library().seer_graph_destroy(graph))


def seer_lm_head_workspace_bytes(dims, vocab, rows_ub):
    return load_library().seer_lm_head_workspace_bytes(ctypes.byref(dims), int(vocab), int(rows_ub))


def seer_lm_head_prepack(dims, w_lm, vocab, dst, dst_bytes=None, stream=None):
    nbytes = dst_bytes if dst_bytes is not None else dst.numel() * dst.element_size()
    _check(load_library().seer_lm_head_prepack(ctypes.byref(dims), _ptr(w_lm), int(vocab), _ptr(dst), nbytes,
                                               _stream(stream)))


def seer_lm_head_predict(dims, w_packed, vocab, x, rows_ub, cu_seqlens, batch, pred, conf, workspace,
                         workspace_bytes=None, stream=None):
    nbytes = workspace_bytes if workspace_bytes is not None else workspace.numel() * workspace.element_size()
    _check(load_library().seer_lm_head_predict(
        ctypes.byref(dims), _ptr(w_packed), int(vocab), _ptr(x), int(rows_ub), _ptr(cu_seqlens), int(batch),
        _ptr(pred), _ptr(conf), _ptr(workspace), nbytes, _stream(stream)))


def seer_remask_step(dims, cu_seqlens, seqused, batch, max_used, steps_left, pred, conf, tokens, x0, emb, vocab,
                     x_next, stream=None):
    _check(load_library().seer_remask_step(
        ctypes.byref(dims), _ptr(cu_seqlens), _ptr(seqused), int(batch), int(max_used), int(steps_left),
        _ptr(pred), _ptr(conf), _ptr(tokens), _ptr(x0), _ptr(emb), int(vocab), _ptr(x_next), _stream(stream)))
