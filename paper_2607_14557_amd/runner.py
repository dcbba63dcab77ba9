"""Sequencing of the C-ABI calls for the whole Seer path on one GPU.

Device memory comes from torch (plumbing only); every step of the path --
layer forwards, the fused near-zero count, the SNR scan, routing and
compaction -- is one of libseer's entry points.  The step-0 pipeline follows
the method's order (Sec. 3.2-3.5): layers 0..l_det on the full window with
the count at l_det, boundary detection, route + compaction of the in-flight
residual and of the step-input embeddings in one launch, then the remaining
layers on the compacted batch.  Later denoising steps run every layer on the
compacted batch, or, with the prefix keys/values cached (Appendix D), on the
kept window rows alone.

Graph-compatible execution (Sec. 3.5): every kernel reads its row counts from
device memory, so one recorded launch sequence (a HIP graph, recorded through
the library's seer_graph_* calls) serves any batch whose routed capacity fits
the rows bound it was recorded with.  The repack kernel writes the routed
shape to pinned host memory; the host polls that word, without waiting on the
stream, to pick the recorded sequence for the capacity.
"""
import time
from dataclasses import dataclass
from typing import Dict, List, Optional

import torch

from . import seer as S


def dims_for(d_model, n_heads, head_dim, d_ff, dtype, rms_eps=1e-5, rope_theta=0.0):
    return S.seer_dims(d_model, n_heads, head_dim, d_ff,
                       S.SEER_DTYPE_BF16 if dtype == "bf16" else S.SEER_DTYPE_F32, rms_eps, rope_theta)


def torch_dtype(dtype):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


CTRL_FIELDS = ("total_rows", "capacity_rows", "n_static", "n_varlen", "n_eager", "n_groups", "max_alloc",
               "status", "ready")


def pinned_ctrl():
    """A host-pinned control word (16 int32) for seer_batch_repack."""
    return torch.zeros(16, dtype=torch.int32, pin_memory=True)


def poll_ctrl(ctrl_host, timeout_s=30.0):
    """Spin on the pinned control word until the repack kernel has written it
    (its ready field is stored last), without synchronising any stream.
    Returns the fields as a dict.  The caller clears `ready` (ctrl_host[8] = 0)
    before enqueuing the repack."""
    a = ctrl_host.numpy()
    t_end = time.monotonic() + timeout_s
    spins = 0
    while int(a[8]) != 1:
        spins += 1
        if spins > 1000:
            time.sleep(5e-5)           # past the first ~100 us, yield the core between reads
        if time.monotonic() > t_end:
            raise TimeoutError("control word not written within %.0f s" % timeout_s)
    v = [int(a[i]) for i in range(9)]
    return dict(zip(CTRL_FIELDS, v))


def graph_shape(rows, granule=256):
    """The 1-D graph shape for a routed capacity: the smallest of granule x
    {1, 2, 3, 4, 6, 8, 12, 16, ...} (at most 1.5x over) that holds `rows`."""
    units = max(1, -(-int(rows) // granule))
    u = 1
    while u < units:
        if u >= 2 and u & (u - 1) == 0:
            u += u // 2            # 2^k -> 1.5 x 2^k
        elif u % 3 == 0:
            u = u // 3 * 4         # 1.5 x 2^k -> 2^(k+1)
        else:
            u = 2 * u
    return u * granule


class SeerGraph:
    """A recorded launch sequence; replay() runs it on a stream."""

    def __init__(self, handle):
        self.handle = handle

    def replay(self, stream=None):
        S.seer_graph_launch(self.handle, stream=stream)

    def close(self):
        if self.handle:
            S.seer_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def record(fn, stream):
    """Record the seer calls fn() issues on `stream` (a created torch stream;
    fn must issue nothing else on it) into a SeerGraph."""
    S.seer_graph_begin(stream)
    try:
        fn()
    except BaseException:
        # close the recording, drop what it holds, and report fn's error
        try:
            S.seer_graph_destroy(S.seer_graph_end(stream))
        except S.SeerError:
            pass
        raise
    return SeerGraph(S.seer_graph_end(stream))


@dataclass
class Step0Result:
    counts: torch.Tensor        # [rows_full] int32 at the detection layer
    boundary: torch.Tensor      # [B] int32
    keep_len: torch.Tensor      # [B] int32
    cu_trunc: torch.Tensor      # [B+1] int32
    seqused: torch.Tensor       # [B] int32
    route: torch.Tensor         # [B, 3] int32
    ctrl: torch.Tensor          # [16] int32 (device copy of the control word)
    x_trunc: torch.Tensor       # compacted step-input embeddings
    h_trunc: torch.Tensor       # step-0 residual after the last layer (compacted)
    routed: Optional[dict] = None   # the control word read from pinned memory (if polled)
    rows_ub: int = 0            # rows bound the layers after the repack ran with


class StepGraphs:
    """Recorded denoising steps, one per 1-D graph shape (Sec. 3.5).

    step_fn(rows_ub) issues one step's seer calls on `stream`, on buffers that
    stay fixed for the life of this object; run(capacity_rows) replays the
    recording for graph_shape(capacity_rows) (recorded on first use)."""

    def __init__(self, step_fn, stream, max_rows, granule=256):
        self.step_fn = step_fn
        self.stream = stream
        self.max_rows = int(max_rows)
        self.granule = granule
        self.graphs: Dict[int, SeerGraph] = {}

    def shape(self, capacity_rows):
        return min(graph_shape(capacity_rows, self.granule), self.max_rows)

    def run(self, capacity_rows):
        rows = self.shape(capacity_rows)
        g = self.graphs.get(rows)
        if g is None:
            g = record(lambda: self.step_fn(rows), self.stream)
            self.graphs[rows] = g
        g.replay(self.stream)
        return rows

    def close(self):
        for g in self.graphs.values():
            g.close()
        self.graphs.clear()


class SyntheticSampler:
    """LM head and low-confidence remasking between denoising steps, on
    window-only rows (the layout of the cached-prefix steps): after a step,
    every masked window position gets a prediction and a confidence, the most
    confident are committed, and the next step's input rows are rebuilt from
    the committed tokens' embeddings (uncommitted rows keep their step-0
    input).  Token state: tokens[r] == -1 while masked."""

    def __init__(self, dims, w_lm, emb, rows_ub, device="cuda"):
        self.dims = dims
        self.emb = emb
        self.vocab = int(w_lm.shape[0])
        self.rows_ub = int(rows_ub)
        # the head weight in the matrix cores' operand order (the row-major
        # w_lm is not kept)
        self.w_packed = torch.empty(w_lm.numel() * 2, dtype=torch.uint8, device=device)
        S.seer_lm_head_prepack(dims, w_lm, self.vocab, self.w_packed)
        torch.cuda.current_stream(self.w_packed.device).synchronize()   # later calls may use other streams
        self.ws_bytes = S.seer_lm_head_workspace_bytes(dims, self.vocab, self.rows_ub)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.pred = torch.empty(self.rows_ub, dtype=torch.int32, device=device)
        self.conf = torch.empty(self.rows_ub, dtype=torch.float32, device=device)
        self.tokens = torch.full((self.rows_ub,), -1, dtype=torch.int32, device=device)

    def reset(self):
        self.tokens.fill_(-1)

    def predict(self, h, cu, batch, rows_ub, stream=None):
        S.seer_lm_head_predict(self.dims, self.w_packed, self.vocab, h, rows_ub, cu, batch, self.pred, self.conf,
                               self.workspace, self.ws_bytes, stream=stream)

    def step(self, h, cu, used, batch, rows_ub, x0, x_next, steps_left, max_used, stream=None):
        """Predict on the step's output rows h, commit, write the next inputs."""
        self.predict(h, cu, batch, rows_ub, stream=stream)
        S.seer_remask_step(self.dims, cu, used, batch, max_used, steps_left, self.pred, self.conf, self.tokens,
                           x0, self.emb, self.vocab, x_next, stream=stream)


class SeerStack:
    """A stack of prepacked layers plus the scratch the ABI calls need."""

    def __init__(self, dims, n_layers, max_rows, device="cuda"):
        S.load_library()
        self.dims = dims
        self.n_layers = n_layers
        self.max_rows = int(max_rows)
        self.device = device
        self.dtype = torch.bfloat16 if dims.dtype == S.SEER_DTYPE_BF16 else torch.float32
        self.packed_bytes = S.seer_prepacked_bytes(dims)
        if self.packed_bytes == 0:
            raise S.SeerError(S.SEER_EUNSUPPORTED, S.seer_last_error())
        self.packed: List[Optional[torch.Tensor]] = [None] * n_layers
        self.ws_bytes = S.seer_layer_workspace_bytes(dims, self.max_rows)
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        S.seer_layer_status_reset(self.workspace, self.ws_bytes)
        d = dims.d_model
        self.buf = [torch.zeros(self.max_rows, d, dtype=self.dtype, device=device) for _ in range(2)]
        self._trunc_bufs = {}

    def layer_status(self, stream=None):
        """The workspace status word (SEER_STATUS_* bits accumulated by every
        layer call since construction or the last reset); waits for `stream`."""
        (stream or torch.cuda.current_stream(self.workspace.device)).synchronize()
        return int(self.workspace[:4].view(torch.int32).item())

    def check_status(self, stream=None):
        """Raise SeerError if a layer call reported a value out of range."""
        st = self.layer_status(stream)
        if st & S.SEER_STATUS_V_RANGE:
            raise S.SeerError(S.SEER_EUNSUPPORTED, "an attention value exceeded the fp16 range (|v| > 65504)")

    def reset_status(self, stream=None):
        S.seer_layer_status_reset(self.workspace, self.ws_bytes, stream=stream)

    def set_layer(self, l, weights, stream=None):
        if self.packed[l] is None:
            self.packed[l] = torch.empty(self.packed_bytes, dtype=torch.uint8, device=self.device)
        S.seer_prepack_weights(self.dims, weights, self.packed[l], stream=stream)

    def layer(self, l, x_in, x_out, cu, seqused, batch, rows_ub, act_eps=0.0, act_count=None,
              stream=None):
        S.seer_layer_forward_varlen(self.dims, self.packed[l], x_in, x_out, rows_ub, cu, seqused,
                                    batch, act_eps, act_count, self.workspace, self.ws_bytes,
                                    stream=stream)

    def forward(self, x, cu, seqused, batch, rows_ub, layers=None, out=None, stream=None):
        """Run layers (default all) over x; returns the output tensor."""
        layers = range(self.n_layers) if layers is None else layers
        cur = x
        for i, l in enumerate(layers):
            nxt = self.buf[i % 2] if cur is not self.buf[i % 2] else self.buf[(i + 1) % 2]
            self.layer(l, cur, nxt, cu, seqused, batch, rows_ub, stream=stream)
            cur = nxt
        if out is not None and cur is not out:
            out[:rows_ub].copy_(cur[:rows_ub])
            cur = out
        return cur

    # ---- truncated steps with the prefix keys/values cached (Appendix D) ----
    def alloc_kv_caches(self, kv_rows):
        """One [kv_rows, 2 d] cache per layer (K | V, the qkv element types)."""
        return [torch.empty(max(int(kv_rows), 1), 2 * self.dims.d_model, dtype=self.dtype,
                            device=self.device) for _ in range(self.n_layers)]

    def forward_export(self, x, cu, seqused, batch, rows_ub, caches, cu_kv, kv_rows_ub, out=None,
                       stream=None):
        """A full truncated step over [prefix; kept window] rows that also
        caches, per layer, the K | V of each sequence's first cu_kv[b+1] - cu_kv[b]
        rows."""
        cur = x
        for l in range(self.n_layers):
            nxt = self.buf[l % 2] if cur is not self.buf[l % 2] else self.buf[(l + 1) % 2]
            self.layer(l, cur, nxt, cu, seqused, batch, rows_ub, stream=stream)
            S.seer_kv_export(self.dims, self.workspace, rows_ub, cu, batch, cu_kv, kv_rows_ub, caches[l],
                             workspace_bytes=self.ws_bytes, stream=stream)
            cur = nxt
        if out is not None and cur is not out:
            out[:rows_ub].copy_(cur[:rows_ub])
            cur = out
        return cur

    def forward_cached(self, x_w, cu_w, used_w, batch, rows_ub, caches, cu_kv, kv_rows_ub, out=None,
                       stream=None):
        """A truncated step on the kept window rows only, every layer reading
        its cached prefix keys/values."""
        cur = x_w
        for l in range(self.n_layers):
            nxt = self.buf[l % 2] if cur is not self.buf[l % 2] else self.buf[(l + 1) % 2]
            S.seer_layer_forward_cached(self.dims, self.packed[l], cur, nxt, rows_ub, cu_w, used_w, batch,
                                        caches[l], cu_kv, kv_rows_ub, self.workspace, self.ws_bytes,
                                        stream=stream)
            cur = nxt
        if out is not None and cur is not out:
            out[:rows_ub].copy_(cur[:rows_ub])
            cur = out
        return cur

    def window_rows(self, src, cu_src, win_off, win_len, keep, batch, capacity, policy=S.SEER_ROUTE_HYBRID,
                    tau_pad=(1, 5), granule=256, ctrl_host=None, stream=None):
        """The kept window rows of each sequence of `src`, routed and compacted
        (no prefix rows): returns (rows, cu, seqused, route).  The buffers are
        owned by the stack and reused by the next call of the same shape.  With
        ctrl_host (pinned_ctrl()), the routed shape is also written there for
        poll_ctrl; its ready field is cleared here before the launch."""
        dev = self.device
        key = ("win", capacity, batch)
        if key not in self._trunc_bufs:
            self._trunc_bufs[key] = (
                torch.empty(capacity, self.dims.d_model, dtype=self.dtype, device=dev),
                torch.empty(batch + 1, dtype=torch.int32, device=dev),
                torch.empty(batch, dtype=torch.int32, device=dev),
                torch.empty(batch, 3, dtype=torch.int32, device=dev))
        dst, cu, used, route = self._trunc_bufs[key]
        desc = S.seer_repack_desc(policy, tau_pad[0], tau_pad[1], granule,
                                  self.dims.d_model * (2 if self.dtype == torch.bfloat16 else 4),
                                  capacity, 0, S.SEER_REPACK_WINDOW_ONLY)
        if ctrl_host is not None:
            ctrl_host[8] = 0
        S.seer_batch_repack(desc, [src], [dst], cu_src, win_off, win_len, keep, batch, cu, used, route,
                            ctrl_host=ctrl_host, stream=stream)
        return dst, cu, used, route

    def step0(self, x_full, cu_full, win_off, win_len, batch, rows_full, l_det, act_eps,
              snr=(3, 100, 3, 5, 3), policy=S.SEER_ROUTE_HYBRID, tau_pad=(1, 5), granule=256,
              trunc_capacity=None, ctrl_host=None, check_status=True, stream=None):
        """Step 0 (Sec. 3.2-3.5): layers 0..l_det on the full window with the
        near-zero count at l_det and the SNR scan inside that layer (whose
        down projection then runs on the kept rows only), routing +
        compaction of the step-input embeddings and the in-flight residual,
        then the remaining layers on the compacted batch.

        trunc_capacity: rows of the compacted buffers.  By default the worst
        case of the routing: every window padded to the longest one,
        sum(win_off) + batch * max(win_len) rounded up to the granule (read
        from the device once).  A routed batch that does not fit is reported
        by the repack kernel in the control word; with ctrl_host it is read
        from the polled word, otherwise (check_status) from the device copy,
        and SeerError is raised before any later layer runs; that check also
        reads the workspace status word (check_status()).  The polled path
        never waits on the stream: its caller checks the status word when it
        syncs."""
        dev = self.device
        if trunc_capacity is None:
            wo = win_off[:batch].cpu().to(torch.int64)
            wl_ = win_len[:batch].cpu().to(torch.int64)
            worst = int(wo.sum()) + batch * int(wl_.max()) if batch > 0 else 0
            trunc_capacity = max(granule, -(-worst // granule) * granule)
        counts = torch.empty(rows_full, dtype=torch.int32, device=dev)
        cur = x_full
        for l in range(l_det):
            nxt = self.buf[l % 2]
            self.layer(l, cur, nxt, cu_full, None, batch, rows_full, stream=stream)
            cur = nxt
        cap = trunc_capacity
        key = (cap, batch)
        if key not in self._trunc_bufs:
            # compacted buffers, reused by every step0 call of this shape so that
            # recorded truncated steps keep valid addresses
            d = self.dims.d_model
            self._trunc_bufs[key] = dict(
                boundary=torch.empty(batch, dtype=torch.int32, device=dev),
                keep=torch.empty(batch, dtype=torch.int32, device=dev),
                x_t=torch.empty(cap, d, dtype=self.dtype, device=dev),
                h_t=torch.empty(cap, d, dtype=self.dtype, device=dev),
                cu_t=torch.empty(batch + 1, dtype=torch.int32, device=dev),
                used=torch.empty(batch, dtype=torch.int32, device=dev),
                route=torch.empty(batch, 3, dtype=torch.int32, device=dev),
                ctrl=torch.zeros(16, dtype=torch.int32, device=dev))
        tb = self._trunc_bufs[key]
        boundary, keep, x_t, h_t = tb["boundary"], tb["keep"], tb["x_t"], tb["h_t"]
        cu_t, used, route, ctrl = tb["cu_t"], tb["used"], tb["route"], tb["ctrl"]
        # the detection layer: count, scan, and its down projection on the kept rows only
        nxt = self.buf[l_det % 2]
        S.seer_layer_forward_detect(self.dims, self.packed[l_det], cur, nxt, rows_full, cu_full, batch, act_eps,
                                    counts, win_off, win_len, S.seer_snr_params(*snr), boundary, keep,
                                    self.workspace, self.ws_bytes, stream=stream)
        cur = nxt
        desc = S.seer_repack_desc(policy, tau_pad[0], tau_pad[1], granule,
                                  self.dims.d_model * (2 if self.dtype == torch.bfloat16 else 4),
                                  cap, 0, 0)
        if ctrl_host is not None:
            ctrl_host[8] = 0
        S.seer_batch_repack(desc, [x_full, cur], [x_t, h_t], cu_full, win_off, win_len, keep, batch,
                            cu_t, used, route, ctrl, ctrl_host, stream=stream)
        routed = None
        rows_ub = cap
        if ctrl_host is not None:
            # the routed capacity sizes the remaining launches (no stream sync)
            routed = poll_ctrl(ctrl_host)
            if routed["status"] != 0:
                raise S.SeerError(routed["status"], "compacted batch exceeds the %d-row buffers" % cap)
            rows_ub = max(1, min(cap, routed["capacity_rows"]))
        elif check_status:
            (stream or torch.cuda.current_stream(ctrl.device)).synchronize()   # the repack has written it
            status = int(ctrl[7].item())
            if status != 0:
                raise S.SeerError(status, "compacted batch exceeds the %d-row buffers" % cap)
            self.check_status(stream)           # the step-0 layers so far kept V in range
        if l_det + 1 < self.n_layers:
            h_t = self.forward(h_t, cu_t, used, batch, rows_ub, layers=range(l_det + 1, self.n_layers),
                               out=h_t, stream=stream)
        return Step0Result(counts=counts, boundary=boundary, keep_len=keep, cu_trunc=cu_t,
                           seqused=used, route=route, ctrl=ctrl, x_trunc=x_t, h_trunc=h_t,
                           routed=routed, rows_ub=rows_ub)
