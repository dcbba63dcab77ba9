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
"""
from dataclasses import dataclass
from typing import List, Optional

import torch

from . import seer as S


def dims_for(d_model, n_heads, head_dim, d_ff, dtype, rms_eps=1e-5):
    return S.seer_dims(d_model, n_heads, head_dim, d_ff,
                       S.SEER_DTYPE_BF16 if dtype == "bf16" else S.SEER_DTYPE_F32, rms_eps)


def torch_dtype(dtype):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


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
        d = dims.d_model
        self.buf = [torch.zeros(self.max_rows, d, dtype=self.dtype, device=device) for _ in range(2)]

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
                    tau_pad=(1, 5), granule=256, stream=None):
        """The kept window rows of each sequence of `src`, routed and compacted
        (no prefix rows): returns (rows, cu, seqused, route)."""
        dev = self.device
        dst = torch.empty(capacity, self.dims.d_model, dtype=self.dtype, device=dev)
        cu = torch.empty(batch + 1, dtype=torch.int32, device=dev)
        used = torch.empty(batch, dtype=torch.int32, device=dev)
        route = torch.empty(batch, 3, dtype=torch.int32, device=dev)
        desc = S.seer_repack_desc(policy, tau_pad[0], tau_pad[1], granule,
                                  self.dims.d_model * (2 if self.dtype == torch.bfloat16 else 4),
                                  capacity, 0, S.SEER_REPACK_WINDOW_ONLY)
        S.seer_batch_repack(desc, [src], [dst], cu_src, win_off, win_len, keep, batch, cu, used, route,
                            stream=stream)
        return dst, cu, used, route

    def step0(self, x_full, cu_full, win_off, win_len, batch, rows_full, l_det, act_eps,
              snr=(3, 100, 3, 5, 3), policy=S.SEER_ROUTE_HYBRID, tau_pad=(1, 5), granule=256,
              trunc_capacity=None, ctrl_host=None, stream=None):
        dev = self.device
        counts = torch.empty(rows_full, dtype=torch.int32, device=dev)
        cur = x_full
        for l in range(l_det + 1):
            nxt = self.buf[l % 2]
            self.layer(l, cur, nxt, cu_full, None, batch, rows_full,
                       act_eps=act_eps, act_count=counts if l == l_det else None, stream=stream)
            cur = nxt
        boundary = torch.empty(batch, dtype=torch.int32, device=dev)
        keep = torch.empty(batch, dtype=torch.int32, device=dev)
        S.seer_step0_detect(counts, cu_full, win_off, win_len, batch, self.dims.d_ff,
                            S.seer_snr_params(*snr), boundary, keep, stream=stream)
        cap = trunc_capacity if trunc_capacity is not None else rows_full + granule
        x_t = torch.empty(cap, self.dims.d_model, dtype=self.dtype, device=dev)
        h_t = torch.empty(cap, self.dims.d_model, dtype=self.dtype, device=dev)
        cu_t = torch.empty(batch + 1, dtype=torch.int32, device=dev)
        used = torch.empty(batch, dtype=torch.int32, device=dev)
        route = torch.empty(batch, 3, dtype=torch.int32, device=dev)
        ctrl = torch.zeros(16, dtype=torch.int32, device=dev)
        desc = S.seer_repack_desc(policy, tau_pad[0], tau_pad[1], granule,
                                  self.dims.d_model * (2 if self.dtype == torch.bfloat16 else 4),
                                  cap, 0, 0)
        S.seer_batch_repack(desc, [x_full, cur], [x_t, h_t], cu_full, win_off, win_len, keep, batch,
                            cu_t, used, route, ctrl, ctrl_host, stream=stream)
        if l_det + 1 < self.n_layers:
            h_t = self.forward(h_t, cu_t, used, batch, cap, layers=range(l_det + 1, self.n_layers),
                               out=h_t, stream=stream)
        return Step0Result(counts=counts, boundary=boundary, keep_len=keep, cu_trunc=cu_t,
                           seqused=used, route=route, ctrl=ctrl, x_trunc=x_t, h_trunc=h_t)
