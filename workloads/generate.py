"""Seeded synthetic inputs for the Seer hot path.

Everything here is input construction: random weights, prefix / prompt /
content embeddings, the planted end-of-sequence (EOS) suffix and the planted
boundary positions.  None of the method's arithmetic (normalisation,
attention, SwiGLU, the sparsity count, the SNR criterion, routing) lives here;
the oracle and the GPU path each implement that on their own and both consume
the arrays produced here.

Recipe (one base seed per workload, split into independent streams):
  * weights ~ N(0, 0.02^2) per layer, rounded to the workload dtype; norm gains 1;
  * visual prefix and prompt rows ~ N(0, 1);
  * window positions before the planted boundary b ~ N(0, 1) per element;
  * window positions >= b: one shared EOS vector plus N(0, 0.01^2) noise;
  * planted b fixed, log-uniform (b = round(exp(U(ln lo, ln hi)))) or uniform
    integer in [lo, hi] per sequence;
  * optional confounders (sweep workloads): up to n runs per sequence of
    1..r content positions replaced by EOS rows (same vector and noise),
    starting at position >= 1 and ending >= 2 positions before b, disjoint.

The shared EOS vector is e = A * sqrt(d) * v, where v is the unit eigenvector of
the smallest eigenvalue of Wg^T Wg + Wu^T Wu of the detection layer, summed over
several layers for the sweep workloads (the input direction the SwiGLU
amplifies least), with the sign fixed so that its largest
magnitude component is positive.  With random weights every other input
direction has the same expected activation statistics, so a generic EOS vector
plants no boundary; the least-amplified direction makes the suffix rows'
activations cluster near zero, which is the behaviour the method relies on for
padding tokens (Sec. 1 and Sec. 3.2).
"""
from dataclasses import dataclass
from typing import List, Optional, Tuple

import numpy as np

from .configs import Workload

WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def round_to_dtype(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round float values to the workload dtype, returned as float32 (exact)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    if dtype != "bf16":
        raise ValueError(dtype)
    import torch
    return torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()


def weight_shapes(w: Workload):
    d, i = w.shape.d_model, w.shape.d_ff
    return {"wq": (d, d), "wk": (d, d), "wv": (d, d), "wo": (d, d),
            "wg": (i, d), "wu": (i, d), "wd": (d, i)}


def _streams(w: Workload):
    ss = np.random.SeedSequence(w.seed)
    kids = ss.spawn(7)
    return {"weights": kids[0], "boundary": kids[1], "visual": kids[2],
            "prompt": kids[3], "content": kids[4], "noise": kids[5], "dips": kids[6]}


def layer_weights(w: Workload, layer: int) -> dict:
    """float32 arrays (values representable in the workload dtype), [out, in] layout."""
    wss = _streams(w)["weights"].spawn(w.n_layers)[layer]
    rng = np.random.default_rng(wss)
    out = {}
    for name, shp in weight_shapes(w).items():
        a = rng.standard_normal(shp, dtype=np.float32)
        a *= np.float32(w.weight_std)
        out[name] = round_to_dtype(a, w.dtype)
    d = w.shape.d_model
    out["g1"] = np.ones(d, np.float32)
    out["g2"] = np.ones(d, np.float32)
    return out


def layer_weights_torch(w: Workload, layer: int, device):
    """Device-side weights for the deep stacks, drawn by torch's generator.

    Drawing 32 LLaDA-sized layers on the host takes minutes, so the stacked
    workloads take their weights from torch's device generator instead.  These
    are inputs only; the oracle reads the same tensors back for its checks.
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(w.seed) * 1000 + layer)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    out = {}
    for name, shp in weight_shapes(w).items():
        t = torch.empty(shp, device=device, dtype=torch.float32)
        t.normal_(0.0, w.weight_std, generator=gen)
        out[name] = t.to(dt)
    d = w.shape.d_model
    out["g1"] = torch.ones(d, device=device, dtype=torch.float32)
    out["g2"] = torch.ones(d, device=device, dtype=torch.float32)
    return out


def gate_up_gram(wg: np.ndarray, wu: np.ndarray) -> np.ndarray:
    g = wg.astype(np.float64)
    u = wu.astype(np.float64)
    return g.T @ g + u.T @ u


def lm_head_torch(w: Workload, vocab: int, device, seed_offset: int = 0):
    """Synthetic LM head [vocab, d] and token embedding table [vocab, d] (bf16
    on the device): head ~ N(0, weight_std^2), embeddings ~ N(0, 1) like the
    content rows.  Inputs only; drawn by torch's device generator."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(w.seed) * 1000 + 997 + seed_offset)
    d = w.shape.d_model
    head = torch.empty(vocab, d, device=device, dtype=torch.float32).normal_(0.0, w.weight_std, generator=gen)
    emb = torch.empty(vocab, d, device=device, dtype=torch.float32).normal_(0.0, 1.0, generator=gen)
    return head.to(torch.bfloat16), emb.to(torch.bfloat16)


def eos_vector(wg: np.ndarray, wu: np.ndarray, amplitude: float, dtype: str, gram=None) -> np.ndarray:
    """The planted EOS embedding: least SwiGLU-amplified direction, scaled.
    ``gram`` (optional) replaces Wg^T Wg + Wu^T Wu, e.g. summed over layers."""
    import scipy.linalg
    if gram is None:
        gram = gate_up_gram(wg, wu)
    d = gram.shape[0]
    _, vecs = scipy.linalg.eigh(gram, subset_by_index=[0, 0])
    v = vecs[:, 0]
    if v[np.argmax(np.abs(v))] < 0:
        v = -v
    return round_to_dtype(amplitude * np.sqrt(d) * v, dtype)


def planted_boundaries(w: Workload) -> np.ndarray:
    rng = np.random.default_rng(_streams(w)["boundary"])
    kind = w.boundary[0]
    if kind == "fixed":
        b = np.full(w.batch, int(w.boundary[1]), np.int64)
    elif kind == "loguniform":
        lo, hi = w.boundary[1], w.boundary[2]
        b = np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=w.batch))).astype(np.int64)
    elif kind == "uniform":
        lo, hi = w.boundary[1], w.boundary[2]
        b = rng.integers(lo, hi + 1, size=w.batch).astype(np.int64)
    else:
        raise ValueError(kind)
    if np.any(b < 1) or np.any(b > w.window - 1):
        raise ValueError("planted boundary out of window")
    return b


@dataclass
class Batch:
    """A packed full-window batch: rows of all sequences back to back."""
    x: np.ndarray            # [T_full, d] float32 (dtype-representable)
    cu_seqlens: np.ndarray   # [B+1] int32
    win_off: np.ndarray      # [B] int32, window start inside each sequence
    win_len: np.ndarray      # [B] int32
    planted: np.ndarray      # [B] int64 planted boundary (first EOS position)
    eos: np.ndarray          # [d] float32
    dips: Optional[List[List[Tuple[int, int]]]] = None   # per sequence: (start, length) window positions


def make_batch(w: Workload, eos: np.ndarray) -> Batch:
    d = w.shape.d_model
    st = _streams(w)
    planted = planted_boundaries(w)
    rv = np.random.default_rng(st["visual"])
    rp = np.random.default_rng(st["prompt"])
    rc = np.random.default_rng(st["content"])
    rn = np.random.default_rng(st["noise"])
    rd = np.random.default_rng(st["dips"])
    dips = []
    S = w.seq_len_full
    x = np.empty((w.batch * S, d), np.float32)
    for b in range(w.batch):
        r0 = b * S
        x[r0:r0 + w.n_visual] = rv.standard_normal((w.n_visual, d), dtype=np.float32)
        r1 = r0 + w.n_visual
        x[r1:r1 + w.n_prompt] = rp.standard_normal((w.n_prompt, d), dtype=np.float32)
        r2 = r1 + w.n_prompt
        nb = int(planted[b])
        x[r2:r2 + nb] = rc.standard_normal((nb, d), dtype=np.float32)
        n_eos = w.window - nb
        noise = rn.standard_normal((n_eos, d), dtype=np.float32) * np.float32(w.noise_std)
        x[r2 + nb:r2 + w.window] = eos[None, :] + noise
        runs = []
        n_runs, max_len = w.dips
        for _ in range(n_runs):
            ln = int(rd.integers(1, max_len + 1))
            last = nb - 2 - ln                 # the run ends >= 2 positions before b
            if last < 1:
                continue
            st0 = int(rd.integers(1, last + 1))
            if any(st0 < s1 + l1 + 1 and s1 < st0 + ln + 1 for s1, l1 in runs):
                continue                       # keep runs disjoint and apart
            dn = rd.standard_normal((ln, d), dtype=np.float32) * np.float32(w.noise_std)
            x[r2 + st0:r2 + st0 + ln] = eos[None, :] + dn
            runs.append((st0, ln))
        dips.append(sorted(runs))
    x = round_to_dtype(x, w.dtype)
    cu = (np.arange(w.batch + 1, dtype=np.int64) * S).astype(np.int32)
    win_off = np.full(w.batch, w.prefix_len, np.int32)
    win_len = np.full(w.batch, w.window, np.int32)
    return Batch(x=x, cu_seqlens=cu, win_off=win_off, win_len=win_len,
                 planted=planted, eos=eos, dips=dips)


def make_stack_batch(w: Workload, device) -> Batch:
    """Host batch of a deep stack whose weights come from layer_weights_torch.

    The EOS direction is taken from the detection layer's device-drawn gate
    and up weights (read back to the host), so the planted suffix matches the
    weights the stack actually runs with.
    """
    gram = None
    for l in (w.eos_layers or (w.l_det,)):
        det = layer_weights_torch(w, l, device)
        g = det["wg"].double()
        u = det["wu"].double()
        gl = (g.T @ g + u.T @ u).cpu().numpy()
        gram = gl if gram is None else gram + gl
        del det, g, u
    return make_batch(w, eos_vector(None, None, w.eos_amplitude, w.dtype, gram=gram))


def make_workload(w: Workload, with_weights: bool = True):
    """Host-side inputs: (list of per-layer weight dicts, Batch).

    Only used for workloads whose weights fit a host draw (single-layer
    shapes); the stacks draw weights on the device (layer_weights_torch).
    """
    layers: List[dict] = [layer_weights(w, l) for l in range(w.n_layers)] if with_weights else []
    gram = None
    for l in (w.eos_layers or (w.l_det,)):
        det = layers[l] if with_weights else layer_weights(w, l)
        gl = gate_up_gram(det["wg"], det["wu"])
        gram = gl if gram is None else gram + gl
    eos = eos_vector(None, None, w.eos_amplitude, w.dtype, gram=gram)
    return layers, make_batch(w, eos)
