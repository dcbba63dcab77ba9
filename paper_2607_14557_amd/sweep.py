"""Detector-sensitivity sweeps on synthetic batches.

The paper studies how the SNR boundary detector's knobs move the
accuracy/throughput trade-off: the look-ahead window (2..10, appendix table on
the look-ahead window size), the jump threshold tau_jump against the
tolerance ratio gamma (Sec. 4, hyper-parameter table) and the depth of the
layer whose MLP sparsity is used (Sec. 3.2 and the appendix heat maps).  Its
measurements need trained models and benchmark answers; here the same knobs
are swept against the planted boundaries of a seeded synthetic batch, with
proxies for both sides of the trade-off:

  * premature -- fraction of sequences cut before their planted boundary
    (content lost: the accuracy side);
  * kept      -- mean kept window fraction keep_len / N (the compute the later
    steps still pay: the throughput side);
  * exact, late, none -- cut exactly at the boundary, after it, or not at all.

Everything runs through the library: step 0 over the full window with the
near-zero count fused at every swept layer, then one seer_step0_detect launch
per grid point on those counts.

    python -m paper_2607_14557_amd.sweep --workload sweep_small [--out sweep.json]
"""
import argparse
import json
import sys
import time
from fractions import Fraction

import numpy as np
import torch

from . import seer as S
from .runner import SeerStack, dims_for

LOOKAHEADS = (2, 3, 4, 5, 6, 8, 10)
TAUS = (Fraction(1, 100), Fraction(2, 100), Fraction(3, 100), Fraction(4, 100), Fraction(5, 100),
        Fraction(6, 100))
GAMMAS = tuple(Fraction(g, 10) for g in range(2, 11))
DEFAULT = (Fraction(3, 100), Fraction(3, 5), 3)


def layer_counts(st, x, cu, batch, rows, act_eps, n_layers, stream=None):
    """Run layers 0..n_layers-1 over the packed rows; returns the per-row
    near-zero count of every layer (list of [rows] int32 device tensors)."""
    counts = []
    cur = x
    for l in range(n_layers):
        cnt = torch.empty(rows, dtype=torch.int32, device=x.device)
        nxt = st.buf[l % 2]
        st.layer(l, cur, nxt, cu, None, batch, rows, act_eps=act_eps, act_count=cnt, stream=stream)
        counts.append(cnt)
        cur = nxt
    return counts


def detect(counts, cu, win_off, win_len, batch, d_ff, tau, gamma, lookahead, stream=None):
    """Boundaries and kept lengths (host arrays) for one grid point."""
    dev = counts.device
    bnd = torch.empty(batch, dtype=torch.int32, device=dev)
    keep = torch.empty(batch, dtype=torch.int32, device=dev)
    tau, gamma = Fraction(tau), Fraction(gamma)
    S.seer_step0_detect(counts, cu, win_off, win_len, batch, d_ff,
                        S.seer_snr_params(tau.numerator, tau.denominator, gamma.numerator,
                                          gamma.denominator, int(lookahead)),
                        bnd, keep, stream=stream)
    return bnd.cpu().numpy().astype(np.int64), keep.cpu().numpy().astype(np.int64)


def summarize(boundary, keep, planted, win_len):
    boundary, keep = np.asarray(boundary), np.asarray(keep)
    planted, win_len = np.asarray(planted), np.asarray(win_len)
    none = boundary >= win_len
    return {"exact": float(np.mean(boundary == planted)),
            "premature": float(np.mean(boundary < planted)),
            "late": float(np.mean((boundary > planted) & ~none)),
            "none": float(np.mean(none)),
            "kept": float(np.mean(keep / win_len)),
            "mean_abs_err": float(np.mean(np.abs(boundary - planted)))}


def load_inputs(w, device):
    """Stack, packed input rows and the batch description of a workload."""
    from workloads.generate import layer_weights_torch, make_stack_batch, make_workload
    sh = w.shape
    dims = dims_for(sh.d_model, sh.n_heads, sh.head_dim, sh.d_ff, w.dtype, w.rms_eps)
    st = SeerStack(dims, w.n_layers, w.rows_full, device=device)
    if sh.d_model >= 2048:
        # large layers: weights drawn on the device
        batch = make_stack_batch(w, device)
        for l in range(w.n_layers):
            st.set_layer(l, layer_weights_torch(w, l, device))
    else:
        layers, batch = make_workload(w)
        tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        for l, W in enumerate(layers):
            st.set_layer(l, {k: torch.from_numpy(v).to(device=device, dtype=torch.float32 if k in ("g1", "g2")
                                                       else tdt) for k, v in W.items()})
    x = torch.from_numpy(batch.x).to(device=device, dtype=st.dtype)
    return st, x, batch


def run_sweep(w, device="cuda", lookaheads=LOOKAHEADS, taus=TAUS, gammas=GAMMAS, keep_counts=False):
    """The three sweeps on workload w; returns a dict of tables (and, with
    keep_counts, the host copies of the per-layer counts for checking)."""
    t0 = time.perf_counter()
    st, x, batch = load_inputs(w, device)
    i32 = lambda a: torch.from_numpy(np.asarray(a, np.int32)).to(device)
    cu, off, wl = i32(batch.cu_seqlens), i32(batch.win_off), i32(batch.win_len)
    B, I = w.batch, w.shape.d_ff
    counts = layer_counts(st, x, cu, B, w.rows_full, w.act_eps, w.n_layers)
    torch.cuda.synchronize()
    t_inputs = time.perf_counter() - t0
    planted, wlen = batch.planted, np.asarray(batch.win_len)
    tau0, gamma0, la0 = DEFAULT
    out = {"workload": w.name, "batch": B, "window": w.window, "d_model": w.shape.d_model, "d_ff": I,
           "planted_layer": w.l_det, "noise_std": w.noise_std, "dips": list(w.dips),
           "default": {"tau_jump": str(tau0), "gamma": str(gamma0), "lookahead": la0},
           "lookahead": [], "tau_gamma": [], "layer": [], "points": []}

    def point(kind, layer, tau, gamma, la):
        bnd, keep = detect(counts[layer], cu, off, wl, B, I, tau, gamma, la)
        row = {"layer": layer, "tau_jump": str(Fraction(tau)), "gamma": str(Fraction(gamma)), "lookahead": la}
        row.update(summarize(bnd, keep, planted, wlen))
        out[kind].append(row)
        out["points"].append({"kind": kind, "layer": layer, "tau": [Fraction(tau).numerator, Fraction(tau).denominator],
                              "gamma": [Fraction(gamma).numerator, Fraction(gamma).denominator],
                              "lookahead": la, "boundary": bnd.tolist()})

    for la in lookaheads:
        point("lookahead", w.l_det, tau0, gamma0, la)
    for g in gammas:
        for t in taus:
            point("tau_gamma", w.l_det, t, g, la0)
    for l in range(w.n_layers):
        point("layer", l, tau0, gamma0, la0)
    out["seconds"] = {"inputs_and_layers": round(t_inputs, 2), "total": round(time.perf_counter() - t0, 2)}
    if keep_counts:
        out["_counts"] = [c.cpu().numpy() for c in counts]
        out["_batch"] = batch
    return out


def markdown(res):
    """The three tables as markdown."""
    lines = ["Look-ahead (layer %d, tau_jump %s, gamma %s):" % (res["planted_layer"], res["default"]["tau_jump"],
                                                               res["default"]["gamma"]), "",
             "| look-ahead | exact | premature | late | none | kept |", "|---:|---:|---:|---:|---:|---:|"]
    for r in res["lookahead"]:
        lines.append("| %d | %.2f | %.2f | %.2f | %.2f | %.2f |" % (r["lookahead"], r["exact"], r["premature"],
                                                                   r["late"], r["none"], r["kept"]))
    taus = sorted({r["tau_jump"] for r in res["tau_gamma"]}, key=Fraction)
    gammas = sorted({r["gamma"] for r in res["tau_gamma"]}, key=Fraction)
    lines += ["", "tau_jump x gamma (look-ahead %d): premature / kept" % res["default"]["lookahead"], "",
              "| gamma \\ tau_jump | " + " | ".join(taus) + " |", "|---" * (len(taus) + 1) + "|"]
    cell = {(r["gamma"], r["tau_jump"]): r for r in res["tau_gamma"]}
    for g in gammas:
        lines.append("| %s | " % g + " | ".join("%.2f / %.2f" % (cell[(g, t)]["premature"], cell[(g, t)]["kept"])
                                              for t in taus) + " |")
    lines += ["", "Detection layer (defaults):", "", "| layer | exact | premature | late | none | kept |",
              "|---:|---:|---:|---:|---:|---:|"]
    for r in res["layer"]:
        lines.append("| %d | %.2f | %.2f | %.2f | %.2f | %.2f |" % (r["layer"], r["exact"], r["premature"],
                                                                   r["late"], r["none"], r["kept"]))
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="sweep_small")
    ap.add_argument("--out", default=None, help="write the full result (JSON) here")
    args = ap.parse_args(argv)
    from workloads import WORKLOADS
    w = WORKLOADS[args.workload]
    S.load_library()
    res = run_sweep(w)
    print(markdown(res), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump(res, f)
    print(json.dumps({k: v for k, v in res.items() if k != "points"}), file=sys.stderr)
    return 0


if __name__ == "__main__":
    sys.exit(main())
