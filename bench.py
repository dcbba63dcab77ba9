#!/usr/bin/env python3
"""Benchmark of the Seer hot path on one MI355X.

One bench step is one pass of the whole path over one batch:
  step 0   the full-window layer with the fused near-zero count (the
           detection layer; the LLaDA-8B-shaped layer, B=16 ragged batch of
           [729 visual ; 64 prompt ; 1024 window] rows),
           the SNR boundary scan,
           routing + compaction of the step-input embeddings and of the
           in-flight residual (one launch),
  step 1   one truncated denoising step: the layer on the compacted batch.
Everything is queued on one HIP stream with no host synchronisation inside
the step (kernels read row counts from device memory; grids are sized from
the full-window bound).

value = effective generated tokens per second = (sum of kept window lengths)
x (2 denoising steps per bench step) / step time.  The untruncated step (the
same layer over the full window) is timed separately for the speedup.

The roofline object is for the dominant kernel of every truncated step, the
gate/up GEMM with the SwiGLU epilogue, timed live with HIP events recorded
around it inside the timed steps.  The CPU baseline times the oracle (fp64
NumPy) on a bounded sample of the same batch on this host.

Prints exactly one JSON line on stdout; progress goes to stderr.
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective gen tokens/sec per denoising step (B=16 ragged); MFMA util %"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0
VOCAB = 126464          # LLaDA-8B vocabulary size (the synthetic LM head's width)


# HBM traffic of the dominant kernel per launch, from two rocprofv3 --pmc passes
# (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch) over this workload, each
# scaled by what the same counter reads for a streaming kernel of known size
# (the --copy-calibration dispatches).  Valid only for the kernel sources it
# was taken on: when their hash differs the figure is reported as null.
TRAFFIC_SOURCES = ("paper_2607_14557_amd/csrc/gemm_bf16.hip", "paper_2607_14557_amd/csrc/kernels.h",
                   "paper_2607_14557_amd/csrc/common.h")
TRAFFIC = {"sources_sha256": "cec661a564e9b32974640d76f3f4769bb77f142ef6f097df252703dab8c1b9a4",
           "rows": 14280, "fetch_bytes": 4225459378, "write_bytes": 350945301}


def sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(rows_exec):
    if TRAFFIC is None or TRAFFIC["sources_sha256"] != sources_sha256() or TRAFFIC["rows"] != rows_exec:
        return None
    return TRAFFIC["fetch_bytes"] + TRAFFIC["write_bytes"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Hip:
    """HIP events through the runtime torch already loaded (same soname)."""

    def __init__(self):
        self.L = ctypes.CDLL("libamdhip64.so.7")
        self.L.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.L.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                               ctypes.c_void_p]
        self.L.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.L.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        if self.L.hipEventCreate(ctypes.byref(e)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return e.value

    def record(self, e, stream):
        if self.L.hipEventRecord(e, stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def ms(self, a, b):
        f = ctypes.c_float()
        if self.L.hipEventElapsedTime(ctypes.byref(f), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(f.value)


def host_cpu():
    """The host's CPU model, logical CPU count, the CPUs this process may run
    on, and the BLAS threads NumPy uses (what the oracle actually runs on)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    try:
        import numpy  # noqa: F401  (loads the BLAS threadpool)
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
                   or [avail])
    except Exception:
        blas = avail
    return {"cpu_model": model, "nproc": os.cpu_count(), "cpus_available": avail, "blas_threads": int(blas)}


def layer_flop(sh, seq_rows, used=None):
    """Algorithmic flop of one layer over sequences of seq_rows rows (keys: the
    used rows): 2 rows (4 d^2 + 3 d I) in the projections, 4 S_q S_k d in
    attention (scores and the weighted sum)."""
    d, I = sh.d_model, sh.d_ff
    used = seq_rows if used is None else used
    g = sum(2 * int(s) * (4 * d * d + 3 * d * I) for s in seq_rows)
    a = sum(4 * int(min(u, s)) * int(u) * d for s, u in zip(seq_rows, used))
    return g + a


def cpu_baseline(w, layers, batch, seconds):
    """Oracle (fp64 NumPy) on the first sequences of the batch, ~`seconds` of work."""
    import numpy as np
    import oracle
    hc = host_cpu()
    cores = hc["blas_threads"]
    sh = w.shape
    t0 = time.perf_counter()
    toks = 0
    nseq = 0
    S = w.seq_len_full
    for b in range(w.batch):
        x = batch.x[b * S:(b + 1) * S]
        res = oracle.run_pipeline(layers, x, [0, S], batch.win_off[b:b + 1], batch.win_len[b:b + 1],
                                  sh.n_heads, sh.d_ff, w.rms_eps, w.act_eps, w.l_det)
        toks += 2 * int(res.keep_len[0])
        nseq += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    return {"value": toks / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": "oracle step 0 (full-window layer + count + SNR scan + routing/compaction) and "
                      "one truncated step, fp64 NumPy, on the first %d of %d sequences (%.1f s)"
                      % (nseq, w.batch, dt),
            "cpu_model": hc["cpu_model"], "nproc": hc["nproc"], "cpus_available": hc["cpus_available"]}


def oracle_timing(names):
    """The oracle timed on this host's cores, per workload (one JSON line).

    Single-layer workloads: the whole path end to end (step 0: full-window
    layer with the count, SNR scan, routing + compaction; then one truncated
    step), in fp64 (the oracle) and in fp32 (the same definitions, for
    reference).  32-layer stacks: the step-0 detection pass (the layers up to
    and including the detection layer on the full window, the count, the scan,
    routing + compaction) and one layer of a truncated step, fp64; their
    weights are drawn on the GPU (inputs only) and read back one layer at a
    time.  Seconds are measured, flop counted from the shapes; nothing is
    extrapolated."""
    import numpy as np
    import oracle
    from oracle.detect import detect_batch
    from oracle.route import repack_rows, route_batch
    from workloads import WORKLOADS
    from workloads.generate import layer_weights_torch, make_stack_batch, make_workload

    hc = host_cpu()
    out = []
    for name in names:
        w = WORKLOADS[name]
        sh = w.shape
        S_full = [int(w.seq_len_full)] * w.batch
        if w.n_layers == 1:
            layers, batch = make_workload(w)
            for dt in (np.float64, np.float32):
                log("oracle %s %s: end to end" % (name, np.dtype(dt).name))
                t0 = time.perf_counter()
                res = oracle.run_pipeline(layers, batch.x, batch.cu_seqlens, batch.win_off, batch.win_len,
                                          sh.n_heads, sh.d_ff, w.rms_eps, w.act_eps, w.l_det, dtype=dt)
                sec = time.perf_counter() - t0
                cu_t = np.asarray(res.cu_trunc)
                f0 = layer_flop(sh, S_full)
                f1 = layer_flop(sh, np.diff(cu_t), res.seqused)
                assert np.array_equal(res.boundary, batch.planted)
                out.append({"workload": name, "what": "step 0 + one truncated step, end to end",
                            "precision": np.dtype(dt).name, "seconds": round(sec, 3),
                            "flop": f0 + f1, "gflop_per_s": round((f0 + f1) / sec / 1e9, 1),
                            "sum_keep_len": int(np.sum(res.keep_len))})
                log("  %.2f s, %.1f GFLOP/s" % (sec, (f0 + f1) / sec / 1e9))
            continue
        import torch
        batch = make_stack_batch(w, "cuda")
        host_w = lambda l: {k: v.double().cpu().numpy() for k, v in layer_weights_torch(w, l, "cuda").items()}
        log("oracle %s: detection pass, layers 0..%d on the full window" % (name, w.l_det))
        t_pass, h, counts = 0.0, np.asarray(batch.x, np.float64), None
        for l in range(w.l_det + 1):
            W = host_w(l)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            h, c = oracle.layer_forward(h, batch.cu_seqlens, W, sh.n_heads, w.rms_eps,
                                        act_eps=w.act_eps if l == w.l_det else None)
            t_pass += time.perf_counter() - t0
            if l == w.l_det:
                counts = c
            del W
            log("  layer %d done (%.1f s so far)" % (l, t_pass))
        t0 = time.perf_counter()
        bnd, keep = detect_batch(counts, batch.cu_seqlens, batch.win_off, batch.win_len, sh.d_ff)
        rt = route_batch(keep, batch.win_len)
        x_t, cu_t, used, _ = repack_rows(batch.x, batch.cu_seqlens, batch.win_off, keep, rt.alloc, 256)
        t_pass += time.perf_counter() - t0
        assert np.array_equal(bnd, batch.planted)
        f_pass = (w.l_det + 1) * layer_flop(sh, S_full)
        out.append({"workload": name, "what": "step-0 detection pass (layers 0..%d, count, scan, "
                    "routing + compaction)" % w.l_det, "precision": "float64", "seconds": round(t_pass, 3),
                    "flop": f_pass, "gflop_per_s": round(f_pass / t_pass / 1e9, 1)})
        del h
        W = host_w(0)
        log("oracle %s: one layer of a truncated step (%d rows)" % (name, int(cu_t[-1])))
        t0 = time.perf_counter()
        oracle.layer_forward(x_t[:int(cu_t[-1])], cu_t, W, sh.n_heads, w.rms_eps, seqused=used)
        sec = time.perf_counter() - t0
        f1 = layer_flop(sh, np.diff(cu_t), used)
        out.append({"workload": name, "what": "one layer of a truncated step", "precision": "float64",
                    "seconds": round(sec, 3), "flop": f1, "gflop_per_s": round(f1 / sec / 1e9, 1)})
        log("  %.1f s" % sec)
        del W
    line = {"metric": "oracle seconds on the host cores", "kind": "oracle", **hc, "entries": out}
    print(json.dumps(line), flush=True)


def bench_stack(args, w):
    """A 32-layer stack: one job = step 0 (layers up to the detection layer on
    the full window with the count, the SNR scan, routing + compaction, the
    remaining layers on the compacted batch) plus the truncated denoising steps
    (every layer on the compacted batch).  Prints one JSON line."""
    import numpy as np
    import torch
    from paper_2607_14557_amd import seer as S
    from paper_2607_14557_amd.runner import (SeerStack, StepGraphs, SyntheticSampler, dims_for, pinned_ctrl,
                                             poll_ctrl)
    from workloads.generate import layer_weights_torch, lm_head_torch, make_stack_batch

    sh = w.shape
    d, I, B, L = sh.d_model, sh.d_ff, w.batch, w.n_layers
    dev = torch.device("cuda:0")
    log("generating stack workload %s (%d layers)" % (w.name, L))
    t0 = time.perf_counter()
    batch = make_stack_batch(w, dev)
    T = w.rows_full
    granule = 256
    cap = ((T + granule - 1) // granule) * granule + granule
    dims = dims_for(d, sh.n_heads, sh.head_dim, I, "bf16", w.rms_eps, rope_theta=args.rope)
    st = SeerStack(dims, L, cap)
    for l in range(L):
        Wl = layer_weights_torch(w, l, dev)
        st.set_layer(l, Wl)
        del Wl
    x = torch.from_numpy(batch.x).to(torch.bfloat16).to(dev)
    i32 = lambda a: torch.from_numpy(np.asarray(a, np.int32)).to(dev)
    cu, off, wl = i32(batch.cu_seqlens), i32(batch.win_off), i32(batch.win_len)
    log("  inputs and %d prepacked layers ready in %.1f s" % (L, time.perf_counter() - t0))
    if args.graph:
        # recorded steps need a created stream; everything runs on it
        gs = torch.cuda.Stream()
        torch.cuda.set_stream(gs)
        ctrl_t, ctrl_w = pinned_ctrl(), pinned_ctrl()
    sp = torch.cuda.current_stream().cuda_stream
    hip = Hip()
    n_trunc = w.trunc_steps
    graphs = {}

    kv = None
    if args.kv_cache:
        # prefix keys/values of every layer, cached by the first truncated step
        P = np.asarray(batch.win_off, np.int64)
        kv_rows = int(P.sum())
        cu_kv = i32(np.concatenate([[0], np.cumsum(P)]))
        caches = st.alloc_kv_caches(kv_rows)
        kv = (caches, cu_kv, kv_rows)
        log("  prefix K/V caches: %d rows x %d layers (%.1f GB)" % (kv_rows, L, kv_rows * 2 * d * 2 * L / 1e9))

    smp = None
    if args.sampler:
        w_lm, emb = lm_head_torch(w, VOCAB, dev)
        smp = SyntheticSampler(dims, w_lm, emb, cap)
        x_cur = torch.empty(cap, d, dtype=torch.bfloat16, device=dev)
        log("  synthetic LM head and embeddings: vocab %d (%.1f GB)" % (VOCAB, 2 * VOCAB * d * 2 / 1e9))

    def job():
        if args.graph:
            return job_graph()
        if smp is not None:
            return job_sampled()
        r = st.step0(x, cu, off, wl, B, T, w.l_det, w.act_eps, granule=granule, trunc_capacity=cap, stream=sp)
        if kv is None:
            for _ in range(n_trunc):
                st.forward(r.x_trunc, r.cu_trunc, r.seqused, B, cap, stream=sp)
            return r
        caches, cu_kv, kv_rows = kv
        # the kept window rows alone, and their routed capacity (one host read per job)
        x_w, cu_w, used_w, _ = st.window_rows(x, cu, off, wl, r.keep_len, B, cap, granule=granule, stream=sp)
        rows_w = int(cu_w[B].item())
        rows_w = ((rows_w + granule - 1) // granule) * granule
        st.forward_export(r.x_trunc, r.cu_trunc, r.seqused, B, cap, caches, cu_kv, kv_rows, stream=sp)
        for _ in range(n_trunc - 1):
            st.forward_cached(x_w, cu_w, used_w, B, max(rows_w, 1), caches, cu_kv, kv_rows, stream=sp)
        r.cached = (x_w, cu_w, used_w, rows_w)
        return r

    def job_sampled():
        # cached steps whose inputs evolve: LM head + remasking after each one
        r = st.step0(x, cu, off, wl, B, T, w.l_det, w.act_eps, granule=granule, trunc_capacity=cap, stream=sp)
        caches, cu_kv, kv_rows = kv
        x_w, cu_w, used_w, _ = st.window_rows(x, cu, off, wl, r.keep_len, B, cap, granule=granule, stream=sp)
        rows_w = int(cu_w[B].item())
        rows_w = max(1, ((rows_w + granule - 1) // granule) * granule)
        st.forward_export(r.x_trunc, r.cu_trunc, r.seqused, B, cap, caches, cu_kv, kv_rows, stream=sp)
        smp.reset()
        x_cur[:rows_w].copy_(x_w[:rows_w])
        n = n_trunc - 1
        for s_ in range(n):
            h = st.forward_cached(x_cur, cu_w, used_w, B, rows_w, caches, cu_kv, kv_rows, stream=sp)
            # the next inputs overwrite x_cur: layer 0 has consumed it
            smp.step(h, cu_w, used_w, B, rows_w, x_w, x_cur, n - s_, w.window, stream=sp)
        r.cached = (x_w, cu_w, used_w, rows_w)
        return r

    def job_graph():
        # step 0 eager; the host polls the pinned control word of each repack
        # (no stream sync) and replays the truncated steps recorded for the
        # routed capacity's 1-D graph shape
        r = st.step0(x, cu, off, wl, B, T, w.l_det, w.act_eps, granule=granule, trunc_capacity=cap,
                     ctrl_host=ctrl_t, stream=sp)
        if kv is None:
            if "trunc" not in graphs:
                graphs["trunc"] = StepGraphs(
                    lambda rows: st.forward(r.x_trunc, r.cu_trunc, r.seqused, B, rows, stream=sp), gs, cap,
                    granule)
            for _ in range(n_trunc):
                graphs["trunc"].run(r.routed["capacity_rows"])
            return r
        caches, cu_kv, kv_rows = kv
        x_w, cu_w, used_w, _ = st.window_rows(x, cu, off, wl, r.keep_len, B, cap, granule=granule,
                                              ctrl_host=ctrl_w, stream=sp)
        st.forward_export(r.x_trunc, r.cu_trunc, r.seqused, B, r.rows_ub, caches, cu_kv, kv_rows, stream=sp)
        routed_w = poll_ctrl(ctrl_w)
        rows_w = routed_w["capacity_rows"]
        if "cached" not in graphs:
            graphs["cached"] = StepGraphs(
                lambda rows: st.forward_cached(x_w, cu_w, used_w, B, rows, caches, cu_kv, kv_rows, stream=sp),
                gs, cap, granule)
        for _ in range(n_trunc - 1):
            graphs["cached"].run(rows_w)
        r.cached = (x_w, cu_w, used_w, max(rows_w, 1))
        return r

    log("warmup %d job(s)" % args.warmup)
    r = None
    for _ in range(args.warmup):
        r = job()
    torch.cuda.synchronize()
    log("timing %d job(s) of 1 + %d denoising steps" % (args.steps, n_trunc))
    t0 = time.perf_counter()
    for _ in range(args.steps):
        r = job()
    torch.cuda.synchronize()
    ms_job = (time.perf_counter() - t0) * 1e3 / args.steps
    keep = r.keep_len.cpu().numpy()
    if not np.array_equal(r.boundary.cpu().numpy(), batch.planted):
        log("WARNING: detected boundaries differ from the planted ones")
    rows_t = int(r.seqused.cpu().numpy().sum())

    def timed(fn, reps=3):
        e0, e1 = hip.event(), hip.event()
        fn()
        hip.record(e0, sp)
        for _ in range(reps):
            fn()
        hip.record(e1, sp)
        torch.cuda.synchronize()
        return hip.ms(e0, e1) / reps

    log("timing one truncated and one untruncated %d-layer step" % L)
    t_trunc = timed(lambda: st.forward(r.x_trunc, r.cu_trunc, r.seqused, B, cap, stream=sp))
    t_full = timed(lambda: st.forward(x, cu, None, B, T, stream=sp), reps=1)
    t_cached = None
    if kv is not None:
        x_w, cu_w, used_w, rows_w = r.cached
        t_cached = timed(lambda: st.forward_cached(x_w, cu_w, used_w, B, max(rows_w, 1), kv[0], kv[1], kv[2],
                                                   stream=sp))
    t_sampler = None
    if smp is not None:
        x_w, cu_w, used_w, rows_w = r.cached
        h = st.buf[0]
        t_sampler = timed(lambda: smp.step(h, cu_w, used_w, B, rows_w, x_w, x_cur, 2, w.window, stream=sp))
        committed = int((smp.tokens[:rows_w] >= 0).sum().item())
        log("  sampler: %d of %d window rows committed after the job" % (committed, int(used_w.sum().item())))
    t_graph = {}
    host_ms = {}
    if args.graph:
        log("timing one replay of each recorded step")
        if kv is None:
            eager_fn = lambda: st.forward(r.x_trunc, r.cu_trunc, r.seqused, B, r.rows_ub, stream=sp)
            graph_fn = lambda: graphs["trunc"].run(r.routed["capacity_rows"])
            t_graph["trunc"] = timed(graph_fn)
        else:
            x_w, cu_w, used_w, rows_w = r.cached
            eager_fn = lambda: st.forward_cached(x_w, cu_w, used_w, B, rows_w, kv[0], kv[1], kv[2], stream=sp)
            graph_fn = lambda: graphs["cached"].run(rows_w)
            t_graph["cached"] = timed(graph_fn)

        # host time to enqueue one step (the GPU is idle at the start of each)
        def enqueue_ms(fn, reps=5):
            best = None
            for _ in range(reps):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                fn()
                dt = (time.perf_counter() - t0) * 1e3
                best = dt if best is None else min(best, dt)
            torch.cuda.synchronize()
            return best
        host_ms = {"eager": enqueue_ms(eager_fn), "graph": enqueue_ms(graph_fn)}
    # the dominant kernel: gate/up GEMM of a truncated step, timed inside one layer
    ev = [hip.event() for _ in range(8)]
    y = torch.empty(cap, d, dtype=torch.bfloat16, device=dev)
    for _ in range(2):
        S.seer_layer_forward_varlen_timed(dims, st.packed[0], r.x_trunc, y, cap, r.cu_trunc, r.seqused, B,
                                          0.0, None, st.workspace, ev, stream=sp)
    torch.cuda.synchronize()
    gu_ms = hip.ms(ev[5], ev[6])
    flop = rows_t * 2 * 2 * I * d
    achieved = flop / (gu_ms * 1e-3) / 1e12
    n_den = 1 + n_trunc
    value = int(keep.sum()) * n_den / (ms_job * 1e-3)
    out = {
        "metric": "effective gen tokens/sec over step 0 + %d truncated denoising steps (%d-layer stack%s)"
                  % (n_trunc, L, (", prefix K/V cached after the first truncated step" if kv else "")
                     + (", LM head + remasking after each cached step" if smp is not None else "")),
        "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_job, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; random-init LLaDA-8B-shaped %d-layer stack, planted EOS suffixes)" % L,
        "config": {"workload": w.name, "rope_theta": args.rope, "batch": B, "visual_prefix": w.n_visual,
                   "prompt": w.n_prompt,
                   "window": w.window, "layers": L, "detection_layer": w.l_det,
                   "denoising_steps_per_job": n_den, "sum_keep_len": int(keep.sum()), "rows_full": T,
                   "rows_trunc": rows_t, "d_model": d, "heads": sh.n_heads, "head_dim": sh.head_dim,
                   "d_ff": I},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "kernel": "gemm_bf16_kernel<EPI_SWIGLU> (truncated-step gate/up GEMM, layer 0)",
                     "flop_per_launch": flop, "launch_ms": round(gu_ms, 4)},
        "trunc_step_ms": round(t_trunc, 3), "full_step_ms": round(t_full, 3),
        "speedup_trunc_vs_full": round(t_full / t_trunc, 3),
        # raw packed rows through all layers of one step per second
        "trunc_step_rows_per_s": round(rows_t / (t_trunc * 1e-3), 1),
        "full_step_rows_per_s": round(T / (t_full * 1e-3), 1),
        "job_speedup_vs_untruncated": round(n_den * t_full / ms_job, 3),
        "cached_step_ms": None if t_cached is None else round(t_cached, 3),
        "speedup_cached_vs_trunc": None if t_cached is None else round(t_trunc / t_cached, 3),
        "graph": bool(args.graph),
        "sampler": {"vocab": VOCAB, "ms_per_step": round(t_sampler, 3)} if t_sampler is not None else None,
        "trunc_step_ms_graph": round(t_graph["trunc"], 3) if "trunc" in t_graph else None,
        "cached_step_ms_graph": round(t_graph["cached"], 3) if "cached" in t_graph else None,
        "graph_shapes": {k: sorted(g.graphs) for k, g in graphs.items()} if args.graph else None,
        "host_enqueue_ms_eager": round(host_ms["eager"], 3) if host_ms else None,
        "host_enqueue_ms_graph": round(host_ms["graph"], 3) if host_ms else None,
        "cpu_baseline": None,
        "cpu_baseline_note": "one oracle step of a 32-layer stack takes hours; the default workload's line "
                             "carries the CPU baseline",
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 20; 1 for the 32-layer stacks, where a step is a whole job)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 5; 1 for the stacks)")
    ap.add_argument("--workload", default="llada_b16_ragged")
    ap.add_argument("--policy", default="hybrid", choices=["hybrid", "naive_pad", "varlen_only"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run a 1 GiB fill and a 1 GiB read+write streaming kernel "
                         "(the known-size dispatches that scale the HBM byte counters)")
    ap.add_argument("--no-untruncated", action="store_true",
                    help="skip the separate untruncated-step and cached-prefix-step timings (they "
                         "launch the gate/up GEMM kernel at other sizes, which a per-kernel profile "
                         "would mix in)")
    ap.add_argument("--rope", type=float, default=0.0,
                    help="rotary embedding of q and k with this theta (0: none, the paper's layer)")
    ap.add_argument("--graph", action="store_true",
                    help="32-layer stacks: the host polls the pinned control word of each repack and "
                         "replays the truncated (or cached) steps from HIP graphs recorded per 1-D graph "
                         "shape of the routed capacity")
    ap.add_argument("--sampler", action="store_true",
                    help="32-layer stacks with --kv-cache: a synthetic LM head (vocab %d) and low-confidence "
                         "remasking after every cached step, so each step's inputs differ" % VOCAB)
    ap.add_argument("--kv-cache", action="store_true",
                    help="32-layer stacks: after step 0, one full truncated step caches every layer's "
                         "prefix keys/values and the remaining steps run on the kept window rows")
    ap.add_argument("--oracle-timing", default=None, metavar="WORKLOADS",
                    help="comma-separated workloads: time the oracle on this host's cores instead "
                         "(single layers end to end in fp64 and fp32; stacks: the step-0 detection "
                         "pass and one truncated layer) and print one JSON line")
    args = ap.parse_args()
    if args.oracle_timing:
        return oracle_timing(args.oracle_timing.split(","))

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU; there is no multi-GPU path "
              "(requested --gpus %d, WORLD_SIZE %d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_14557_amd import seer as S
    from paper_2607_14557_amd.runner import dims_for
    from workloads import WORKLOADS
    from workloads.generate import make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    S.load_library()
    w = WORKLOADS[args.workload]
    if args.steps is None:
        args.steps = 20 if w.n_layers == 1 else 1
    if args.warmup is None:
        args.warmup = 5 if w.n_layers == 1 else 1
    if w.dtype != "bf16":
        raise SystemExit("bench.py times bf16 workloads")
    if args.sampler and (args.graph or not args.kv_cache):
        print("--sampler needs --kv-cache and excludes --graph", file=sys.stderr)
        sys.exit(2)
    if w.n_layers > 1:
        return bench_stack(args, w)
    if args.graph or args.kv_cache or args.sampler:
        print("--graph, --kv-cache and --sampler apply to the layer stacks (--workload llada32_video_b4 or "
              "llada32_multicrop_b8)", file=sys.stderr)
        sys.exit(2)
    sh = w.shape
    d, I = sh.d_model, sh.d_ff
    policy = {"hybrid": S.SEER_ROUTE_HYBRID, "naive_pad": S.SEER_ROUTE_NAIVE_PAD,
              "varlen_only": S.SEER_ROUTE_VARLEN_ONLY}[args.policy]

    log("generating workload %s" % w.name)
    t0 = time.perf_counter()
    layers, batch = make_workload(w)
    log("  inputs ready in %.1f s" % (time.perf_counter() - t0))
    dev = torch.device("cuda:0")
    dims = dims_for(d, sh.n_heads, sh.head_dim, I, "bf16", w.rms_eps, rope_theta=args.rope)
    T = w.rows_full
    granule = 256
    cap = ((T + granule - 1) // granule) * granule
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    wdev = {k: torch.from_numpy(np.asarray(v, np.float32)).to(
        torch.bfloat16 if k not in ("g1", "g2") else torch.float32).to(dev) for k, v in layers[0].items()}
    packed = torch.empty(S.seer_prepacked_bytes(dims), dtype=torch.uint8, device=dev)
    S.seer_prepack_weights(dims, wdev, packed, stream=sp)
    del wdev
    ws_bytes = S.seer_layer_workspace_bytes(dims, cap)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    x_full = torch.from_numpy(batch.x).to(torch.bfloat16).to(dev)
    i32 = lambda a: torch.from_numpy(np.asarray(a, np.int32)).to(dev)
    cu_full, win_off, win_len = i32(batch.cu_seqlens), i32(batch.win_off), i32(batch.win_len)
    y_full = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    counts = torch.empty(T, dtype=torch.int32, device=dev)
    bnd = torch.empty(w.batch, dtype=torch.int32, device=dev)
    keep = torch.empty(w.batch, dtype=torch.int32, device=dev)
    x_t = torch.zeros(cap, d, dtype=torch.bfloat16, device=dev)
    h_t = torch.zeros(cap, d, dtype=torch.bfloat16, device=dev)
    y_t = torch.zeros(cap, d, dtype=torch.bfloat16, device=dev)
    cu_t = torch.empty(w.batch + 1, dtype=torch.int32, device=dev)
    used = torch.empty(w.batch, dtype=torch.int32, device=dev)
    route = torch.empty(w.batch, 3, dtype=torch.int32, device=dev)
    ctrl = torch.zeros(16, dtype=torch.int32, device=dev)
    snr = S.seer_snr_params(3, 100, 3, 5, 3)
    desc = S.seer_repack_desc(policy, 1, 5, granule, d * 2, cap, 0, 0)

    hip = Hip()
    n_ev = args.warmup + args.steps
    # The timed steps record only the two events around the roofline kernel
    # (the truncated step's gate/up GEMM): every record delays the next launch
    # by a few microseconds.  The per-kernel breakdown comes from a separate
    # pass with an event around every kernel, after the timed steps.
    n_instr = max(3, min(args.steps, 10))
    ev_roof = [[hip.event() for _ in range(2)] for _ in range(n_ev)]
    ev_full = [[hip.event() for _ in range(9)] for _ in range(n_instr)]
    ev_trunc = [[hip.event() for _ in range(8)] for _ in range(n_instr)]
    ev_mid = [[hip.event() for _ in range(2)] for _ in range(n_instr)]

    def step(i, instr=False):
        # the detection layer: count, SNR scan, down projection on the kept rows
        S.seer_layer_forward_detect(dims, packed, x_full, y_full, T, cu_full, w.batch, w.act_eps, counts,
                                    win_off, win_len, snr, bnd, keep, ws, stream=sp,
                                    events=ev_full[i] if instr else None)
        S.seer_batch_repack(desc, [x_full, y_full], [x_t, h_t], cu_full, win_off, win_len, keep,
                            w.batch, cu_t, used, route, ctrl, None, stream=sp)
        if instr:
            hip.record(ev_mid[i][0], sp)
        ev = ev_trunc[i] if instr else [None] * 5 + ev_roof[i] + [None]
        S.seer_layer_forward_varlen_timed(dims, packed, x_t, y_t, cap, cu_t, used, w.batch, 0.0,
                                          None, ws, ev, stream=sp)
        if instr:
            hip.record(ev_mid[i][1], sp)

    log("warmup %d steps" % args.warmup)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    keep_h = keep.cpu().numpy()
    used_h = used.cpu().numpy()
    route_h = route.cpu().numpy()
    ctrl_h = ctrl.cpu().numpy()
    if not np.array_equal(bnd.cpu().numpy(), batch.planted):
        log("WARNING: detected boundaries differ from the planted ones")
    sum_keep = int(keep_h.sum())
    rows_alg = int(used_h.sum())          # prefix + kept window rows (no padding)
    rows_exec = int(ctrl_h[0])            # rows the truncated kernels process

    log("timing %d steps" % args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.warmup, n_ev):
        step(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    # the roofline kernel's launches inside the timed region
    roof_ms = float(np.mean([hip.ms(ev_roof[i][0], ev_roof[i][1]) for i in range(args.warmup, n_ev)]))

    log("per-kernel pass: %d steps with an event around every kernel" % n_instr)
    for i in range(n_instr):
        step(i, instr=True)
    torch.cuda.synchronize()
    rng = range(n_instr)
    kern = ["rms1", "qkv", "attn", "o", "rms2", "gateup", "down"]
    kern_det = ["rms1", "qkv", "attn", "o", "rms2", "gateup", "detect", "down"]

    def kernel_ms(evs, names):
        return {k: float(np.mean([hip.ms(evs[i][j], evs[i][j + 1]) for i in rng]))
                for j, k in enumerate(names)}

    kf, kt = kernel_ms(ev_full, kern_det), kernel_ms(ev_trunc, kern)
    t_full_layer = float(np.mean([hip.ms(ev_full[i][0], ev_full[i][8]) for i in rng]))
    t_trunc = float(np.mean([hip.ms(ev_mid[i][0], ev_mid[i][1]) for i in rng]))
    t_mid = float(np.mean([hip.ms(ev_full[i][8], ev_mid[i][0]) for i in rng]))

    def time_untruncated():
        log("timing the untruncated step")
        for _ in range(3):
            S.seer_layer_forward_varlen(dims, packed, x_full, y_full, T, cu_full, None, w.batch, 0.0,
                                        None, ws, stream=sp)
        e0, e1 = hip.event(), hip.event()
        reps = max(5, args.steps // 2)
        hip.record(e0, sp)
        for _ in range(reps):
            S.seer_layer_forward_varlen(dims, packed, x_full, y_full, T, cu_full, None, w.batch, 0.0,
                                        None, ws, stream=sp)
        hip.record(e1, sp)
        torch.cuda.synchronize()
        return hip.ms(e0, e1) / reps

    def time_cached():
        """A truncated step on the kept window rows alone, the prefix keys and
        values cached from a full truncated step (Appendix D, KV caching)."""
        log("timing the cached-prefix truncated step")
        x_w = torch.zeros(cap, d, dtype=torch.bfloat16, device=dev)
        y_w = torch.zeros(cap, d, dtype=torch.bfloat16, device=dev)
        cu_w = torch.empty(w.batch + 1, dtype=torch.int32, device=dev)
        used_w = torch.empty(w.batch, dtype=torch.int32, device=dev)
        route_w = torch.empty(w.batch, 3, dtype=torch.int32, device=dev)
        ctrl_w = torch.zeros(16, dtype=torch.int32, device=dev)
        desc_w = S.seer_repack_desc(policy, 1, 5, granule, d * 2, cap, 0, S.SEER_REPACK_WINDOW_ONLY)
        S.seer_batch_repack(desc_w, [x_full], [x_w], cu_full, win_off, win_len, keep, w.batch, cu_w,
                            used_w, route_w, ctrl_w, None, stream=sp)
        P = np.asarray(batch.win_off, np.int64)
        kv_rows = int(P.sum())
        cu_kv = i32(np.concatenate([[0], np.cumsum(P)]))
        kv = torch.empty(kv_rows, 2 * d, dtype=torch.bfloat16, device=dev)
        S.seer_layer_forward_varlen(dims, packed, x_t, y_t, cap, cu_t, used, w.batch, 0.0, None, ws, stream=sp)
        S.seer_kv_export(dims, ws, cap, cu_t, w.batch, cu_kv, kv_rows, kv, stream=sp)
        torch.cuda.synchronize()
        rows_w = int(ctrl_w[1].item())          # routed capacity of the window rows
        for _ in range(3):
            S.seer_layer_forward_cached(dims, packed, x_w, y_w, rows_w, cu_w, used_w, w.batch, kv, cu_kv,
                                        kv_rows, ws, stream=sp)
        e0, e1 = hip.event(), hip.event()
        reps = max(10, args.steps)
        hip.record(e0, sp)
        for _ in range(reps):
            S.seer_layer_forward_cached(dims, packed, x_w, y_w, rows_w, cu_w, used_w, w.batch, kv, cu_kv,
                                        kv_rows, ws, stream=sp)
        hip.record(e1, sp)
        torch.cuda.synchronize()
        return hip.ms(e0, e1) / reps, int(ctrl_w[0].item())

    # untruncated denoising step (same layer over the full window, no count) for the speedup,
    # and the cached-prefix variant of the truncated step
    t_full = t_cached = rows_cached = None
    if not args.no_untruncated:
        t_full = time_untruncated()
        t_cached, rows_cached = time_cached()

    gemm_flop_row = {"qkv": 2 * 3 * d * d, "o": 2 * d * d, "gateup": 2 * 2 * I * d, "down": 2 * I * d}
    seqlens_full = np.diff(batch.cu_seqlens).astype(np.int64)
    seqlens_t = used_h.astype(np.int64)
    attn_flop = lambda lens: int(np.sum(4 * lens * lens * d))

    def tflops(flop, ms):
        return flop / (ms * 1e-3) / 1e12

    kernels = {}
    for tag, kms, rows, lens in (("full", kf, T, seqlens_full), ("trunc", kt, rows_alg, seqlens_t)):
        for k in ("qkv", "o", "gateup", "down"):
            # the detection layer's down projection runs on the kept rows: its
            # algorithmic flop count is that of the kept (prefix + window) rows
            r = rows_alg if (tag, k) == ("full", "down") else rows
            kernels["%s_%s" % (tag, k)] = {"ms": round(kms[k], 4),
                                           "tflops": round(tflops(r * gemm_flop_row[k], kms[k]), 1)}
        kernels["%s_attn" % tag] = {"ms": round(kms["attn"], 4),
                                    "tflops": round(tflops(attn_flop(lens), kms["attn"]), 1)}
        kernels["%s_rms" % tag] = {"ms": round(kms["rms1"] + kms["rms2"], 4)}
    gemm_ms_t = sum(kt[k] for k in ("qkv", "o", "gateup", "down"))
    gemm_flop_t = rows_alg * sum(gemm_flop_row.values())

    dom_flop = rows_alg * gemm_flop_row["gateup"]
    dom_ms = roof_ms
    achieved = tflops(dom_flop, dom_ms)
    traffic = measured_traffic(rows_exec)
    # compulsory bytes: both weight halves once, the A rows once, the activation rows written once
    alg_bytes = 2 * (2 * I * d + rows_exec * d + rows_exec * I)
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                "traffic_unit": "bytes per launch (HBM, counters)", "compulsory_bytes": alg_bytes,
                "kernel": "gemm_bf16_kernel<EPI_SWIGLU> (truncated-step gate/up GEMM)",
                "flop_per_launch": dom_flop, "launch_ms": round(dom_ms, 4)}

    value = 2 * sum_keep / (ms_step * 1e-3)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; random-init LLaDA-8B-shaped layer, planted EOS suffixes)",
        "config": {"workload": w.name, "rope_theta": args.rope, "batch": w.batch, "visual_prefix": w.n_visual,
                   "prompt": w.n_prompt, "window": w.window, "layers": w.n_layers,
                   "d_model": d, "heads": sh.n_heads, "head_dim": sh.head_dim, "d_ff": I,
                   "policy": args.policy, "denoising_steps_per_bench_step": 2,
                   "sum_keep_len": sum_keep, "rows_full": T, "rows_trunc": rows_alg,
                   "rows_trunc_executed": rows_exec},
        "roofline": roofline,
        "trunc_step_ms": round(t_trunc, 4),
        "full_step_ms": None if t_full is None else round(t_full, 4),
        "speedup_trunc_vs_full": None if t_full is None else round(t_full / t_trunc, 3),
        "trunc_step_tokens_per_s": round(sum_keep / (t_trunc * 1e-3), 1),
        # raw packed rows (prefix + kept window; full window) per second of one step
        "trunc_step_rows_per_s": round(rows_alg / (t_trunc * 1e-3), 1),
        "full_step_rows_per_s": None if t_full is None else round(T / (t_full * 1e-3), 1),
        "full_step_tokens_per_s": None if t_full is None else round(sum_keep / (t_full * 1e-3), 1),
        "cached_step_ms": None if t_cached is None else round(t_cached, 4),
        "cached_step_tokens_per_s": None if t_cached is None else round(sum_keep / (t_cached * 1e-3), 1),
        "speedup_cached_vs_trunc": None if t_cached is None else round(t_trunc / t_cached, 3),
        "speedup_cached_vs_full": None if t_cached is None or t_full is None else round(t_full / t_cached, 3),
        "rows_cached_executed": rows_cached,
        "step0_layer_ms": round(t_full_layer, 4),
        "detect_ms": round(kf["detect"], 4),
        "repack_ms": round(t_mid, 4),
        "detect_repack_ms": round(kf["detect"] + t_mid, 4),
        "trunc_gemm_mfma_util": round(tflops(gemm_flop_t, gemm_ms_t) / PEAK_BF16_TFLOPS, 4),
        "kernels": kernels,
        "paper_context": "up to ~31x end-to-end tokens/s (MMaDA, InfoVQA) on 1x NVIDIA A100 "
                         "(context only, different hardware and workload)",
    }
    if args.copy_calibration:
        n = 1 << 28                       # int32 elements: 1 GiB
        log("calibration: 1 GiB fill, then 1 GiB read + 1 GiB write")
        a = torch.ones(n, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        torch.neg(a, out=b)
        torch.cuda.synchronize()
        del a, b
    if not args.no_cpu_baseline and not args.rope:
        log("CPU baseline (oracle on host cores)")
        out["cpu_baseline"] = cpu_baseline(w, layers, batch, args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
        if args.rope:
            out["cpu_baseline_note"] = "the CPU baseline is taken on the layer without rotary embedding"
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
