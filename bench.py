#!/usr/bin/env python3
"""Throughput of the compressed multi-adapter layer (cts_apply) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]

A step is one call of the whole layer (bucketing, shrink, core product, fused
base + up-projection GEMM) over one batch of seeded synthetic inputs that are
already resident in HBM; for the workload stack32 it is one pass over all 224
linear projections of a 32-layer 7B-shaped decoder (q, k, v, o, gate, up,
down) with their own weights: q/k/v and gate/up through one cts_apply_multi
call each (they read the same x), o and down through cts_apply; the same
pass with every projection its own cts_apply call is reported beside it.  The timed region is
K consecutive steps between two HIP events on the stream the library launches
on; the steps are launched call by call.  The same steps replayed from a HIP
graph captured from their calls are reported under "graph_replay": one graph
holds the calls on every rotated input set in turn (for stack32, one whole
step), as a serving loop replays one graph per forward pass; single-layer
lines also give the time with one graph per call ("one_call_graph_ms_per_step"),
which pays the graph's launch every call.  Single-layer inputs are rotated over enough device copies (>= 512 MB in
total) that the 256 MB last-level cache cannot hold them between steps; the
stack's weights (about 32 GB) are distinct per projection anyway.

By default (--workload all) the line's throughput is prefill_mix's (4096
tokens of a 4096 x 4096 projection, 1000 LoRAs in 25 clusters), and the other
four configurations (decode_q, mlp_up, tiny_fp32, stack32) are measured in
the same run and reported under "configs", each with the keys below.

One JSON line is printed.  Besides the throughput it carries:
  roofline        the dominant kernel (the fused GEMM): algorithmic flops or
                  bytes of one launch over its mean duration, measured here
                  with HIP events recorded around it, against MI355X's peak
                  (stack32: all GEMM launches of a step over their summed time)
  cpu_baseline    the fp64 CPU oracle timed on this host on a bounded sample
                  of the same batch (about --cpu-seconds of work)
  uncompressed    the same layer through the uncompressed gather path
                  (cts_apply_uncompressed, rank-16 B_i A_i) on the same batch
  single_adapter  the same batch with every token on one LoRA (n = K = 1);
                  ratio = this throughput / that one
  stages_us       mean duration of each stage of the layer (per step)
  layer_roofline  the whole layer call (all stages, ms_per_step) against the
                  chip: algorithmic flops or bytes of the layer over the step

--workload jd_full measures the offline compressor instead (cts_jd_full, the
eigenvalue iteration of App. A.2 on 1000 rank-16 LoRAs of a 4096 x 4096
projection at r = 64): a step is one iteration over the whole collection, a
timed call runs 10 of them, and the roofline line is the larger of its two
fp32 matrix-core kernels (projection, expansion).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time
import types

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/s and HBM GB/s (or MFMA util) of cts_apply at 1000 LoRAs, one MI355X"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 matrix cores
PEAK_F32_TFLOPS = 157.3        # MI355X dense fp32 matrix cores
MALL_BYTES = 256 << 20


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def to_dev(a, device):
    import numpy as np
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def main_kernel_model(w, touched_clusters, ranks=None):
    """Algorithmic flops and bytes of one launch of the fused GEMM
    Y = W X + U_k Z' (bytes: W, X, Y, each touched U_k once, Z').  With
    `ranks` (a rank per cluster) the U_k terms count r_k columns."""
    e = 2 if w.dtype == "bf16" else 4
    if ranks is None:
        flops = 2.0 * w.T * w.d_in * w.d_out + 2.0 * w.T * w.r * w.d_out
        nbytes = e * (w.d_out * w.d_in + w.T * w.d_in + w.T * w.d_out
                      + touched_clusters * w.d_out * w.r + w.T * w.r)
        return flops, nbytes
    ks = w.cluster_of[w.adapter_id]
    r_tok = ranks[ks].astype(float)
    touched_r = float(sum(ranks[k] for k in set(ks.tolist())))
    flops = 2.0 * w.T * w.d_in * w.d_out + 2.0 * r_tok.sum() * w.d_out
    nbytes = e * (w.d_out * w.d_in + w.T * w.d_in + w.T * w.d_out + touched_r * w.d_out + r_tok.sum())
    return flops, nbytes


def layer_model(T, d_in, d_out, r, e, touched_clusters, distinct_adapters, sigma_elems=None):
    """Algorithmic flops and bytes of one whole layer call: W X + U_k Sigma_i
    V_k^T X with every touched U_k, V_k and Sigma_i read once, X read and Y
    written once (the bucketing's ids and the intermediates Z, Z' are under
    1% and not counted)."""
    sig = r * r if sigma_elems is None else sigma_elems
    flops = 2.0 * T * d_in * d_out + 2.0 * T * (d_in * r + sig + d_out * r)
    nbytes = e * (d_out * d_in + T * d_in + T * d_out + touched_clusters * r * (d_in + d_out)
                  + distinct_adapters * sig)
    return flops, nbytes


def layer_roofline(flops, nbytes, t_s, dtype):
    """The whole layer call against the chip: its algorithmic flops or bytes
    (whichever bound is tighter) over the measured step time."""
    roof = roofline_of(flops, nbytes, t_s, dtype)
    return {"bound": roof["bound"], "achieved": roof["achieved"], "unit": roof["unit"], "frac": roof["frac"],
            "algorithmic_flops": flops, "algorithmic_bytes": nbytes}


def cpu_baseline(w, target_s, sigma=None, ranks=None):
    """The oracle on a prefix of the batch (in batch order), grown until about
    target_s seconds of oracle time; tokens/s = tokens / oracle seconds.  With
    `sigma` ([n][r] diagonals) the diagonal-Sigma oracle is timed, with
    `ranks` (a rank per cluster) the mixed-rank one."""
    import numpy as np
    from oracle import oracle
    f64 = [oracle.to_f64(a) for a in (w.x, w.W, w.U, w.Vt, w.Sigma if sigma is None else sigma)]
    fn = oracle.apply if sigma is None else oracle.apply_diag
    if ranks is not None:
        fn = lambda *a, **k: oracle.apply_ranked(*a[:7], ranks, **k)
    spent, done, chunk = 0.0, 0, min(64, w.T)
    while done < w.T and spent < target_s:
        toks = np.arange(done, min(w.T, done + chunk))
        tm = {}
        fn(f64[0], w.adapter_id, w.cluster_of, f64[1], f64[2], f64[3], f64[4], tokens=toks, timing=tm)
        spent += tm["s"]
        done += len(toks)
        per_tok = spent / done
        chunk = int(max(1, min(w.T - done, (target_s - spent) / per_tok + 1)))
    distinct = len(set(w.adapter_id[:done].tolist()))
    sample = "first %d of %d tokens of the batch (%d distinct adapters)" % (done, w.T, distinct)
    # a batch the oracle finishes early is run again, whole, until about
    # target_s seconds (at most 20 passes)
    passes = 1
    if done == w.T:
        while spent < target_s and passes < 20:
            tm = {}
            fn(f64[0], w.adapter_id, w.cluster_of, f64[1], f64[2], f64[3], f64[4], timing=tm)
            spent += tm["s"]
            done += w.T
            passes += 1
        sample = "the whole batch of %d tokens (%d distinct adapters), %d pass%s" % (
            w.T, distinct, passes, "" if passes == 1 else "es")
    return {"value": done / spent, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": sample + ", %.1f s of fp64 oracle time" % spent}


def copy_calibration(torch, device, nbytes=256 << 20, reps=3):
    """A plain device-to-device copy of known size (read nbytes, write nbytes),
    run outside the timed region.  Under rocprofv3 --pmc its FETCH_SIZE and
    WRITE_SIZE readings give the scale between the counters and real bytes."""
    src = torch.empty(nbytes, dtype=torch.uint8, device=device).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


GEMM_SOURCES = [os.path.join(ROOT, "paper_2407_00066_amd", "csrc", f) for f in ("gemm.hip", "ldsdma.h")]


def traffic_from_profile(workload):
    """HBM bytes per launch of the fused GEMM measured with rocprofv3 --pmc
    (FETCH_SIZE + WRITE_SIZE, each scaled by the copy calibration), read from
    the committed summary of this workload; None when there is none or the
    GEMM's sources (gemm.hip followed by ldsdma.h) have changed since the
    counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_seg_gemm_%s.md" % workload)
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    h = hashlib.sha256()
    for src in GEMM_SOURCES:
        h.update(open(src, "rb").read())
    if fields.get("kernel_source_sha256") != h.hexdigest() or "hbm_bytes_per_launch" not in fields:
        return None
    return float(fields["hbm_bytes_per_launch"])


def time_steps(fn, sets, steps, warmup, torch):
    for i in range(warmup):
        fn(sets[i % len(sets)])
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for i in range(steps):
        fn(sets[i % len(sets)])
    ev1.record()
    torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) / steps          # ms per step


def captured(fn, sets, torch):
    """One HIP graph per input set holding the launches of fn(set) (the
    library allocates, copies and clears nothing inside a call, so a whole
    step is captured); a replay runs the same kernels on the same buffers
    without the host-side work of the calls."""
    torch.cuda.synchronize()
    graphs = []
    for st in sets:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(st)
        graphs.append(g)
    torch.cuda.synchronize()
    return graphs


def time_chain(fn, sets, steps, warmup, torch):
    """ms per step of one HIP graph holding fn(set) for every input set in
    turn, replayed until at least `steps` steps have run: consecutive calls on
    different inputs, as a serving loop replays one graph holding the calls of
    a whole forward pass (the launch of a graph, ~5-10 us on this ROCm, is paid
    once per replay, not once per call)."""
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for st in sets:
            fn(st)
    torch.cuda.synchronize()
    reps = max(1, math.ceil(steps / len(sets)))
    for _ in range(max(1, math.ceil(warmup / len(sets)))):
        g.replay()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(reps):
        g.replay()
    ev1.record()
    torch.cuda.synchronize()
    del g
    return ev0.elapsed_time(ev1) / (reps * len(sets))


def time_launches(fn, sets, args, torch, one_call=False):
    """(eager ms, graph-replay ms) per step: the step launched call by call,
    then from one captured graph holding the calls of every input set in turn;
    with one_call, also (third) one graph per call, replayed call by call."""
    eager = time_steps(fn, sets, args.steps, args.warmup, torch)
    chain = time_chain(fn, sets, args.steps, args.warmup, torch)
    if not one_call:
        return eager, chain
    graphs = captured(fn, sets, torch)
    single = time_steps(lambda g: g.replay(), graphs, args.steps, args.warmup, torch)
    del graphs
    return eager, chain, single


STAGES = ["sort", "shrink", "sigma", "fused_gemm", "splitk_reduce"]


def stage_times(fn, sets, steps, torch, cts):
    """Mean duration (us) of each stage, from events at its boundaries, and
    the marker cost: the interval between the last boundary event and one
    more event recorded right after it with no work between (every stage
    interval holds one such marker interval besides its kernel)."""
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(cts.N_STAGE_EVENTS + 1)]
           for _ in range(steps)]
    for i in range(steps):
        cts.set_stage_events(evs[i][:-1])
        fn(sets[i % len(sets)])
        evs[i][-1].record()
    cts.set_stage_events(None)
    torch.cuda.synchronize()
    out = {}
    for s, name in enumerate(STAGES + ["marker"]):
        out[name] = 1e3 * sum(e[s].elapsed_time(e[s + 1]) for e in evs) / steps
    return out


def gemm_times(fn, sets, steps, warmup, torch, cts):
    """Mean duration (us) of the fused GEMM with the steps run back to back
    as in the timed region, but with only two events around the GEMM, less
    the marker cost: the interval of two events recorded back to back after
    each step.  Returns (gemm interval, marker interval)."""
    n = warmup + steps
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n)]
    for i in range(n):
        e3, e4, ea, eb = evs[i]
        cts.set_stage_events([None, None, None, e3, e4, None])
        fn(sets[i % len(sets)])
        ea.record()
        eb.record()
    cts.set_stage_events(None)
    torch.cuda.synchronize()
    m = evs[warmup:]
    g = 1e3 * sum(e[0].elapsed_time(e[1]) for e in m) / steps
    mk = 1e3 * sum(e[2].elapsed_time(e[3]) for e in m) / steps
    return g, mk


def roofline_of(flops, nbytes, t_s, dtype):
    peak_fl = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS
    if flops / (peak_fl * 1e12) >= nbytes / (PEAK_HBM_GBS * 1e9):
        achieved = flops / t_s / 1e12
        return {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak_fl, "unit": "TFLOP/s",
                "frac": round(achieved / peak_fl, 4), "traffic": None}
    achieved = nbytes / t_s / 1e9
    return {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None}


JD_N, JD_D, JD_RL, JD_R, JD_ITERS = 1000, 4096, 16, 64, 10


def jd_kernel_models(n, d_out, d_in, r_l, r, split):
    """Algorithmic flops and bytes of one iteration's two large stages
    (fp32).  projection: P_i = A_i V, Q_i = B_i^T U, G_i = P_i P_i^T,
    H_i = Q_i Q_i^T, C_i = G_i Q_i, D_i = H_i P_i (reads A, B, the bases;
    writes C, D).  expand: U' = sum_i B_i C_i, V' = sum_i A_i^T D_i (reads A,
    B, C, D; writes the split partials)."""
    rows = n * r_l
    proj_f = 2.0 * rows * r * (d_in + d_out) + 2 * (4.0 * n * r_l * r_l * r)
    proj_b = 4.0 * (rows * (d_in + d_out) + r * (d_in + d_out) + 2 * rows * r)
    exp_f = 2.0 * rows * r * (d_in + d_out)
    exp_b = 4.0 * (rows * (d_in + d_out) + 2 * rows * r + split * r * (d_in + d_out))
    return (proj_f, proj_b), (exp_f, exp_b)


def jd_diag_kernel_models(n, d_out, d_in, r_l, r, split):
    """Flops and bytes of the JD-Diag sweep's U-step stages: projection of
    one half (P_i = A_i V, C_i = P_i S_i: reads A and V, writes C) and the
    expansion of one half (U' = sum_i B_i C_i: reads B and C, writes the
    split partials)."""
    rows = n * r_l
    proj = (2.0 * rows * r * d_in + rows * r, 4.0 * (rows * d_in + r * d_in + rows * r))
    expd = (2.0 * rows * r * d_out, 4.0 * (rows * d_out + rows * r + split * r * d_out))
    return proj, expd


def bench_jd(args, torch, np, cts, B, device):
    """One step = one iteration of the App. A.2 eigenvalue iteration over the
    whole collection (1000 rank-16 LoRAs of a 4096 x 4096 projection, r = 64);
    a timed call runs the paper's 10 iterations (no early stop).  With
    --workload jd_diag a step is one sweep of the JD-Diag alternating least
    squares (App. A.1 case 2) from random bases, 10 sweeps per call."""
    from paper_2407_00066_amd import compress as GC
    n, d, r_l, r, iters = JD_N, JD_D, JD_RL, JD_R, JD_ITERS
    log("generating %d LoRAs of rank %d, %d x %d" % (n, r_l, d, d))
    rs = np.random.default_rng(2407)
    A = rs.standard_normal((n, r_l, d), dtype=np.float32) / np.float32(64.0)
    Bm = rs.standard_normal((n, d, r_l), dtype=np.float32) / np.float32(4.0)
    U0 = np.linalg.qr(rs.standard_normal((d, r)))[0].astype(np.float32)
    V0 = np.linalg.qr(rs.standard_normal((d, r)))[0].astype(np.float32)
    gA, gB = to_dev(A, device), to_dev(Bm, device)
    gU0, gVt0 = to_dev(U0, device), to_dev(np.ascontiguousarray(V0.T), device)
    ws = torch.empty(GC.workspace_size(gA, gB, r), dtype=torch.uint8, device=device)

    diag = args.workload == "jd_diag"
    if diag:
        gU0 = to_dev((rs.standard_normal((d, r)) / np.sqrt(d)).astype(np.float32), device)
        gVt0 = to_dev((rs.standard_normal((r, d)) / np.sqrt(d)).astype(np.float32), device)

    def call():
        if diag:
            return GC.jd_diag(gA, gB, gU0, gVt0, sweeps=iters, workspace=ws)
        return GC.jd_full(gA, gB, gU0, gVt0, iters=iters, workspace=ws)

    log("timing %s: %d warmup + %d calls of %d steps" % ("cts_jd_diag" if diag else "cts_jd_full", args.warmup,
                                                         args.steps, iters))
    ms_call = time_steps(lambda _: call(), [None], args.steps, args.warmup, torch)
    ms_iter = ms_call / iters
    # the two large kernels of the last iteration of each call, between stage
    # events, less the interval of two back-to-back events
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    for i in range(args.steps):
        e1, e2, e3, ea, eb = evs[i]
        B.set_stage_events([None, e1, e2, e3, None, None])
        call()
        ea.record()
        eb.record()
    B.set_stage_events(None)
    torch.cuda.synchronize()
    mk = 1e3 * sum(e[3].elapsed_time(e[4]) for e in evs) / args.steps
    proj_us = 1e3 * sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps - mk
    exp_us = 1e3 * sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps - mk
    # the expansion's pieces of the collection, as the library picks them:
    # the fewest that fill the resident slots (256 CUs x 3 workgroups at
    # r = 64) within 5%, at most 16 and at least 8 k-tiles each
    rowt = (d + 63) // 64
    ntile = (n * r_l + 31) // 32
    occ = 4 if r <= 32 else (3 if r <= 64 else 2)
    base = rowt * (1 if diag else 2)
    split, best = 1, 0.0
    for s_ in range(1, max(1, min(16, ntile // 8)) + 1):
        w_ = base * s_
        eff = w_ / (-(-w_ // (256 * occ)) * 256 * occ)
        if eff > best + 0.05:
            split, best = s_, eff
    if diag:
        (pf, pb), (ef, eb_) = jd_diag_kernel_models(n, d, d, r_l, r, split)
        if exp_us >= proj_us:
            name, fl, nb, us = "jd_expand_kernel, U step (U' = sum B_i C_i)", ef, eb_, exp_us
        else:
            name, fl, nb, us = ("projection, U step: jd_pq_kernel + jd_combine_kernel (A_i V, C_i = P_i S_i)",
                                pf, pb, proj_us)
    else:
        (pf, pb), (ef, eb_) = jd_kernel_models(n, d, d, r_l, r, split)
        if exp_us >= proj_us:
            name, fl, nb, us = "jd_expand_kernel (U' = sum B_i C_i, V' = sum A_i^T D_i)", ef, eb_, exp_us
        else:
            name, fl, nb, us = ("projection: jd_pq_kernel + jd_combine_kernel (A_i V, B_i^T U, per-LoRA "
                                "products)", pf, pb, proj_us)
    roof = roofline_of(fl, nb, us * 1e-6, "f32")
    roof.update({"kernel": name, "mean_us": round(us, 2), "marker_us": round(mk, 2),
                 "algorithmic_flops": fl, "algorithmic_bytes": nb,
                 "project_us": round(proj_us, 2), "expand_us": round(exp_us, 2)})
    cpu = None
    if not args.no_cpu_baseline and not diag:
        cpu = jd_cpu_baseline(A, Bm, U0, V0, args.cpu_seconds)
    if diag:
        cpu = None if args.no_cpu_baseline else jd_diag_cpu_baseline(A, Bm, host_of(gU0), host_of(gVt0).T,
                                                                       args.cpu_seconds)
    return {
        "metric": ("LoRA-sweeps/s of the JD-Diag alternating least squares" if diag else
                   "LoRA-iterations/s of the JD-Full eigenvalue iteration") +
                  " (1000 rank-16 LoRAs, 4096 x 4096, r = 64), one MI355X",
        "value": round(n * iters / (ms_call * 1e-3), 1), "unit": "LoRA-sweeps/s" if diag else "LoRA-iterations/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_iter, 5), "ms_per_compression": round(ms_call, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded Gaussian LoRAs; random %s initial bases)" % ("Gaussian" if diag else "orthonormal"),
        "config": {"workload": args.workload, "n_loras": n, "d_out": d, "d_in": d, "r_lora": r_l, "r": r,
                   ("sweeps" if diag else "iterations"): iters, "parallelism": "single GPU"},
        "roofline": roof, "cpu_baseline": cpu,
    }


def host_of(t):
    return t.detach().cpu().numpy().astype("float64")


def jd_diag_cpu_baseline(A, Bm, U0, V0, target_s):
    """The oracle's JD-Diag sweep (fp64) on the first LoRAs of the collection,
    grown until about target_s / 4 seconds or 32 LoRAs (it forms every
    d_out x d_in update B_i A_i, 134 MB each here); LoRA-sweeps/s."""
    import numpy as np
    from oracle import compress as OC
    m = 4
    while True:
        a, b = A[:m].astype(np.float64), Bm[:m].astype(np.float64)
        t0 = time.perf_counter()
        OC.jd_diag_als(a, b, U0.shape[1], U0, V0, sweeps=1)
        dt = time.perf_counter() - t0
        if dt >= target_s / 4 or m >= min(32, A.shape[0]):
            break
        m = min(32, A.shape[0], int(m * max(2.0, target_s / 4 / max(dt, 1e-3))))
    try:
        from threadpoolctl import threadpool_info
        cores = max([t.get("num_threads", 1) for t in threadpool_info() if t.get("user_api") == "blas"] or [1])
    except ImportError:
        cores = os.cpu_count()
    return {"value": m / dt, "unit": "LoRA-sweeps/s", "cores": cores, "kind": "oracle",
            "sample": "one fp64 JD-Diag sweep (plus its initial diagonals) over the first %d of %d LoRAs, %.1f s"
                      % (m, A.shape[0], dt)}


def jd_cpu_baseline(A, Bm, U0, V0, target_s):
    """The oracle's eigenvalue-iteration step (fp64) on the first LoRAs of the
    collection, grown until about target_s seconds; LoRA-iterations/s."""
    import numpy as np
    from oracle import compress as OC
    from oracle import oracle
    U, V = U0.astype(np.float64), V0.astype(np.float64)
    spent, m = 0.0, 16
    while True:
        a, b = A[:m].astype(np.float64), Bm[:m].astype(np.float64)
        t0 = time.perf_counter()
        OC.eig_step(a, b, U, V)
        dt = time.perf_counter() - t0
        if dt >= target_s / 4 or m >= A.shape[0]:
            spent = dt
            break
        m = min(A.shape[0], int(m * max(2.0, target_s / 4 / max(dt, 1e-3))))
    try:
        from threadpoolctl import threadpool_info
        cores = max([t.get("num_threads", 1) for t in threadpool_info() if t.get("user_api") == "blas"] or [1])
    except ImportError:
        cores = oracle.num_threads()
    return {"value": m / spent, "unit": "LoRA-iterations/s", "cores": cores, "kind": "oracle",
            "sample": "one fp64 eigenvalue-iteration step over the first %d of %d LoRAs, %.1f s"
                      % (m, A.shape[0], spent)}


def bench_layer(args, torch, np, cts, B, wl, device):
    log("generating %s" % args.workload)
    w = wl.make(args.workload)
    diag = args.sigma == "diag"
    cfg = wl.CONFIGS[args.workload]["cfg"]
    if diag:   # the diagonal-Sigma variant (Sec. 3.1, JD-Diag): Sigma holds [n][r] diagonals
        w.Sigma = wl.sigma_diagonals(cfg, w.n, w.r, w.dtype)
    layer = layer1 = cts.apply_diag if diag else cts.apply
    rk = ra = None
    if args.ranks == "mixed":   # a rank per cluster (Sec. 3.2), per uncompressed LoRA (App. H)
        rk = wl.mixed_ranks(cfg, w.K, w.r)
        ra = wl.mixed_ranks(cfg + 500, w.n, w.r_l, lo=8)
        rk_d, ra_d = to_dev(rk, device), to_dev(ra, device)
        layer = lambda *a, **k: cts.apply_ranked(*a, rk_d, **k)
        # the one-adapter comparison keeps cluster 0 and its rank
        layer1 = lambda *a, **k: cts.apply_ranked(*a, rk_d[:1], **k)

    set_bytes = sum(a.nbytes for a in (w.x, w.W, w.U, w.Vt, w.Sigma))
    # (at most 64: a set that small stays in the last-level cache whatever
    # the rotation, and its launches, not its bytes, set the pace)
    n_sets = min(64, max(1, math.ceil(2 * MALL_BYTES / set_bytes)))
    base = [to_dev(a, device) for a in (w.x, w.W, w.U, w.Vt, w.Sigma)]
    sets = [base] + [[t.clone() for t in base] for _ in range(n_sets - 1)]
    aid = to_dev(w.adapter_id, device)
    cof = to_dev(w.cluster_of, device)
    y = torch.empty((w.T, w.d_out), dtype=base[0].dtype, device=device)
    dt = B.CTS_BF16 if w.dtype == "bf16" else B.CTS_F32
    p = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=w.n, n_clusters=w.K, dtype=dt)
    ws = torch.empty(max(1, cts.workspace_size(p)), dtype=torch.uint8, device=device)

    def step(s):
        x, W, U, Vt, S = s
        layer(x, aid, cof, W, U, Vt, S, out=y, workspace=ws)

    log("timing cts_apply: %d sets of %.1f MB, %d warmup + %d steps" %
        (n_sets, set_bytes / 1e6, args.warmup, args.steps))
    ms, ms_g, ms_g1 = time_launches(step, sets, args, torch, one_call=True)
    stages = stage_times(step, sets, args.steps, torch, B)
    g_int, g_mark = gemm_times(step, sets, args.steps, args.warmup, torch, B)

    # one adapter: the same batch, every token on LoRA 0 of cluster 0
    aid1 = torch.zeros_like(aid)
    cof1 = torch.zeros(1, dtype=torch.int32, device=device)
    p1 = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=1, n_clusters=1, dtype=dt)
    ws1 = torch.empty(max(1, cts.workspace_size(p1)), dtype=torch.uint8, device=device)

    def step1(s):
        x, W, U, Vt, S = s
        layer1(x, aid1, cof1, W, U[:1], Vt[:1], S[:1], out=y, workspace=ws1)

    log("timing cts_apply with one adapter")
    ms1, ms1_g = time_launches(step1, sets, args, torch)

    # uncompressed comparison on the same batch
    uA, uB = to_dev(w.A, device), to_dev(w.B, device)
    pu = cts.make_problem(w.T, w.d_in, w.d_out, n_adapters=w.n, r_lora=w.r_l, dtype=dt)
    wsu = torch.empty(max(1, cts.workspace_size(pu, compressed=False)), dtype=torch.uint8, device=device)

    def step_u(s):
        x, W = s[0], s[1]
        if ra is None:
            cts.apply_uncompressed(x, aid, W, uA, uB, out=y, workspace=wsu)
        else:
            cts.apply_uncompressed_ranked(x, aid, W, uA, uB, ra_d, out=y, workspace=wsu)

    log("timing cts_apply_uncompressed")
    ms_u, ms_u_g = time_launches(step_u, sets, args, torch)
    stages_u = stage_times(step_u, sets, args.steps, torch, B)
    del uA, uB

    touched = len(set(w.cluster_of[w.adapter_id].tolist()))
    flops, nbytes = main_kernel_model(w, touched, rk)
    # the GEMM's duration: its event interval less the marker interval
    gemm_us = g_int - g_mark
    roof = roofline_of(flops, nbytes, gemm_us * 1e-6, w.dtype)
    roof["traffic"] = traffic_from_profile(args.workload)
    gemm_kernel = "seg_gemm_dma_kernel" if w.dtype == "bf16" else "seg_gemm_kernel"
    roof.update({"kernel": gemm_kernel + " (fused W X + U_k Z')", "mean_us": round(gemm_us, 2),
                 "event_interval_us": round(g_int, 2), "marker_us": round(g_mark, 2),
                 "algorithmic_flops": flops, "algorithmic_bytes": nbytes})

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (about %.0f s)" % args.cpu_seconds)
        cpu = cpu_baseline(w, args.cpu_seconds, sigma=w.Sigma if diag else None, ranks=rk)

    value = w.T / (ms * 1e-3)
    value1 = w.T / (ms1 * 1e-3)
    distinct = len(set(w.adapter_id.tolist()))
    lf, lb = layer_model(w.T, w.d_in, w.d_out, w.r, 2 if w.dtype == "bf16" else 4, touched, distinct,
                         sigma_elems=w.r if diag else None)
    return {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "graph_replay": {"value": round(w.T / (ms_g * 1e-3), 1), "ms_per_step": round(ms_g, 5),
                         "calls_per_graph": len(sets), "one_call_graph_ms_per_step": round(ms_g1, 5)},
        "dtype": w.dtype, "data": "synthetic (seeded; inputs resident in HBM, rotated over %d copies)" % n_sets,
        "config": {"workload": args.workload, "sigma": args.sigma, "ranks": args.ranks,
                   "cluster_ranks": None if rk is None else rk.tolist(), "T": w.T, "d_in": w.d_in, "d_out": w.d_out, "r": w.r,
                   "n_adapters": w.n, "n_clusters": w.K, "touched_clusters": touched,
                   "distinct_adapters": len(set(w.adapter_id.tolist())), "parallelism": "single GPU"},
        "roofline": roof,
        "layer_roofline": layer_roofline(lf, lb, ms * 1e-3, w.dtype),
        "cpu_baseline": cpu,
        "uncompressed": {"value": round(w.T / (ms_u * 1e-3), 1), "unit": "tokens/s",
                         "ms_per_step": round(ms_u, 5), "graph_replay_ms_per_step": round(ms_u_g, 5),
                         "r_lora": w.r_l,
                         "stages_us": {k: round(v, 2) for k, v in stages_u.items()}},
        "single_adapter": {"value": round(value1, 1), "unit": "tokens/s", "ms_per_step": round(ms1, 5),
                           "graph_replay_ms_per_step": round(ms1_g, 5), "ratio": round(value / value1, 4)},
        "stages_us": {k: round(v, 2) for k, v in stages.items()},
    }


def stack_cpu_baseline(projs, aid_h, cof_h, target_s, torch, np):
    """The oracle on the first layer's projections, one of each shape, for a
    prefix of the batch; the stack's tokens/s is extrapolated as tokens over
    the summed per-token oracle time of all 224 projections."""
    from oracle import oracle
    from paper_2407_00066_amd import workloads as wl
    per_tok, cores, detail = {}, oracle.num_threads(), []
    budget = target_s / 4
    for name, d_in, d_out in wl.STACK_PROJ:
        shape = (d_in, d_out)
        if shape in per_tok:
            continue
        x, W, U, Vt, S = projs[0][name][:5]
        host = [t.view(torch.int16).cpu().numpy().view(np.uint16) for t in (x, W, U, Vt, S)]
        f64 = [oracle.to_f64(a) for a in host]
        spent, done, chunk = 0.0, 0, 2
        while done < len(aid_h) and spent < budget:
            toks = np.arange(done, min(len(aid_h), done + chunk))
            tm = {}
            oracle.apply(f64[0], aid_h, cof_h, f64[1], f64[2], f64[3], f64[4], tokens=toks, timing=tm)
            spent += tm["s"]
            done += len(toks)
            chunk = max(1, min(len(aid_h) - done, int((budget - spent) / (spent / done)) + 1))
        per_tok[shape] = spent / done
        detail.append("%dx%d: %d tokens in %.1f s" % (d_in, d_out, done, spent))
    t_tok = wl.STACK_LAYERS * sum(per_tok[(d_in, d_out)] for _, d_in, d_out in wl.STACK_PROJ)
    return {"value": 1.0 / t_tok, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": "layer-0 projections, one per shape (%s), per-token time x 32 layers x 7 "
                      "projections" % "; ".join(detail)}


def bench_stack(args, torch, np, cts, B, wl, device):
    T, r, n, K = wl.STACK["T"], wl.STACK["r"], wl.STACK["n"], wl.STACK["K"]
    aid_h, cof_h = wl.stack_ids()
    aid, cof = to_dev(aid_h, device), to_dev(cof_h, device)

    log("generating the 32-layer stack on the device")
    xs = {4096: wl.stack_x(torch, device, 4096), 14336: wl.stack_x(torch, device, 14336)}
    x_o = wl.stack_x_o(torch, device)
    ys = {d: torch.empty((T, d), dtype=torch.bfloat16, device=device) for d in (1024, 4096, 14336)}
    projs, wsz = [], 1
    for li in range(wl.STACK_LAYERS):
        layer = {}
        for name, d_in, d_out in wl.STACK_PROJ:
            layer[name] = ((x_o if name == "o" else xs[d_in]),) + wl.stack_module(torch, device, li, name) + \
                (ys[d_out],)
            pb = cts.make_problem(T, d_in, d_out, r=r, n_adapters=n, n_clusters=K, dtype=B.CTS_BF16)
            wsz = max(wsz, cts.workspace_size(pb))
        projs.append(layer)
    # multi-module batching: q/k/v and gate/up each read one x; their V_k^T
    # stacked along r (separate outputs, since the modules run in one call)
    groups = (("q", "k", "v"), ("gate", "up"))
    extra_y = {("k",): torch.empty((T, 1024), dtype=torch.bfloat16, device=device),
               ("v",): torch.empty((T, 1024), dtype=torch.bfloat16, device=device),
               ("up",): torch.empty((T, 14336), dtype=torch.bfloat16, device=device)}
    stacked = []
    for L in projs:
        stacked.append({grp: torch.cat([L[nm][3] for nm in grp], dim=1).contiguous() for grp in groups})
    outs_of = {("q", "k", "v"): [ys[4096], extra_y[("k",)], extra_y[("v",)]],
               ("gate", "up"): [ys[14336], extra_y[("up",)]]}
    wszm = wszm1 = 1
    for grp in groups + (("o",), ("down",)):
        d_in = dict((nm, di) for nm, di, _ in wl.STACK_PROJ)[grp[0]]
        dims = [dict((nm, do) for nm, _, do in wl.STACK_PROJ)[g_] for g_ in grp]
        pm = cts.make_problem(T, d_in, 8, r=r, n_adapters=n, n_clusters=K, dtype=B.CTS_BF16)
        wszm = max(wszm, cts.workspace_size_multi(pm, dims))
        pm1 = cts.make_problem(T, d_in, 8, r=r, n_adapters=1, n_clusters=1, dtype=B.CTS_BF16)
        wszm1 = max(wszm1, cts.workspace_size_multi(pm1, dims))
    torch.cuda.synchronize()
    ws = torch.empty(wsz, dtype=torch.uint8, device=device)
    wsm = torch.empty(wszm, dtype=torch.uint8, device=device)
    wsm1 = torch.empty(wszm1, dtype=torch.uint8, device=device)
    # one bucketing of the batch for the whole step (every projection shares
    # the cluster map): perm and the sort's workspace
    perm_s = torch.empty(T, dtype=torch.int32, device=device)
    offs_s = torch.empty(K + 1, dtype=torch.int32, device=device)
    bk = torch.empty(cts.bucketing_size(T, n, K), dtype=torch.uint8, device=device)
    perm_1 = torch.empty(T, dtype=torch.int32, device=device)
    offs_1 = torch.empty(2, dtype=torch.int32, device=device)
    bk1 = torch.empty(cts.bucketing_size(T, 1, 1), dtype=torch.uint8, device=device)
    aid1 = torch.zeros_like(aid)
    cof1 = torch.zeros(1, dtype=torch.int32, device=device)
    resident = sum(t.numel() * t.element_size() for L in projs for v in L.values() for t in v[1:5])

    def step(_):
        for L in projs:
            for name, _, _ in wl.STACK_PROJ:
                x, W, U, Vt, S, y = L[name]
                cts.apply(x, aid, cof, W, U, Vt, S, out=y, workspace=ws)

    def step_multi(_):
        for L, SV in zip(projs, stacked):
            for grp in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
                if len(grp) == 1:
                    x, W, U, Vt, S, y = L[grp[0]]
                    cts.apply(x, aid, cof, W, U, Vt, S, out=y, workspace=ws)
                else:
                    cts.apply_multi(L[grp[0]][0], aid, cof, [L[nm][1] for nm in grp], [L[nm][2] for nm in grp],
                                    SV[grp], [L[nm][4] for nm in grp], outs=outs_of[grp], workspace=wsm)

    def step_shared(_):
        cts.sort_by_cluster(aid, cof, n, K, perm=perm_s, offsets=offs_s, bucketing=bk)
        for L, SV in zip(projs, stacked):
            for grp in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
                if len(grp) == 1:
                    x, W, U, Vt, S, y = L[grp[0]]
                    cts.apply_multi_sorted(perm_s, bk, x, [W], [U], Vt, [S], outs=[y], workspace=wsm)
                else:
                    cts.apply_multi_sorted(perm_s, bk, L[grp[0]][0], [L[nm][1] for nm in grp],
                                           [L[nm][2] for nm in grp], SV[grp], [L[nm][4] for nm in grp],
                                           outs=outs_of[grp], workspace=wsm)

    def step1(_):
        # the same calls with every token on LoRA 0 of cluster 0 (n = K = 1)
        cts.sort_by_cluster(aid1, cof1, 1, 1, perm=perm_1, offsets=offs_1, bucketing=bk1)
        for L, SV in zip(projs, stacked):
            for grp in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",)):
                if len(grp) == 1:
                    x, W, U, Vt, S, y = L[grp[0]]
                    cts.apply_multi_sorted(perm_1, bk1, x, [W], [U[:1]], Vt[:1], [S[:1]], outs=[y], workspace=wsm1)
                else:
                    cts.apply_multi_sorted(perm_1, bk1, L[grp[0]][0], [L[nm][1] for nm in grp],
                                           [L[nm][2][:1] for nm in grp], SV[grp][:1], [L[nm][4][:1] for nm in grp],
                                           outs=outs_of[grp], workspace=wsm1)

    log("timing the stack: %.1f GB of weights, %d warmup + %d steps" % (resident / 1e9, args.warmup, args.steps))
    ms_sep, ms_sep_g = time_launches(step, [None], args, torch)
    log("timing the stack with q/k/v and gate/up batched (cts_apply_multi), a sort per call")
    ms_m, ms_m_g = time_launches(step_multi, [None], args, torch)
    log("timing the stack with one sort per step (cts_apply_multi_sorted)")
    ms, ms_g = time_launches(step_shared, [None], args, torch)
    log("timing the stack with one adapter")
    ms1, ms1_g = time_launches(step1, [None], args, torch)

    # the uncompressed comparison: every projection with its 1000 rank-16
    # LoRAs (A_i, B_i) resident, one cts_apply_uncompressed call each
    r_l = 16
    log("generating the stack's uncompressed LoRAs on the device")
    loras = [{name: wl.stack_lora(torch, device, li, name, r_l) for name, _, _ in wl.STACK_PROJ}
             for li in range(wl.STACK_LAYERS)]
    lora_bytes = sum(t.numel() * t.element_size() for L in loras for v in L.values() for t in v)
    wszu = 1
    for name, d_in, d_out in wl.STACK_PROJ:
        pu = cts.make_problem(T, d_in, d_out, n_adapters=n, r_lora=r_l, dtype=B.CTS_BF16)
        wszu = max(wszu, cts.workspace_size(pu, compressed=False))
    wsu = torch.empty(wszu, dtype=torch.uint8, device=device)

    def step_u(_):
        for L, LA in zip(projs, loras):
            for name, _, _ in wl.STACK_PROJ:
                x, W, _U, _V, _S, y = L[name]
                A_, B_ = LA[name]
                cts.apply_uncompressed(x, aid, W, A_, B_, out=y, workspace=wsu)

    log("timing the uncompressed stack: %.1f GB of LoRAs" % (lora_bytes / 1e9))
    ms_u, ms_u_g = time_launches(step_u, [None], args, torch)
    del loras, wsu
    torch.cuda.empty_cache()

    # per-call stage events over a few steps: the GEMM time of a step
    n_ev = min(args.steps, 3)
    calls = wl.STACK_LAYERS * len(wl.STACK_PROJ)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(B.N_STAGE_EVENTS + 1)]
           for _ in range(calls * n_ev)]
    c = 0
    for _ in range(n_ev):
        for L in projs:
            for name, _, _ in wl.STACK_PROJ:
                x, W, U, Vt, S, y = L[name]
                B.set_stage_events(evs[c][:-1])
                cts.apply(x, aid, cof, W, U, Vt, S, out=y, workspace=ws)
                evs[c][-1].record()
                c += 1
    B.set_stage_events(None)
    torch.cuda.synchronize()
    stages = {nm: 1e3 * sum(e[i].elapsed_time(e[i + 1]) for e in evs) / n_ev
              for i, nm in enumerate(STAGES + ["marker"])}
    # the GEMM alone: two events around each GEMM launch, and a back-to-back
    # pair after each call for the marker cost
    gev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(calls * n_ev)]
    c = 0
    for _ in range(n_ev):
        for L in projs:
            for name, _, _ in wl.STACK_PROJ:
                x, W, U, Vt, S, y = L[name]
                e3, e4, ea, eb = gev[c]
                B.set_stage_events([None, None, None, e3, e4, None])
                cts.apply(x, aid, cof, W, U, Vt, S, out=y, workspace=ws)
                ea.record()
                eb.record()
                c += 1
    B.set_stage_events(None)
    torch.cuda.synchronize()
    g_int = 1e3 * sum(e[0].elapsed_time(e[1]) for e in gev) / n_ev          # per step
    g_mark = 1e3 * sum(e[2].elapsed_time(e[3]) for e in gev) / n_ev

    touched = len(set(cof_h[aid_h].tolist()))
    flops = nbytes = 0.0
    for name, d_in, d_out in wl.STACK_PROJ:
        f, b = main_kernel_model(types.SimpleNamespace(T=T, d_in=d_in, d_out=d_out, r=r, dtype="bf16"),
                                 touched)
        flops += f * wl.STACK_LAYERS
        nbytes += b * wl.STACK_LAYERS
    gemm_us = g_int - g_mark          # per step: over all calls, (GEMM interval - marker)
    roof = roofline_of(flops, nbytes, gemm_us * 1e-6, "bf16")
    roof.update({"kernel": "seg_gemm_dma_kernel (fused W X + U_k Z'), all %d launches of a step" % calls,
                 "mean_us": round(gemm_us / calls, 2), "event_interval_us": round(g_int / calls, 2),
                 "marker_us": round(g_mark / calls, 2),
                 "algorithmic_flops": flops, "algorithmic_bytes": nbytes})
    lf = lb = 0.0
    distinct = len(set(aid_h.tolist()))
    for name, d_in, d_out in wl.STACK_PROJ:
        f, b = layer_model(T, d_in, d_out, r, 2, touched, distinct)
        lf += f * wl.STACK_LAYERS
        lb += b * wl.STACK_LAYERS
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (about %.0f s)" % args.cpu_seconds)
        cpu = stack_cpu_baseline(projs, aid_h, cof_h, args.cpu_seconds, torch, np)
    value, value1 = T / (ms * 1e-3), T / (ms1 * 1e-3)
    return {
        "separate_calls": {"value": round(T / (ms_sep * 1e-3), 1), "ms_per_step": round(ms_sep, 5),
                           "graph_replay_ms_per_step": round(ms_sep_g, 5),
                           "note": "every projection its own cts_apply call"},
        "sort_per_call": {"value": round(T / (ms_m * 1e-3), 1), "ms_per_step": round(ms_m, 5),
                          "graph_replay_ms_per_step": round(ms_m_g, 5),
                          "note": "q/k/v and gate/up per cts_apply_multi call, o and down per cts_apply call, "
                                  "each call sorting the ids itself"},
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "graph_replay": {"value": round(T / (ms_g * 1e-3), 1), "ms_per_step": round(ms_g, 5)},
        "dtype": "bf16",
        "data": "synthetic (seeded, generated on the device; %.1f GB of weights resident in HBM)" % (resident / 1e9),
        "config": {"workload": "stack32", "T": T, "layers": wl.STACK_LAYERS,
                   "batching": "one cts_sort_by_cluster per step; q/k/v and gate/up per "
                               "cts_apply_multi_sorted call (V_k^T stacked), o and down per call of their own",
                   "projections": [list(pr) for pr in wl.STACK_PROJ], "r": r, "n_adapters": n,
                   "n_clusters": K, "touched_clusters": touched,
                   "distinct_adapters": len(set(aid_h.tolist())), "parallelism": "single GPU"},
        "roofline": roof,
        "layer_roofline": layer_roofline(lf, lb, ms * 1e-3, "bf16"),
        "cpu_baseline": cpu,
        "single_adapter": {"value": round(value1, 1), "unit": "tokens/s", "ms_per_step": round(ms1, 5),
                           "graph_replay_ms_per_step": round(ms1_g, 5), "ratio": round(value / value1, 4)},
        "uncompressed": {"value": round(T / (ms_u * 1e-3), 1), "unit": "tokens/s", "ms_per_step": round(ms_u, 5),
                         "graph_replay_ms_per_step": round(ms_u_g, 5), "r_lora": r_l,
                         "resident_lora_gb": round(lora_bytes / 1e9, 1),
                         "note": "every projection its own cts_apply_uncompressed call"},
        "stages_us": {k: round(v, 2) for k, v in stages.items()},
    }


# Every configuration of the layer: the headline line (prefill_mix) carries
# the other four under "configs", each measured the same way in this run.
ALL_CONFIGS = ("decode_q", "mlp_up", "tiny_fp32", "stack32")
SUB_KEYS = ("value", "unit", "ms_per_step", "graph_replay", "dtype", "data", "config", "roofline",
            "layer_roofline", "cpu_baseline", "uncompressed", "single_adapter", "separate_calls", "sort_per_call",
            "stages_us")


def bench_all(args, torch, np, cts, B, wl, device):
    import copy
    import gc
    a = copy.copy(args)
    a.workload = "prefill_mix"
    rec = bench_layer(a, torch, np, cts, B, wl, device)
    rec["configs"] = {}
    for name in ALL_CONFIGS:
        gc.collect()
        torch.cuda.empty_cache()
        a = copy.copy(args)
        a.workload = name
        t0 = time.time()
        sub = bench_stack(a, torch, np, cts, B, wl, device) if name == "stack32" else \
            bench_layer(a, torch, np, cts, B, wl, device)
        sub = {k: sub[k] for k in SUB_KEYS if k in sub}
        sub["steps"], sub["warmup"] = a.steps, a.warmup
        sub["bench_seconds"] = round(time.time() - t0, 1)
        rec["configs"][name] = sub
        log("%s: %.1f tokens/s, %.5f ms per step" % (name, sub["value"], sub["ms_per_step"]))
    gc.collect()
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="all",
                    choices=["all", "prefill_mix", "decode_q", "mlp_up", "tiny_fp32", "stack32", "jd_full",
                             "jd_diag"],
                    help="all (the default): prefill_mix as the headline line, the other four "
                         "configurations under its key 'configs'")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sigma", default="full", choices=["full", "diag"],
                    help="full r x r Sigma_i (JD-Full, the default) or diagonal Sigma_i "
                         "(JD-Diag, cts_apply_diag); single-layer workloads only")
    ap.add_argument("--ranks", default="uniform", choices=["uniform", "mixed"],
                    help="one rank r for every cluster (default) or a rank per cluster drawn in "
                         "[16, r] and per uncompressed LoRA in [8, r_l] (cts_apply_ranked); "
                         "single-layer workloads with the full Sigma only")
    args = ap.parse_args()

    if args.sigma == "diag" and args.ranks == "mixed":
        print("--sigma diag and --ranks mixed are separate variants", file=sys.stderr)
        sys.exit(2)
    if args.workload in ("all", "stack32", "jd_full", "jd_diag") and (args.sigma != "full" or args.ranks != "uniform"):
        print("--sigma diag and --ranks mixed apply to the single-layer workloads", file=sys.stderr)
        sys.exit(2)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X (the layer's tokens would shard across GPUs with no "
              "communication inside the layer; that path is not run here); run it with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2407_00066_amd as cts
    from paper_2407_00066_amd import _binding as B
    from paper_2407_00066_amd import workloads as wl

    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    copy_calibration(torch, device)
    if args.workload in ("jd_full", "jd_diag"):
        rec = bench_jd(args, torch, np, cts, B, device)
    elif args.workload == "all":
        rec = bench_all(args, torch, np, cts, B, wl, device)
    elif args.workload == "stack32":
        rec = bench_stack(args, torch, np, cts, B, wl, device)
    else:
        rec = bench_layer(args, torch, np, cts, B, wl, device)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
