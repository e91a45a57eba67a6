#!/usr/bin/env python3
"""Benchmark of the ProtoKV far-memory hot path on one MI355X.

Headline workload (`--workload multi`, the default): 64 concurrent streams of
a 7B-class video LLM on one GPU, each 28 layers x 4 KV heads (28 query
heads), head_dim 128, bf16 KV, 196 visual tokens per frame on a 14x14 grid,
near window 8 frames, K = 512 prototypes per (stream, layer, kv head) unit;
frames are appended round-robin (one batched append gives every stream one
frame), and stream b issues a 32-token query at the rounds r with
(r - 2b) mod 128 = 127, so every stream queries once per 128 frames and one
query lands on every other round.  Seeded synthetic frames are drawn on the
GPU outside the timed region (the paper's video datasets stand in).

A step = one round: every stream's frame appended to its near window, the
evicted frames folded into the banks (seed / screen + assign / aggregate),
and the queries due in that round (synthesize + attend).  Before anything is
timed the windows and banks are filled (W + ceil(K / T) + 1 frames per
stream, always, whatever --warmup says), then --warmup more steady-state
rounds run untimed, then --profile-frames rounds with every launch timed by
library HIP events (to find the dominant kernel), then the timed region of
--steps rounds.  `value` = evicted model tokens folded per second over the
timed region (a token is folded into all 112 units of its stream), queries
included.

The other workloads (7B single stream, long delay K = 1024, high resolution
32 x 8 units, K = 2048, 576 tokens per frame) run after the headline as
sub-objects with --sub-steps timed frames each and one query at the end.

Roofline.  Algorithmic bytes are the per-unit formulas of the method (the
fold: evicted keys and values, every slot's bf16 unit centre and screening
meta, and per touched slot its 3108-byte statistics row read and written
plus its bf16 centre written; append: the frame read and the ring written;
readout: K and V of every context row, the biases, queries in and outputs
out), with the touched slots per fold measured by the device counters.  The
fold's bytes are split between its kernels, each byte once: the screen is
charged with the evicted keys and values, the centres and meta and the two
PQ histograms of each touched slot (read and written); the aggregation
with the rest of each touched row and the centre rewrite.  `roofline` is the
dominant kernel of a step (most device time): its bytes per launch divided by
its average launch time, measured live inside the timed region with HIP
events recorded on the launch stream.  `traffic` is the HBM bytes per
launch from the committed FETCH_SIZE / WRITE_SIZE summary under profiles/
(null when that kernel's source has changed since the counters were taken).

CPU baseline.  The oracle (untuned) on the host cores, run before the GPU is
touched: a sample of one stream's units, the bank filled untimed, then a
fixed number of steady-state frames timed, scaled to the whole job; once on
one thread, once on a pool of worker processes (one thread each).
"""
import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TF = 2500.0   # dense bf16 TFLOP/s
D = 128
G, C = 8, 16
ROW_BYTES = 16 * D + 8 * G * C + 36      # sums, squared sums, histograms, n, n_res, mu, Sigma, tau = 3108
HIST_BYTES = 2 * G * C * 4               # the K and V histograms of one row = 1024
CENTRE_META_BYTES = 2 * D + 32           # bf16 unit centre + (mu, Sigma^-1, idle) meta = 288

FOLD_KERNELS = ("ring_insert", "seed", "screen", "aggregate", "maintain", "rope_ring", "warm_collect",
                "warm_kmeans")
QUERY_KERNELS = ("decode", "materialize", "attend", "attend_merge", "rope_q")
KERNEL_SOURCES = {k: "fold.hip" for k in FOLD_KERNELS}
KERNEL_SOURCES.update({k: "query.hip" for k in QUERY_KERNELS + ("rope_ring",)})
KERNEL_SOURCES.update({k: "warmup.hip" for k in ("warm_collect", "warm_kmeans")})
SUB_WORKLOADS = ("7b", "long", "hires")


def parse(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64, help="timed rounds of the headline workload")
    ap.add_argument("--warmup", type=int, default=8,
                    help="untimed steady-state rounds after the windows and banks are filled")
    ap.add_argument("--workload", default="multi")
    ap.add_argument("--profile-frames", type=int, default=8)
    ap.add_argument("--sub-workloads", default=",".join(SUB_WORKLOADS),
                    help="comma-separated workloads reported as sub-objects ('' = none)")
    ap.add_argument("--sub-steps", type=int, default=32)
    ap.add_argument("--query-reps", type=int, default=20)
    ap.add_argument("--pool", type=int, default=0,
                    help="distinct device frames cycled per multi-stream run (0: every frame distinct, "
                         "up to 100 GB of frames)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-units", type=int, default=16)
    ap.add_argument("--cpu-frames", type=int, default=32)
    ap.add_argument("--cpu-workers", type=int, default=16)
    ap.add_argument("--maintenance", action="store_true",
                    help="fold with prototype maintenance (aging, merging, recycling) after every frame")
    ap.add_argument("--ema", action="store_true",
                    help="fixed-rate EMA centres (alpha = beta = 0.05) instead of running means")
    ap.add_argument("--rope-theta", type=float, default=0.0,
                    help="rotary positions in the readout with this base (0 = off)")
    ap.add_argument("--warm-frames", type=int, default=0, help="PQ codebook warm-up folds (0 = given codebooks)")
    return ap.parse_args(argv)


def plan(wl, steps, warmup, profile_frames, warm_frames=0):
    """Frame counts per stream: the untimed fill (window, bank, codebook
    warm-up), the untimed steady-state warm-up, the profile pass and the timed
    steps.  Any non-negative --warmup / --steps is accepted."""
    fill = wl.window_frames + math.ceil(wl.capacity / wl.tokens_per_frame) + 1 + max(0, warm_frames)
    warmup, steps, profile_frames = max(0, warmup), max(1, steps), max(1, profile_frames)
    return {"fill": fill, "warmup": warmup, "profile": profile_frames, "steps": steps,
            "total": fill + warmup + profile_frames + steps}


def query_due(wl, r):
    """Stream that queries after round r of a multi-stream run (None if none):
    stream b queries at the rounds with (r - 2 b) mod query_every = query_every - 1."""
    if wl.streams <= 1 or wl.query_every <= 0:
        return None
    x = (r - (wl.query_every - 1)) % wl.query_every
    if x % 2 or x // 2 >= wl.streams:
        return None
    return x // 2


# ---------------------------------------------------------------------------
# algorithmic bytes
# ---------------------------------------------------------------------------


def kv_bytes(wl):
    return 4 if wl.kv_dtype == "fp32" else 2


def fold_bytes_per_unit(wl, touched):
    """Fold bytes of one unit and frame: 2 N D b + K (2D + 32) + U (2 * 3108 + 2D)."""
    N, K, b = wl.tokens_per_frame, wl.capacity, kv_bytes(wl)
    return 2 * N * D * b + K * CENTRE_META_BYTES + touched * (2 * ROW_BYTES + 2 * D)


def algorithmic_bytes(kernel, wl, units, touched_per_unit=0.0, seeded_per_unit=0.0, n_active=0,
                      ctx=0, rows=0):
    """Bytes the method must move per launch of `kernel` over `units` units
    (a fold kernel: every unit of every folded stream; a query kernel: the
    units of one stream)."""
    N, K, b = wl.tokens_per_frame, wl.capacity, kv_bytes(wl)
    if kernel in ("ring_insert", "rope_ring"):
        return units * 4 * N * D * b                      # frame read, ring written
    if kernel == "seed":
        return units * seeded_per_unit * (2 * D * b + ROW_BYTES + CENTRE_META_BYTES)
    if kernel == "screen":
        return units * (2 * N * D * b + K * CENTRE_META_BYTES + touched_per_unit * 2 * HIST_BYTES)
    if kernel == "aggregate":
        return units * touched_per_unit * (2 * (ROW_BYTES - HIST_BYTES) + 2 * D)
    if kernel in ("decode", "materialize", "attend", "attend_merge"):
        # the readout as a whole is charged to its kernels together: see readout_bytes
        return 0
    return 0


def readout_bytes(wl, units, ctx, n_active, rows):
    """Readout bytes for one query of one stream: per kv head K and V of every
    context row, the K biases, the R query rows in and outputs out."""
    b = kv_bytes(wl)
    return units * (2 * b * D * ctx + 4 * wl.capacity + 2 * b * rows * D)


def readout_flops(units, ctx, rows):
    """Q K^T and P V: 4 R L_ctx D per kv head."""
    return units * 4 * rows * ctx * D


def kernel_source_hash(kernel):
    """sha256 over the HIP source file holding `kernel` and the shared header."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2606_26762_amd", "csrc")
    hs = hashlib.sha256()
    for f in (KERNEL_SOURCES[kernel], "pkv_internal.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            hs.update(fh.read())
    return hs.hexdigest()


def recorded_traffic(kernel, wl):
    """HBM bytes per launch from a committed FETCH_SIZE/WRITE_SIZE summary under
    profiles/ (a fenced json block), or None when there is none for this kernel
    and workload or the kernel's source has changed since the counters were taken."""
    import glob
    import re
    want = kernel_source_hash(kernel)
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        text = open(path).read()
        for block in re.findall(r"```json\n(.*?)\n```", text, re.S):
            try:
                rec = json.loads(block)
            except ValueError:
                continue
            if (isinstance(rec, dict) and rec.get("kernel") == kernel and rec.get("workload") == wl.name
                    and rec.get("source_sha256") == want and "traffic_bytes_per_launch" in rec):
                rec = dict(rec)
                rec["file"] = os.path.relpath(path, ROOT)
                return rec
    return None


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on the host cores
# ---------------------------------------------------------------------------


def _oracle_units(args):
    """Worker: fill the bank of `units` untimed, then time `frames` folds and
    one unit's readout.  -> (fold seconds, readout seconds)."""
    wl_name, units, frames, readout = args
    from threadpoolctl import threadpool_limits
    from oracle import protokv_oracle as O
    from paper_2606_26762_amd import workloads as W
    wl = next(w for w in W.WORKLOADS.values() if w.name == wl_name)
    with threadpool_limits(1):
        cb = W.make_codebooks(wl, units=units, samples=512, iters=6)
        p = O.Params(head_dim=wl.head_dim, grid_h=wl.grid_h, grid_w=wl.grid_w,
                     window_frames=wl.window_frames, capacity=wl.capacity, kv_dtype=wl.kv_dtype)
        gen = W.HostStream(wl, units=units)
        st = O.OracleStream(p, units, cb)
        for _ in range(wl.window_frames + math.ceil(wl.capacity / wl.tokens_per_frame) + 1):
            st.append_frame(*gen.next_frame())
        fr = [gen.next_frame() for _ in range(frames)]
        t0 = time.perf_counter()
        for k, v in fr:
            st.append_frame(k, v)
        t_fold = time.perf_counter() - t0
        t_read = 0.0
        if readout:
            t0 = time.perf_counter()
            ps = O.synthesize(st.banks[0], st.codebooks[0], p)
            rows = wl.query_tokens * (wl.num_q_heads // wl.num_kv_heads)
            q = np.random.default_rng(0).standard_normal((rows, wl.head_dim))
            kc, vc, bias = st.context(0, ps)
            O.attend(q, kc, vc, bias)
            t_read = time.perf_counter() - t0
    return t_fold, t_read


def cpu_baseline(args, wl):
    """The untuned oracle on a bounded sample of the workload (stream 0's first
    units), scaled to the whole job's tokens/s; one thread, then a pool of
    worker processes with one thread each.  Runs before the GPU is used."""
    import multiprocessing as mp
    units = list(range(min(args.cpu_units, wl.units)))
    t_fold, t_read = _oracle_units((wl.name, units, args.cpu_frames, True))
    job_units = wl.units * wl.streams
    tok_1 = args.cpu_frames * wl.tokens_per_frame * len(units) / (t_fold * job_units)
    workers = max(1, min(args.cpu_workers, os.cpu_count() or 1))
    per = max(1, len(units) // 4)
    chunks = [(wl.name, [(w * per + i) % wl.units for i in range(per)], args.cpu_frames, False)
              for w in range(workers)]
    with mp.get_context("fork").Pool(workers) as pool:
        res = pool.map(_oracle_units, chunks)
    t_par = max(r[0] for r in res)
    tok_n = args.cpu_frames * wl.tokens_per_frame * per * workers / (t_par * job_units)
    return {
        "value": round(tok_n, 2), "unit": "tokens/s", "cores": workers, "kind": "oracle",
        "sample": (f"{workers} worker processes x {per} units of stream 0, {args.cpu_frames} steady-state "
                   f"folds each after an untimed bank fill (slowest worker {t_par:.1f} s), scaled to "
                   f"{job_units} units; the same with one thread: {len(units)} units x {args.cpu_frames} "
                   f"folds in {t_fold:.1f} s"),
        "value_1_thread": round(tok_1, 2),
        "readout_us_per_query_1_thread": round(t_read * wl.units * 1e6, 1),
        "readout_sample": "synthesis + attention of 1 unit, scaled to the stream's units",
        "cpu": _cpu_model(), "nproc": os.cpu_count(),
    }


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---------------------------------------------------------------------------
# GPU run of one workload
# ---------------------------------------------------------------------------


def run_workload(wl, args, steps, warmup, profile_frames, query_reps, headline):
    import torch
    from paper_2606_26762_amd import protokv as pk
    from paper_2606_26762_amd import workloads as W

    lib = pk.lib()
    NS = wl.streams
    pl = plan(wl, steps, warmup, profile_frames, args.warm_frames)
    cfg = pk.default_config(num_streams=NS, num_layers=wl.num_layers, num_kv_heads=wl.num_kv_heads,
                            num_q_heads=wl.num_q_heads, grid_h=wl.grid_h, grid_w=wl.grid_w,
                            window_frames=wl.window_frames, capacity=wl.capacity,
                            max_query_tokens=wl.query_tokens,
                            kv_dtype=pk.KV_FP32 if wl.kv_dtype == "fp32" else pk.KV_BF16)
    if args.maintenance:
        cfg.flags |= pk.FLAG_MAINTENANCE
    if args.ema:
        cfg.flags |= pk.FLAG_EMA_CENTRES
    cfg.rope_theta = args.rope_theta
    cfg.warm_frames = args.warm_frames
    print(f"bench: {wl.name}: {NS} stream(s) x {wl.units} units, frames per stream {pl}", file=sys.stderr,
          flush=True)
    cb = W.make_codebooks_device(wl, n_streams=NS, samples=1024 if NS > 1 else 2048)
    eng = pk.ProtoKV(cfg, cb.reshape(-1, *cb.shape[2:]))
    del cb
    gen = W.DeviceStream(wl, n_streams=NS)
    # every frame drawn ahead (each [streams][L][Hkv][T][D]), up to 100 GB of
    # them; beyond that (or --pool) a pool of distinct frames taken in turn
    frame_bytes = 2 * NS * wl.units * wl.tokens_per_frame * D * kv_bytes(wl)
    nframes = min(pl["total"], args.pool or pl["total"], max(1, int(100e9 // frame_bytes)))
    ks, vs = [], []
    for _ in range(nframes):
        k, v = gen.next_frame()
        ks.append(k)
        vs.append(v)
    q = gen.query()
    o = torch.empty_like(q)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    h = eng.h
    ids = (ctypes.c_int32 * NS)(*range(NS))
    kp = [ctypes.c_void_p(t.data_ptr()) for t in ks]
    vp = [ctypes.c_void_p(t.data_ptr()) for t in vs]
    qp, op, lp = ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(o.data_ptr()), ctypes.c_void_p(lse.data_ptr())
    tq = q.shape[1]
    T = wl.tokens_per_frame
    append, fold = lib.protokv_append_frame, lib.protokv_fold
    synth, attend = lib.protokv_synthesize, lib.protokv_attend
    nq = [0]

    def run_query(sid=0):
        if synth(h, sid, sp) or attend(h, sid, qp, tq, op, lp, sp):
            raise RuntimeError(lib.protokv_last_error(h))
        nq[0] += 1

    def run_rounds(lo, hi, queries):
        for r in range(lo, hi):
            j = r % len(kp)
            if append(h, ids, NS, kp[j], vp[j], sp) or fold(h, sp):
                raise RuntimeError(lib.protokv_last_error(h))
            if queries:
                b = query_due(wl, r)
                if b is not None:
                    run_query(b)

    multi = NS > 1
    r = 0
    run_rounds(r, r + pl["fill"] + pl["warmup"], multi)
    r += pl["fill"] + pl["warmup"]
    run_query()
    torch.cuda.synchronize()

    # profile pass: library HIP events around every launch
    c0 = eng.counters()
    eng.profile(True)
    nq0 = nq[0]
    run_rounds(r, r + pl["profile"], multi)
    r += pl["profile"]
    if not multi:
        for _ in range(3):
            run_query()
    kt = eng.profile_read()
    eng.profile(False)
    c1 = eng.counters()
    info = eng.stream_info(0)
    n_active = info.active_slots
    folds = max(1, kt.get("aggregate", {}).get("launches", 1))
    fold_units = NS * wl.units
    touched = (c1.touched - c0.touched) / folds / fold_units
    rows = tq * (wl.num_q_heads // wl.num_kv_heads)
    ctx = min(info.frames, wl.window_frames) * T + n_active * cfg.pseudo_per_proto
    per_step = {}
    kernels = {}
    for name, d in kt.items():
        units = fold_units if name in FOLD_KERNELS else wl.units
        nbytes = algorithmic_bytes(name, wl, units, touched_per_unit=touched)
        kernels[name] = {"avg_us": round(d["avg_us"], 3), "launches": d["launches"],
                         "alg_bytes_per_launch": int(nbytes),
                         "gbs": round(nbytes / (d["avg_us"] * 1e-6) / 1e9, 1) if nbytes else None}
        # device time per round of the kernels a round runs (a single stream's
        # queries come after the rounds, not in them)
        if multi or name in FOLD_KERNELS:
            per_step[name] = d["ms"] * 1e3 / pl["profile"]
    dom = max(per_step, key=per_step.get)

    # timed region: only the dominant kernel's launches are bracketed by the
    # library's events (on the launch stream)
    c2 = eng.counters()
    eng.profile(True, [dom])
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    nq0 = nq[0]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    e0.record(stream)
    run_rounds(r, r + pl["steps"], multi)
    e1.record(stream)
    if not multi:
        run_query()
    e2.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    r += pl["steps"]
    live = eng.profile_read()[dom]
    eng.profile(False)
    c3 = eng.counters()
    queries_timed = nq[0] - nq0
    ms_total = e0.elapsed_time(e2)
    ms_rounds = e0.elapsed_time(e1)
    value = pl["steps"] * T * NS / (ms_total / 1e3)
    touched_live = (c3.touched - c2.touched) / pl["steps"] / fold_units

    # readout latency: median over repeats, synthesize + attend and attend only,
    # and the per-kernel times of one query
    def median_ms(fn, reps):
        out = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            torch.cuda.synchronize()
            out.append(a.elapsed_time(b))
        return float(np.median(out))
    readout_ms = median_ms(run_query, query_reps)
    attend_ms = median_ms(lambda: attend(h, 0, qp, tq, op, lp, sp), query_reps)
    eng.profile(True, [k for k in ("decode", "materialize", "attend", "attend_merge", "rope_q")])
    for _ in range(query_reps):
        run_query()
    qkt = eng.profile_read()
    eng.profile(False)
    torch.cuda.synchronize()
    query_kernels = {k: round(v["avg_us"], 3) for k, v in qkt.items()}
    query_dev_us = sum(query_kernels.values())

    dom_units = fold_units if dom in FOLD_KERNELS else wl.units
    dom_bytes = algorithmic_bytes(dom, wl, dom_units, touched_per_unit=touched_live)
    if dom_bytes == 0:   # a query kernel dominates: charge it the readout's bytes
        dom_bytes = readout_bytes(wl, wl.units, ctx, n_active, rows) * live["avg_us"] / max(query_dev_us, 1e-9)
    achieved = dom_bytes / (live["avg_us"] * 1e-6) / 1e9
    traffic = recorded_traffic(dom, wl)
    # a plain copy of known size measured in the same run (the ring insert:
    # the frame read once and written once) as the practical bandwidth
    copy_gbs = kernels.get("ring_insert", {}).get("gbs")
    roofline = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "copy_gbs": copy_gbs, "frac_of_copy": round(achieved / copy_gbs, 4) if copy_gbs else None,
                "traffic": traffic["traffic_bytes_per_launch"] if traffic else None,
                "alg_bytes_per_launch": int(dom_bytes), "avg_us": round(live["avg_us"], 3),
                "launches_timed": live["launches"],
                "traffic_source": traffic["file"] if traffic else None}
    # the fold pass as a whole (all its kernels, device time per frame)
    fold_names = [n for n in ("seed", "screen", "aggregate") if n in kt]
    fold_us = sum(kt[n]["ms"] * 1e3 for n in fold_names) / pl["profile"]
    fold_b = fold_units * fold_bytes_per_unit(wl, touched)
    roof_fold = {"kernels": fold_names, "alg_bytes_per_frame": int(fold_b), "device_us_per_frame": round(fold_us, 2),
                 "achieved": round(fold_b / (fold_us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": round(fold_b / (fold_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                 "frac_of_copy": round(fold_b / (fold_us * 1e-6) / 1e9 / copy_gbs, 4) if copy_gbs else None,
                 "touched_per_unit": round(touched, 2)}
    rb = readout_bytes(wl, wl.units, ctx, n_active, rows)
    rf = readout_flops(wl.units, ctx, rows)
    roof_read = {"kernels": sorted(query_kernels), "device_us_per_query": round(query_dev_us, 2),
                 "alg_bytes_per_query": int(rb), "flops_per_query": int(rf),
                 "hbm_achieved": round(rb / (query_dev_us * 1e-6) / 1e9, 1), "hbm_peak": HBM_PEAK_GBS,
                 "hbm_frac": round(rb / (query_dev_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                 "hbm_frac_of_copy": round(rb / (query_dev_us * 1e-6) / 1e9 / copy_gbs, 4) if copy_gbs else None,
                 "mfma_tflops": round(rf / (query_dev_us * 1e-6) / 1e12, 2), "mfma_peak": MFMA_BF16_PEAK_TF,
                 "mfma_frac": round(rf / (query_dev_us * 1e-6) / 1e12 / MFMA_BF16_PEAK_TF, 4),
                 "roof_us": round(1e6 * max(rb / (HBM_PEAK_GBS * 1e9), rf / (MFMA_BF16_PEAK_TF * 1e12)), 2),
                 "bound": "mfma" if rf / (MFMA_BF16_PEAK_TF * 1e12) > rb / (HBM_PEAK_GBS * 1e9) else "hbm"}
    # the screen's similarity contraction 2 N K D per unit against the bf16 peak
    if "screen" in kernels:
        sim = fold_units * 2 * T * wl.capacity * D
        kernels["screen"]["similarity_tflops"] = round(sim / (kernels["screen"]["avg_us"] * 1e-6) / 1e12, 2)
        kernels["screen"]["similarity_mfma_frac"] = round(
            sim / (kernels["screen"]["avg_us"] * 1e-6) / 1e12 / MFMA_BF16_PEAK_TF, 4)

    out = {
        "workload": wl.name, "streams": NS, "units_per_stream": wl.units, "tokens_per_frame": T,
        "window_frames": wl.window_frames, "capacity": wl.capacity, "query_tokens": tq,
        "value": round(value, 1), "unit": "tokens/s", "steps": pl["steps"],
        "ms_per_step": round(ms_total / pl["steps"], 5),
        "queries_in_timed_region": queries_timed + (0 if multi else 1),
        "fold_tokens_per_s": round(pl["steps"] * T * NS / (ms_rounds / 1e3), 1),
        "fold_us_per_frame": round(1e3 * ms_rounds / pl["steps"], 2),
        "readout_us_per_query": round(1e3 * readout_ms, 2),
        "attend_us_per_query": round(1e3 * attend_ms, 2),
        "wall_s_timed_region": round(t_wall, 4),
        "touched_per_unit_fold": round(touched_live, 2), "active_slots": n_active, "context_tokens": ctx,
        "distinct_frames": nframes,
        "refined_fraction": round((c3.refined + c3.refined_full) / max(1, c3.tokens_assigned), 5),
        "near_ties": c3.near_ties, "frames_per_stream": r,
        "kernels": kernels, "query_kernels_us": query_kernels,
        "roofline": roofline, "roofline_fold": roof_fold, "roofline_readout": roof_read,
    }
    del eng, ks, vs, kp, vp, q, o, lse, gen
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def main(argv=None):
    args = parse(argv)
    if args.gpus != 1:
        print(f"bench.py: measures one GPU; --gpus {args.gpus} is not supported "
              f"(units are independent and would shard by stream or kv head)",
              file=sys.stderr)
        sys.exit(2)
    from paper_2606_26762_amd import workloads as W
    wl = W.WORKLOADS[args.workload]
    cpu = None
    if not args.no_cpu_baseline:
        # before the GPU is touched (the worker pool forks this process)
        cpu = cpu_baseline(args, wl)
        print(f"bench: cpu baseline {cpu['value']} tokens/s on {cpu['cores']} workers", file=sys.stderr,
              flush=True)
    import torch
    torch.cuda.set_device(0)
    head = run_workload(wl, args, args.steps, args.warmup, args.profile_frames, args.query_reps, True)
    subs = {}
    for name in [s for s in args.sub_workloads.split(",") if s and s != args.workload]:
        subs[name] = run_workload(W.WORKLOADS[name], args, args.sub_steps, 4, 4, args.query_reps, False)
    result = {
        "metric": "evicted tokens folded/sec/GPU + readout µs/query; % HBM/MFMA roofline",
        "value": head["value"], "unit": "tokens/s", "n_gpus": 1, "steps": head["steps"],
        "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": f"synthetic (seeded on-device Gaussian-mixture streams, {wl.name})",
        "config": {"workload": wl.name, "streams": wl.streams, "layers": wl.num_layers,
                   "kv_heads": wl.num_kv_heads, "q_heads": wl.num_q_heads, "head_dim": wl.head_dim,
                   "tokens_per_frame": wl.tokens_per_frame, "window_frames": wl.window_frames,
                   "capacity": wl.capacity, "pseudo_per_proto": 8, "query_tokens": wl.query_tokens,
                   "query_every_frames": wl.query_every, "maintenance": bool(args.maintenance),
                   "centres": "ema" if args.ema else "mean", "rope_theta": args.rope_theta,
                   "warm_frames": args.warm_frames},
        "readout_us_per_query": head["readout_us_per_query"],
        "roofline": head["roofline"],
        "roofline_fold": head["roofline_fold"],
        "roofline_readout": head["roofline_readout"],
        "detail": head,
        "workloads": subs,
    }
    if cpu is not None:
        result["cpu_baseline"] = cpu
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
