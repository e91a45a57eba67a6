#!/usr/bin/env python3
"""Benchmark of the ProtoKV far-memory hot path on one MI355X.

Workload: one stream of a 7B-class video LLM (28 layers x 4 KV heads, 28
query heads, head_dim 128, bf16 KV, 196 visual tokens per frame on a 14x14
grid, near window 8 frames, K = 256 prototypes per (layer, kv head)), seeded
synthetic frames drawn on the GPU (the paper's video datasets stand in).

A step = one frame through the whole hot path's streaming side: append the
frame to the near window of all 112 (layer, kv head) units and fold the
evicted frame (seed / screen + assign / aggregate).  The timed region is
`--steps` such frames followed by one 32-token query (synthesize + attend),
so every hot-path step runs inside it.  `value` = evicted model tokens
folded per second over the timed region (each token folded into all 112
units).  Readout latency per query is timed separately (median of repeats).

Per-kernel device times come from HIP events the library records around
each launch on the launch stream: first around every launch over
--profile-frames frames (to find the fold's dominant kernel), then, inside
the timed region, around that kernel's launches only.  The roofline object
divides that kernel's algorithmic bytes per launch by its live average
duration; `traffic` is the HBM bytes per launch from the committed
FETCH_SIZE/WRITE_SIZE summary under profiles/, null when the kernel's source
has changed since.
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

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, GB/s
MFMA_BF16_PEAK = 2500.0     # dense bf16 TFLOP/s
ROW_STATS_BYTES = 4 * 128 * 4 + 32   # a bank row's four sums and its meta
HIST_BYTES = 2 * 8 * 16 * 4          # a bank row's K and V histograms
CACHE_BYTES = 2 * 128 * 2 + 32       # hi + lo bf16 unit centre + screening meta
CODEBOOK_BYTES = 2 * 8 * 16 * 16 * 4  # a unit's K and V codebooks


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=192)
    ap.add_argument("--warmup", type=int, default=64)
    ap.add_argument("--workload", default="7b")
    ap.add_argument("--profile-frames", type=int, default=32)
    ap.add_argument("--maintenance", action="store_true",
                    help="fold with prototype maintenance (aging, merging, recycling) after every frame")
    ap.add_argument("--ema", action="store_true",
                    help="fixed-rate EMA centres (alpha = beta = 0.05) instead of running means")
    ap.add_argument("--rope-theta", type=float, default=0.0,
                    help="rotary positions in the readout with this base (0 = off)")
    ap.add_argument("--warm-frames", type=int, default=0,
                    help="PQ codebook warm-up folds (0 = given codebooks); 57..88 puts its end inside "
                         "the profile pass with the default warm-up and profile frames")
    ap.add_argument("--query-reps", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-units", type=int, default=32)
    ap.add_argument("--cpu-frames", type=int, default=64)
    return ap.parse_args()


def algorithmic_bytes(kernel, wl, cfg, touched_per_launch=0.0, n_active=0, ctx=0, rows=0, formed=False,
                      maint=None, ema=False):
    """Bytes the method must move per launch of `kernel` (all units of one stream).

    `formed`: the readout forms the pseudo-token rows from the centres, code
    tuples and codebooks as it loads them (no rows in memory).  `maint`: aged,
    merged and recycled slots per maintenance launch.  `ema`: EMA centres, whose
    residual codes the aggregation computes (the screen only assigns)."""
    U, T, D, K, S = wl.units, wl.tokens_per_frame, wl.head_dim, wl.capacity, cfg.pseudo_per_proto
    if kernel in FOLD_KERNELS:  # one launch folds every stream's units
        U *= cfg.num_streams
    b = 4 if wl.kv_dtype == "fp32" else 2
    if kernel == "ring_insert":
        return U * T * D * b * 2 * 2                       # read frame K,V + write ring K,V
    if kernel == "screen":
        # assignment: evicted keys, the unit's centre cache, assignments
        # written; PQ encoding: evicted values, codebooks, per touched slot
        # its K and V sums (centres) and its two histograms read and written
        if ema:
            return U * (T * D * b + K * CACHE_BYTES + T * 4)
        return (U * (2 * T * D * b + K * CACHE_BYTES + T * 4 + CODEBOOK_BYTES)
                + touched_per_launch * (2 * D * 4 + 2 * HIST_BYTES))
    if kernel == "aggregate":
        # evicted K and V, assignments; per touched slot its sums, sums of
        # squares and meta read and written and its screening copy rewritten
        # (EMA centres: also the unit's codebooks and the slot's histograms)
        return (U * (2 * T * D * b + T * 4 + (CODEBOOK_BYTES if ema else 0))
                + touched_per_launch * (2 * ROW_STATS_BYTES + CACHE_BYTES + (2 * HIST_BYTES if ema else 0)))
    if kernel == "maintain":
        # every slot's mass, tau and leading fd key and value dims (the LDS
        # filter: 16, 8 or 4 dims as K grows); an aged slot's sums and squares
        # read and written; a merge reads two rows and writes one; a recycled
        # slot reads its token and writes its row; rewritten screening copies
        m = maint or {}
        fd = 16 if K <= 512 else (8 if K <= 1024 else 4)
        row = 4 * D * 4 + 2 * 8 * 16 * 4 + 32
        return (U * n_active * (8 + 2 * fd * 4) + m.get("aged", 0) * (2 * 4 * D * 4 + CACHE_BYTES)
                + m.get("merged", 0) * (3 * row + CACHE_BYTES)
                + m.get("recycled", 0) * (2 * D * b + row + CACHE_BYTES))
    if kernel == "rope_ring":
        # ring insert with the rotated key copy: K, V read; K, V and rotated K written
        return U * T * D * b * 5
    if kernel == "warm_collect":
        # per non-seed token: its K and V, its slot's two sums, the two
        # residual rows written
        return U * T * (2 * D * b + 2 * D * 4 + 2 * D * 4)
    if kernel == "warm_kmeans":
        # every reservoir row read once per epoch, the codebooks written
        return U * (cfg.kmeans_epochs * 2 * cfg.warm_tokens * D * 4 + CODEBOOK_BYTES)
    if kernel == "rope_q":
        # the query read and written rotated
        return wl.num_layers * wl.query_tokens * wl.num_q_heads * D * b * 2
    if kernel == "decode":
        # histograms, meta, codes out; with formed rows also the sums in and
        # the float32 centres and bias out
        extra = (2 * D * 4 + 2 * D * 4 + 4) if formed else 0
        return U * n_active * (2 * 8 * 16 * 4 + 32 + 2 * (S + 1) * 4 + extra)
    if kernel == "materialize":
        # sums, meta, codes, codebooks per unit, pseudo-token rows out, bias out
        return (U * n_active * (2 * 4 * D + 32 + 2 * (S + 1) * 4 + S * D * b * 2 + 4)
                + U * 2 * 8 * 16 * 16 * 4)
    if kernel == "attend":
        if formed:
            # near-window K, V; per active slot its centres, code tuples and
            # bias; the unit's codebooks; queries in, outputs out
            n_near = ctx - n_active * S
            return U * (2 * n_near * D * b + n_active * (2 * D * 4 + 2 * (S + 1) * 4 + 4)
                        + CODEBOOK_BYTES + 2 * rows * D * b)
        return U * (2 * ctx * D * b + (ctx // max(S, 1)) * 4 + 2 * rows * D * b)
    return 0


FOLD_KERNELS = ("ring_insert", "seed", "screen", "aggregate", "maintain", "rope_ring", "warm_collect",
                "warm_kmeans")
KERNEL_SOURCES = {k: "fold.hip" for k in FOLD_KERNELS}  # maintain too
KERNEL_SOURCES.update({k: "query.hip" for k in ("decode", "materialize", "attend", "attend_merge", "rope_ring",
                                                 "rope_q")})
KERNEL_SOURCES.update({k: "warmup.hip" for k in ("warm_collect", "warm_kmeans")})


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


def cpu_baseline(args, wl):
    """The oracle, untuned, on a bounded sample: --cpu-units units of the same
    workload, bank filled untimed, then --cpu-frames timed steady-state folds;
    scaled to model tokens/s for all units.  Readout: one unit's synthesis +
    attention, scaled to all units."""
    from threadpoolctl import threadpool_limits
    from oracle import protokv_oracle as O
    from paper_2606_26762_amd import workloads as W
    units = list(range(args.cpu_units))
    cb = W.make_codebooks(wl, units=units, samples=1024, iters=8)
    p = O.Params(head_dim=wl.head_dim, grid_h=wl.grid_h, grid_w=wl.grid_w,
                 window_frames=wl.window_frames, capacity=wl.capacity, kv_dtype=wl.kv_dtype)
    gen = W.HostStream(wl, units=units)
    st = O.OracleStream(p, units, cb)
    warm = wl.window_frames + math.ceil(wl.capacity / wl.tokens_per_frame) + 1
    with threadpool_limits(1):
        for _ in range(warm):
            st.append_frame(*gen.next_frame())
        frames = [gen.next_frame() for _ in range(args.cpu_frames)]
        t0 = time.perf_counter()
        for k, v in frames:
            st.append_frame(k, v)
        t_fold = time.perf_counter() - t0
        t0 = time.perf_counter()
        ps = [O.synthesize(st.banks[0], cb[0], p)]
        q = np.random.default_rng(0).standard_normal(
            (1, wl.query_tokens, wl.num_q_heads // wl.num_kv_heads, wl.head_dim))
        kc, vc, bias = st.context(0, ps[0])
        O.attend(q.reshape(-1, wl.head_dim), kc, vc, bias)
        t_read = time.perf_counter() - t0
    scale = wl.units / len(units)
    tok_s = args.cpu_frames * wl.tokens_per_frame / (t_fold * scale)
    return {"value": tok_s, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": (f"{len(units)} of {wl.units} units x {args.cpu_frames} steady-state frames "
                       f"(fold {t_fold:.1f} s), readout of 1 unit ({t_read:.1f} s); scaled to all units"),
            "readout_us_per_query": t_read * wl.units * 1e6,
            "cpu": _cpu_model(), "nproc": os.cpu_count()}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU; --gpus {args.gpus} is not supported "
              f"(units are independent and would shard by stream or kv head)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_26762_amd import protokv as pk
    from paper_2606_26762_amd import workloads as W

    wl = W.WORKLOADS[args.workload]
    frames_needed = args.warmup + args.profile_frames + args.steps
    assert args.warmup >= wl.window_frames + math.ceil(wl.capacity / wl.tokens_per_frame), \
        "warmup must fill the bank"
    lib = pk.lib()
    NS = wl.streams
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
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cb = W.make_codebooks_device(wl, n_streams=NS)
    eng = pk.ProtoKV(cfg, cb.reshape(-1, *cb.shape[2:]))
    gen = W.DeviceStream(wl, n_streams=NS)
    # one stream: every frame drawn ahead; several: a pool of POOL frames
    # (each [streams][L][Hkv][T][D]) taken in turn
    POOL = 8
    ks, vs = [], []
    for _ in range(frames_needed if NS == 1 else POOL):
        k, v = gen.next_frame()
        ks.append(k)
        vs.append(v)
    q = gen.query()
    o = torch.empty_like(q)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=dev)
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

    def run_frames(lo, hi, queries=False):
        for i in range(lo, hi):
            j = i % len(kp)
            if append(h, ids, NS, kp[j], vp[j], sp) or fold(h, sp):
                raise RuntimeError(lib.protokv_last_error(h))
            if queries and i % QEVERY == 0:
                run_query((i // QEVERY) % NS)

    def run_query(sid=0):
        if synth(h, sid, sp) or attend(h, sid, qp, tq, op, lp, sp):
            raise RuntimeError(lib.protokv_last_error(h))

    # several streams: each queries once every query_every frames, so a step
    # (one frame of every stream) carries NS / query_every queries
    QEVERY = max(1, wl.query_every // NS) if NS > 1 else 0

    # warm-up: fill the window and the bank, compile paths, one query
    run_frames(0, args.warmup)
    run_query()
    torch.cuda.synchronize()

    # per-kernel device times: library-recorded HIP events around every launch,
    # over --profile-frames frames and 5 queries, to find the dominant kernel
    lo = args.warmup
    c0 = eng.counters()
    eng.profile(True)
    run_frames(lo, lo + args.profile_frames)
    for _ in range(5):
        run_query()
    kt = eng.profile_read()
    eng.profile(False)
    c1 = eng.counters()
    info = eng.stream_info(0)
    n_active = info.active_slots
    touched = (c1.touched - c0.touched) / max(1, kt.get("aggregate", {}).get("launches", 1))
    rows = tq * (wl.num_q_heads // wl.num_kv_heads)
    ctx = min(info.frames, wl.window_frames) * T + n_active * cfg.pseudo_per_proto
    formed = "materialize" not in kt  # bf16 readout forms the pseudo-token rows itself
    nm = max(1, kt.get("maintain", {}).get("launches", 1))
    maint = {k: (getattr(c1, k) - getattr(c0, k)) / nm for k in ("aged", "merged", "recycled")}
    kernels = {}
    for name, d in kt.items():
        nbytes = algorithmic_bytes(name, wl, cfg, touched_per_launch=touched, n_active=n_active,
                                   ctx=ctx, rows=rows, formed=formed, maint=maint, ema=args.ema)
        kernels[name] = {"avg_us": round(d["avg_us"], 3), "launches": d["launches"],
                         "alg_bytes": int(nbytes),
                         "gbs": round(nbytes / (d["avg_us"] * 1e-6) / 1e9, 1) if nbytes else None}
    # dominant kernel of the streaming step (device time per frame)
    per_frame = {n: kernels[n]["avg_us"] * kernels[n]["launches"] / args.profile_frames
                 for n in FOLD_KERNELS if n in kernels}
    dom = max(per_frame, key=per_frame.get)

    # timed region: --steps frames + one query; only the dominant kernel's
    # launches are bracketed by the library's events (on the launch stream)
    lo += args.profile_frames
    c2 = eng.counters()
    eng.profile(True, [dom])
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    e0.record(stream)
    run_frames(lo, lo + args.steps, queries=NS > 1)
    e1.record(stream)
    run_query()
    e2.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    live = eng.profile_read()[dom]
    eng.profile(False)
    c3 = eng.counters()
    ms_total = e0.elapsed_time(e2)
    ms_fold = e0.elapsed_time(e1)
    ms_query_in_region = e1.elapsed_time(e2)
    value = args.steps * T * NS / (ms_total / 1e3)
    touched_live = (c3.touched - c2.touched) / args.steps

    # readout latency: median over repeats, synthesize+attend and attend only
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
    readout_ms = median_ms(run_query, args.query_reps)
    attend_ms = median_ms(lambda: attend(h, 0, qp, tq, op, lp, sp), args.query_reps)

    dom_bytes = algorithmic_bytes(dom, wl, cfg, touched_per_launch=touched_live, n_active=n_active,
                                  ctx=ctx, rows=rows, formed=formed, maint=maint, ema=args.ema)
    achieved = dom_bytes / (live["avg_us"] * 1e-6) / 1e9
    traffic = recorded_traffic(dom, wl)
    roofline = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic["traffic_bytes_per_launch"] if traffic else None,
                "alg_bytes_per_launch": int(dom_bytes), "avg_us": round(live["avg_us"], 3),
                "launches_timed": live["launches"],
                "traffic_source": traffic["file"] if traffic else None}
    # screen MFMA work, for reference: 2 (hi, lo) x 2 N K D flops per unit
    scr_flops = NS * wl.units * 2 * 2 * T * wl.capacity * wl.head_dim
    if "screen" in kernels:
        kernels["screen"]["mfma_tflops"] = round(scr_flops / (kernels["screen"]["avg_us"] * 1e-6) / 1e12, 2)
    att_flops = wl.units * 4 * rows * ctx * wl.head_dim
    if "attend" in kernels:
        kernels["attend"]["mfma_tflops"] = round(att_flops / (kernels["attend"]["avg_us"] * 1e-6) / 1e12, 2)

    result = {
        "metric": "evicted tokens folded/sec/GPU + readout µs/query; % HBM/MFMA roofline",
        "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_total / args.steps, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": f"synthetic (seeded on-device Gaussian-mixture stream{'s' if NS > 1 else ''}, {wl.name})",
        "config": {"workload": wl.name, "layers": wl.num_layers, "kv_heads": wl.num_kv_heads,
                   "q_heads": wl.num_q_heads, "head_dim": wl.head_dim, "tokens_per_frame": T,
                   "window_frames": wl.window_frames, "capacity": wl.capacity,
                   "pseudo_per_proto": cfg.pseudo_per_proto, "query_tokens": tq,
                   "frames_streamed": lo + args.steps, "maintenance": bool(args.maintenance),
                   "centres": "ema" if args.ema else "mean", "rope_theta": args.rope_theta,
                   "warm_frames": args.warm_frames, "streams": NS},
        # with several streams a step is one frame of every stream, and the
        # fold figures include the queries issued during the steps
        "fold_tokens_per_s": round(args.steps * T * NS / (ms_fold / 1e3), 1),
        "fold_us_per_frame": round(1e3 * ms_fold / args.steps, 2),
        "query_us_in_region": round(1e3 * ms_query_in_region, 2),
        "readout_us_per_query": round(1e3 * readout_ms, 2),
        "attend_us_per_query": round(1e3 * attend_ms, 2),
        "wall_s_timed_region": round(t_wall, 4),
        "touched_per_fold": round(touched_live, 1), "active_slots": n_active,
        "context_tokens": ctx,
        "refined_fraction": round((c3.refined + c3.refined_full) / max(1, c3.tokens_assigned), 5),
        "refined_full": c3.refined_full, "near_ties": c3.near_ties,
        "maintenance_per_fold": ({k: round(v, 1) for k, v in maint.items()} if args.maintenance else None),
        "kernels": kernels,
        "roofline": roofline,
    }
    if not args.no_cpu_baseline and NS == 1:
        result["cpu_baseline"] = cpu_baseline(args, wl)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
