"""Host-side logic of bench.py, no GPU: the one-GPU refusal, the driver's
arguments, the multi-stream query schedule, the algorithmic byte counts
against their closed forms, and the lookup of the recorded HBM traffic
(found for the recorded source hash, refused for any other)."""
import glob
import json
import math
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_26762_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_driver_arguments_fill_the_bank_untimed():
    """The driver runs `bench.py --gpus 1 --steps 20 --warmup 5`: accepted, and
    the window and bank are filled before the timed region whatever --warmup is."""
    for argv in (["--gpus", "1", "--steps", "20", "--warmup", "5"], ["--warmup", "0"], []):
        a = bench.parse(argv)
        assert a.gpus == 1 and a.workload == "multi"
        for name in ("multi", "7b", "long", "hires", "tiny"):
            wl = W.WORKLOADS[name]
            pl = bench.plan(wl, a.steps, a.warmup, a.profile_frames)
            # frames appended before the profile pass and the timed region
            before = pl["fill"] + pl["warmup"]
            evicted = (before - wl.window_frames) * wl.tokens_per_frame
            assert evicted >= wl.capacity, (name, pl)
            assert pl["steps"] == max(1, a.steps) and pl["warmup"] == max(0, a.warmup)
            assert pl["total"] == before + pl["profile"] + pl["steps"]
    a = bench.parse(["--gpus", "1", "--steps", "20", "--warmup", "5"])
    pl = bench.plan(W.WORKLOADS["multi"], a.steps, a.warmup, a.profile_frames)
    assert pl["fill"] == 8 + math.ceil(512 / 196) + 1 and pl["steps"] == 20


def test_query_schedule_of_the_multi_stream_workload():
    """Stream b queries at rounds r with (r - 2b) mod 128 = 127: every stream
    once per 128 rounds, one query every other round."""
    wl = W.WORKLOADS["multi"]
    for start in (0, 5, 128, 1000):
        got = [bench.query_due(wl, r) for r in range(start, start + 128)]
        qs = [b for b in got if b is not None]
        assert sorted(qs) == list(range(64))
        assert all((got[i] is None) != (got[i + 1] is None) for i in range(127))
        for i, b in enumerate(got):
            if b is not None:
                assert (start + i - 2 * b) % 128 == 127
    assert bench.query_due(W.WORKLOADS["7b"], 127) is None


def test_fold_bytes_split_between_kernels_sums_to_the_formula():
    """screen + aggregate = 2 N D b + K (2D + 32) + U (2 * 3108 + 2D) per unit."""
    for name, touched in (("7b", 108.9), ("multi", 130.0), ("hires", 400.0), ("tiny", 20.0)):
        wl = W.WORKLOADS[name]
        b = 4 if wl.kv_dtype == "fp32" else 2
        N, K = wl.tokens_per_frame, wl.capacity
        want = 2 * N * 128 * b + K * (2 * 128 + 32) + touched * (2 * 3108 + 2 * 128)
        assert math.isclose(bench.fold_bytes_per_unit(wl, touched), want)
        s = bench.algorithmic_bytes("screen", wl, 7, touched_per_unit=touched)
        a = bench.algorithmic_bytes("aggregate", wl, 7, touched_per_unit=touched)
        assert math.isclose(s + a, 7 * want)
    assert bench.ROW_BYTES == 3108 and bench.CENTRE_META_BYTES == 288


def test_ring_insert_and_readout_bytes():
    wl = W.WORKLOADS["7b"]
    # read K and V of the frame, write them into the ring: 4 U T D b
    assert bench.algorithmic_bytes("ring_insert", wl, 112) == 4 * 112 * 196 * 128 * 2 == 22478848
    # readout of the 7B stream: 112 kv heads x (4 D L_ctx + 4 K + 4 R D), L_ctx = 1568 + 2048
    rb = bench.readout_bytes(wl, 112, 1568 + 256 * 8, 256, 224)
    assert rb == 112 * (4 * 128 * 3616 + 4 * 256 + 4 * 224 * 128)
    assert abs(rb / 1e6 - 220.3) < 0.5
    # long delay: 291 GFLOP per query (448 rows x 11 328 context rows)
    assert abs(bench.readout_flops(112, 3136 + 8192, 448) / 1e9 - 291) < 1


def _records():
    out = []
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for blk in re.findall(r"```json\n(.*?)\n```", open(path).read(), re.S):
            try:
                rec = json.loads(blk)
            except ValueError:
                continue
            if isinstance(rec, dict) and "traffic_bytes_per_launch" in rec:
                out.append(rec)
    return out


def test_recorded_traffic_needs_the_recorded_source(monkeypatch):
    recs = _records()
    if not recs:
        return
    for rec in recs:
        wl = next(w for w in W.WORKLOADS.values() if w.name == rec["workload"])
        monkeypatch.setattr(bench, "kernel_source_hash", lambda k, h=rec["source_sha256"]: h)
        got = bench.recorded_traffic(rec["kernel"], wl)
        assert got is not None and got["traffic_bytes_per_launch"] == rec["traffic_bytes_per_launch"]
        monkeypatch.setattr(bench, "kernel_source_hash", lambda k: "0" * 64)
        assert bench.recorded_traffic(rec["kernel"], wl) is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda k, h=recs[0]["source_sha256"]: h)
    assert bench.recorded_traffic(recs[0]["kernel"], W.WORKLOADS["tiny"]) is None
