"""Host-side logic of bench.py, no GPU: the one-GPU refusal, the algorithmic
byte counts against their closed forms, and the lookup of the recorded HBM
traffic (found for the recorded source hash, refused for any other)."""
import json
import os
import re
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_26762_amd import workloads as W  # noqa: E402


def _cfg(streams=1, S=8):
    return types.SimpleNamespace(num_streams=streams, pseudo_per_proto=S)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_ring_insert_bytes_are_the_frame_copy():
    """Read K and V of the frame, write them into the ring: 4 U T D b."""
    wl = W.WORKLOADS["7b"]
    assert bench.algorithmic_bytes("ring_insert", wl, _cfg()) == 4 * 112 * 196 * 128 * 2 == 22478848
    # one launch folds every stream's units
    assert bench.algorithmic_bytes("ring_insert", wl, _cfg(streams=3)) == 3 * 22478848


def test_screen_bytes_per_touched_slot():
    """Each touched slot adds its K and V sums (2 D float32) and its two
    histograms read and written (2 x 1 KiB)."""
    wl = W.WORKLOADS["7b"]
    b0 = bench.algorithmic_bytes("screen", wl, _cfg(), touched_per_launch=0.0)
    b1 = bench.algorithmic_bytes("screen", wl, _cfg(), touched_per_launch=1000.0)
    assert b1 - b0 == 1000 * (2 * 128 * 4 + 2 * 2 * 8 * 16 * 4)
    # EMA centres: the screen only assigns (no values, codebooks or slot rows)
    e = bench.algorithmic_bytes("screen", wl, _cfg(), touched_per_launch=1000.0, ema=True)
    assert e == 112 * (196 * 128 * 2 + 256 * bench.CACHE_BYTES + 196 * 4)


def _recorded():
    text = open(os.path.join(ROOT, "profiles", "hot_path_kernels_7b_traffic.md")).read()
    return [json.loads(b) for b in re.findall(r"```json\n(.*?)\n```", text, re.S)]


def test_recorded_traffic_needs_the_recorded_source(monkeypatch):
    recs = _recorded()
    assert recs, "no traffic records"
    wl = W.WORKLOADS["7b"]
    for rec in recs:
        monkeypatch.setattr(bench, "kernel_source_hash", lambda k, h=rec["source_sha256"]: h)
        got = bench.recorded_traffic(rec["kernel"], wl)
        assert got is not None and got["traffic_bytes_per_launch"] == rec["traffic_bytes_per_launch"]
        monkeypatch.setattr(bench, "kernel_source_hash", lambda k: "0" * 64)
        assert bench.recorded_traffic(rec["kernel"], wl) is None
    # another workload has no record
    monkeypatch.setattr(bench, "kernel_source_hash", lambda k, h=recs[0]["source_sha256"]: h)
    assert bench.recorded_traffic(recs[0]["kernel"], W.WORKLOADS["tiny"]) is None
