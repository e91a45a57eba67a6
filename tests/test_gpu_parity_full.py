"""GPU parity at the full sizes of the paper-shaped workloads.

Every unit of every stream runs on the GPU in the launch configuration that
bench.py times (default config, one batched append + fold per frame).  The
oracle follows sampled units: over the whole stream where it can afford it
(7B workload), else by per-frame re-sync (the oracle folds a sampled unit
starting from the GPU's own pre-fold bank and must reproduce the GPU's fold
exactly).  Each test prints its case before any GPU step.
"""
import numpy as np
import pytest

from paper_2606_26762_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26762_amd import protokv as pk
    pk.lib()
    yield


def H():
    from tests import gpu_harness
    return gpu_harness


def test_7b_full_stream_sampled_units():
    """28 layers x 4 kv heads, K=256, W=8 frames, 256 frames: the oracle follows
    units 0, 37, 74, 111 over the whole stream (same bytes); banks bitwise at
    the end, synthesis exact, readout within 2e-2."""
    h = H()
    wl = W.WORKLOADS["7b"]
    sample = [0, 37, 74, 111]
    h.log(f"case: {wl.name} full stream, oracle units {sample}")
    pair = h.Pair(wl, sample=sample)
    for f in range(wl.frames):
        pair.step()
        if f == 12:
            pair.check_bank(bitwise=True)
    pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(3)), pseudo)
    c = pair.gpu.counters()
    h.log(f"assignments checked {pair.assign_checked}, near ties {pair.near_ties}, "
          f"refined {c.refined}+{c.refined_full}, readout max abs err {worst:.2e}")
    assert pair.assign_checked == len(sample) * (wl.frames - wl.window_frames) * wl.tokens_per_frame


def _resync_run(h, wl, sample, check_frames, frames=None, streams=1, readout_streams=(0,), **kw):
    frames = frames or wl.frames
    r = h.Resync(wl, sample, streams=streams, **kw)
    for f in range(frames):
        r.step(check=f in check_frames)
    worst = max(r.check_readout(s) for s in readout_streams)
    c = r.gpu.counters()
    h.log(f"folds re-checked {r.folds_checked}, near ties {r.near_ties}, "
          f"refined {c.refined}+{c.refined_full}, readout max abs err {worst:.2e}")
    expect = len(sample) * sum(1 for f in check_frames if wl.window_frames <= f < frames)
    assert r.folds_checked == expect
    return r


def test_long_delay_full_stream_resync():
    """28x4 units, K=1024, W=16 frames, 4096 frames with a cue cluster only in
    frames 100-102: re-sync checks at the first evictions, the end of seeding,
    the cue's eviction and late frames; readout after frame 4095."""
    h = H()
    wl = W.WORKLOADS["long"]
    sample = [(0, 0), (0, 57), (0, 111)]
    checks = {16, 21, 22, 116, 117, 118, 2048, wl.frames - 1}
    h.log(f"case: {wl.name} re-sync at frames {sorted(checks)}, units {sample}")
    r = _resync_run(h, wl, sample, checks)
    info = r.gpu.stream_info(0)
    assert info.active_slots == wl.capacity
    assert info.evicted_tokens == (wl.frames - wl.window_frames) * wl.tokens_per_frame


def test_hires_full_stream_resync():
    """32 layers x 8 kv heads, 24x24 grid (576 tokens/frame), K=2048, W=8,
    1024 frames: re-sync at the first eviction, the partial-seed frame, and
    late frames; readout after frame 1023."""
    h = H()
    wl = W.WORKLOADS["hires"]
    sample = [(0, 0), (0, 255)]
    checks = {8, 11, 12, 700, wl.frames - 1}
    h.log(f"case: {wl.name} re-sync at frames {sorted(checks)}, units {sample}")
    _resync_run(h, wl, sample, checks)


def test_multistream_full_shape_resync():
    """64 streams x 28x4 units, K=512, W=8, round-robin batched appends (one
    frame of every stream per call) for 24 rounds: re-sync of three
    (stream, unit) pairs across the seeding boundary and after; readout of
    stream 37."""
    h = H()
    wl = W.WORKLOADS["multi"]
    sample = [(0, 0), (37, 50), (63, 111)]
    checks = {8, 10, 11, 23}
    h.log(f"case: {wl.name} 64 streams x 24 rounds, re-sync at {sorted(checks)}, pairs {sample}")
    _resync_run(h, wl, sample, checks, frames=24, streams=wl.streams, readout_streams=(37,),
                cb_samples=256)


@pytest.mark.parametrize("S,frames", [(16, 40), (16, 345), (8, 345)])
def test_decode_wide_counts(S, frames):
    """One unit with K=1 and W=1 on the 7B frame shape: every evicted token
    lands in slot 0, so after 345 frames n_res > 65534 and the histogram
    products outgrow 128 bits (the decoder's wide path); 40 frames keep the
    register path.  Synthesis must be exact and the readout within 2e-2."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=1, num_q_heads=1, capacity=1,
                                  window_frames=1, frames=frames, query_tokens=4)
    h.log(f"case: {wl.name} K=1 W=1 S={S} frames={frames}")
    pair = h.Pair(wl, S=S, B=max(32, S))
    for f in range(frames):
        pair.step()
    gb = pair.check_bank(bitwise=True)
    n_res = int(gb["n_res"][0][0])
    assert (n_res > 65534) == (frames > 340), n_res
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(4)), pseudo)
    h.log(f"n_res {n_res}, readout max abs err {worst:.2e}")
