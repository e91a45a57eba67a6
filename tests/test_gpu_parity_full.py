"""GPU parity at the full sizes of the paper-shaped workloads.

Every unit of every stream runs on the GPU in the launch configuration that
bench.py times (default config, one batched append + fold per frame).  The
oracle follows sampled units free-running (it is authoritative: after an
excused near tie the device's state of those units is replaced by the
oracle's) over the whole 7B stream and over the first hundreds of frames of
the long-delay, high-resolution and 64-stream workloads.  Over the full
length of those three the device runs alone; single folds are checked
against the oracle from the device's own pre-fold state at chosen frames,
and at the end every unit of every stream must satisfy the mass, histogram
and residual-count identities.  Each test prints its case before any GPU
step.
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
        if f % 512 == 511:
            h.log(f"frame {f + 1}")
    worst = max(r.check_readout(s) for s in readout_streams)
    r.check_invariants()
    c = r.gpu.counters()
    h.log(f"folds re-checked {r.folds_checked}, near ties {r.near_ties} (excused {r.excused}), "
          f"refined {c.refined}+{c.refined_full}, readout max abs err {worst:.2e}")
    expect = len(sample) * sum(1 for f in check_frames if wl.window_frames <= f < frames)
    assert r.folds_checked == expect
    return r


def test_long_delay_free_running_through_the_cue():
    """Long-delay workload (K=1024, W=16), one unit followed by the oracle from
    the first frame through frame 320: seeding, the rare cue cluster in frames
    100-102 and its eviction at frames 116-118, then 200 more folds.  Every
    assignment is checked, banks bitwise at the cue's eviction and at the end,
    and a query whose last half is aligned with the cue cluster's mean is
    read out."""
    h = H()
    wl = W.WORKLOADS["long"].with_(frames=320)
    h.log(f"case: {wl.name} free-running through frame 320, unit 57")
    pair = h.Pair(wl, sample=[57])
    for f in range(wl.frames):
        pair.step()
        if f in (119, 319):
            pair.check_bank(bitwise=True)
        if f % 100 == 99:
            h.log(f"frame {f + 1}")
    pseudo = pair.synthesize()
    q = pair.query(np.random.default_rng(31))
    l, hk = divmod(57, wl.num_kv_heads)
    grp = wl.num_q_heads // wl.num_kv_heads
    cue = pair.host[0]._heads[57].means[0]
    q[l, wl.query_tokens // 2:, hk * grp:(hk + 1) * grp] += 4.0 * np.sqrt(wl.head_dim) * cue
    q = W.quantize(q, wl.kv_dtype)
    worst, *_ = pair.attend(q, pseudo)
    b = pair.oracle[0].banks[0]
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties} (excused {pair.excused}, "
          f"resyncs {pair.resyncs}), active {(b.n > 0).sum()}, readout err {worst:.2e}")
    assert pair.assign_checked == (wl.frames - wl.window_frames) * wl.tokens_per_frame


def test_hires_free_running():
    """High-resolution workload (576 tokens/frame, K=2048, W=8), one unit
    followed by the oracle over 40 frames: the bank fills on the 4th fold, then
    28 folds assign 576 tokens against 2048 slots; banks bitwise, readout."""
    h = H()
    wl = W.WORKLOADS["hires"].with_(frames=40)
    h.log(f"case: {wl.name} free-running 40 frames, unit 200")
    pair = h.Pair(wl, sample=[200])
    for f in range(wl.frames):
        pair.step()
    pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(32)), pseudo)
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties} (excused {pair.excused}), "
          f"readout err {worst:.2e}")


def test_multistream_free_running_with_queries():
    """The 64-stream workload (K=512, W=8) in its launch pattern: one batched
    append of every stream and one fold per round, for 136 rounds, and the
    queries of the schedule (stream b at rounds r with (r - 2b) mod 128 = 127).
    The oracle follows unit 90 of streams 0 and 37 from the first frame; the
    queries of those streams (rounds 73 and 127) are checked against it."""
    h = H()
    wl = W.WORKLOADS["multi"]
    tracked = [0, 37]
    h.log(f"case: {wl.name} 136 rounds, oracle on unit 90 of streams {tracked}")
    pair = h.Pair(wl, sample=[90], streams=wl.streams, oracle_streams=tracked, cb_samples=256, cb_iters=4)
    checked = 0
    for r in range(136):
        pair.step()
        b = (r - 127) % 128
        if b % 2 == 0 and b // 2 < wl.streams:
            s = b // 2
            if s in tracked:
                pair.check_bank(stream=s, bitwise=True)
                pseudo = pair.synthesize(stream=s)
                worst, *_ = pair.attend(pair.query(np.random.default_rng(r)), pseudo, stream=s)
                h.log(f"round {r}: stream {s} readout err {worst:.2e}")
                checked += 1
            else:
                pair.gpu.synthesize(s)
                pair.gpu.attend(s, pair.torch.zeros((wl.num_layers, wl.query_tokens, wl.num_q_heads, 128),
                                                    dtype=pair.dtype, device="cuda"))
    assert checked == 2
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties} (excused {pair.excused})")
    assert pair.assign_checked == len(tracked) * (136 - wl.window_frames) * wl.tokens_per_frame


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
