"""GPU parity: libprotokv (through its C-ABI) against the CPU oracle.

Each test names its workload (shape, seed) in its output before any GPU
step, so a failure names the case.
"""
import math

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


def test_tiny_stream_fp32_full():
    """1x1 head, fp32, 8x8 grid, 32 frames, window 4 frames, K=64 (whole stream)."""
    h = H()
    wl = W.WORKLOADS["tiny"]
    h.log(f"case: {wl.name}")
    pair = h.Pair(wl)
    for f in range(wl.frames):
        pair.step()
        if f in (4, 5, 12, wl.frames - 1):
            pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(1)), pseudo)
    c = pair.gpu.counters()
    h.log(f"assignments checked {pair.assign_checked}, near ties {pair.near_ties}, "
          f"refined {c.refined}+{c.refined_full}, readout max abs err {worst:.2e}")
    assert pair.assign_checked == (wl.frames - wl.window_frames) * wl.tokens_per_frame
    pair.check_near_tie_counter()


def test_7b_shape_one_layer():
    """7B shape on one layer (4 kv heads, 28 q heads): 196 tokens/frame, K=256,
    window 8 frames, 48 frames, bf16; every unit checked."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_q_heads=7 * 4, frames=48)
    h.log(f"case: {wl.name} L=1 frames=48")
    pair = h.Pair(wl)
    for f in range(wl.frames):
        pair.step()
    pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(2)), pseudo)
    c = pair.gpu.counters()
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties}, refined {c.refined}"
          f"+{c.refined_full}, touched {c.touched}, readout err {worst:.2e}")
    pair.check_near_tie_counter()


@pytest.mark.parametrize("wl_name", ["7b", "hires"])
def test_squared_mahalanobis(wl_name):
    """Eq. 1 with the squared spatial term (PROTOKV_FLAG_MAH_SQUARED): the 7B
    frame shape (persistent layout) and the high-resolution one (per-position
    spatial bias), one layer, every unit followed: assignments, banks bitwise,
    the near-tie counter, then the readout."""
    h = H()
    base = W.WORKLOADS[wl_name]
    wl = base.with_(num_layers=1, num_kv_heads=2, num_q_heads=2 * (base.num_q_heads // base.num_kv_heads),
                    frames=24 if wl_name == "hires" else 40)
    h.log(f"case: squared Mahalanobis {wl.name} L=1 Hkv=2 frames={wl.frames}")
    pair = h.Pair(wl, mah_squared=True)
    for f in range(wl.frames):
        pair.step()
    pair.check_bank(bitwise=True)
    pair.check_near_tie_counter()
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(17)), pseudo)
    c = pair.gpu.counters()
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties}, refined {c.refined}+{c.refined_full}, "
          f"readout err {worst:.2e}")


@pytest.mark.parametrize("kv,squared", [("bf16", True), ("fp32", False)])
def test_one_wave_screen_options(kv, squared):
    """The one-wave screen form (launches of 8 192 tiles or more: here 64
    streams x 32 units x 4 tiles of a 16x16 frame) with squared distances on
    bf16 keys and with float32 keys; K = 80, so the last slot tile is half
    rows past the active slots.  Two units of two streams are
    followed from the first frame: assignments every fold, banks bitwise,
    then the readout of each followed stream."""
    h = H()
    wl = W.WORKLOADS["multi"].with_(num_layers=1, num_kv_heads=32, num_q_heads=32, grid_h=16, grid_w=16,
                                    frames=12, window_frames=2, capacity=80, query_tokens=4, kv_dtype=kv)
    tracked, sample = [0, 63], [0, 31]
    h.log(f"case: one-wave screen {wl.name} kv={kv} squared={squared} streams={wl.streams} "
          f"units={wl.units} T={wl.tokens_per_frame} K={wl.capacity}")
    assert wl.streams * wl.units * ((wl.tokens_per_frame + 63) // 64) >= 8192
    pair = h.Pair(wl, sample=sample, streams=wl.streams, oracle_streams=tracked, cb_samples=256, cb_iters=4,
                  mah_squared=squared)
    for f in range(wl.frames):
        pair.step()
    for s in tracked:
        pair.check_bank(stream=s, bitwise=True)
        pseudo = pair.synthesize(stream=s)
        worst, *_ = pair.attend(pair.query(np.random.default_rng(40 + s)), pseudo, stream=s)
        h.log(f"stream {s}: readout err {worst:.2e}")
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties} (excused {pair.excused})")
    assert pair.assign_checked == len(tracked) * len(sample) * (wl.frames - wl.window_frames) * wl.tokens_per_frame


@pytest.mark.parametrize("case", ["7b", "tiny", "7b+rope", "ragged"])
def test_variance_aware_allocation(case):
    """PROTOKV_FLAG_VAR_ALLOC (appendix "Dynamic Pseudo-Token Allocation"):
    every slot's S_k equal to the oracle's allocation, the rows (top-S_k
    tuples at the running offsets) bitwise, then the readout; bf16 K=256
    S=8 up to 16, float32 S=3 up to 6, with rotary positions, and a ragged
    shape with C=12."""
    h = H()
    if case == "tiny":
        wl = W.WORKLOADS["tiny"].with_(frames=20)
        kw = dict(S=3, s_max=6)
    elif case == "ragged":
        wl = W.WORKLOADS["7b"].with_(num_layers=2, num_kv_heads=2, num_q_heads=6, grid_h=5, grid_w=7,
                                     frames=16, window_frames=2, capacity=20, query_tokens=5, clusters=6)
        kw = dict(S=5, s_max=9, C=12)
    else:
        wl = W.WORKLOADS["7b"].with_(num_layers=1, num_q_heads=28, frames=30)
        kw = dict(s_max=16)
        if case == "7b+rope":
            kw["rope_theta"] = 1e4
    h.log(f"case: variance-aware allocation {case} {wl.name} {kw}")
    pair = h.Pair(wl, var_alloc=True, **kw)
    for f in range(wl.frames):
        pair.step()
    pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(19)), pseudo)
    counts = [int(v) for v in np.bincount(pseudo[0].slots)]
    h.log(f"S_k range {min(counts)}..{max(counts)} over {len(counts)} slots, readout err {worst:.2e}")
    assert max(counts) > min(counts)


@pytest.mark.parametrize("cap", [4096, 4160])
def test_maximum_frame_and_query_sizes(cap):
    """The largest per-call shapes: 1024 tokens per frame (32x32 grid), 512
    query rows per kv head (64 query tokens x 8 query heads, two row blocks
    in the readout), with K = 4096 (32 768 pseudo tokens at S = 8, 128 slot
    tiles per screen workgroup) and K = 4160 (130 slot tiles, a seeding
    fold that leaves a partial tile).  Both read the pseudo-token biases from
    global memory in the readout (K above the 2048 staged in LDS).  The
    folds seed the bank to capacity, the last two assign at full K; every
    assignment, the bank (bitwise), the rows and the readout are checked.
    The library accepts capacities up to 65535; these are the largest the
    parity tests run."""
    h = H()
    frames = 1 + (cap + 1023) // 1024 + 2
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=1, num_q_heads=8, grid_h=32, grid_w=32,
                                  frames=frames, window_frames=1, capacity=cap, query_tokens=64)
    h.log(f"case: maximum sizes T={wl.tokens_per_frame} K={wl.capacity} rows={wl.query_tokens * 8}")
    pair = h.Pair(wl)
    for f in range(wl.frames):
        pair.step()
    assert pair.gpu.stream_info(0).active_slots == wl.capacity
    pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    worst, *_ = pair.attend(pair.query(np.random.default_rng(23)), pseudo)
    h.log(f"assignments {pair.assign_checked}, near ties {pair.near_ties}, readout err {worst:.2e}")
    assert pair.assign_checked == (wl.frames - wl.window_frames) * wl.tokens_per_frame


@pytest.mark.parametrize("cap,clusters", [(8, 4), (24, 3)])
def test_many_tokens_per_slot(cap, clusters):
    """Few slots, many tokens: T = 1024 (32x32) folded into K = 8 or 24
    slots over 3 or 4 clusters, so a fold gives one slot up to several
    hundred tokens.  The touched-slot aggregation buckets them by slot and
    absorbs each slot's tokens in eviction order: banks bitwise equal to the
    oracle's after every fold (the float32 sums depend on that order), then
    the rows and the readout."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=32, grid_w=32,
                                 frames=6, window_frames=1, capacity=cap, query_tokens=4, clusters=clusters)
    h.log(f"case: many tokens per slot T=1024 K={cap} clusters={clusters}")
    pair = h.Pair(wl)
    for f in range(wl.frames):
        pair.step()
        if f >= wl.window_frames:
            pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    pair.attend(pair.query(np.random.default_rng(29)), pseudo)
    st = pair.oracle[0]
    most = max(int(b.n.max()) for b in st.banks)
    h.log(f"largest slot mass {most}, near ties {pair.near_ties}")
    assert most > 4 * 1024 // cap


def test_ragged_shapes_seed_and_assign_same_fold():
    """T=35 (5x7, ragged tiles), K=20 < T (seed and assign in one fold),
    2 layers x 2 kv heads x 6 q heads, S=3, C=12, tq=5."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=2, num_kv_heads=2, num_q_heads=6, grid_h=5, grid_w=7,
                                 frames=14, window_frames=2, capacity=20, query_tokens=5,
                                 clusters=6)
    h.log("case: ragged T=35 K=20 L=2 Hkv=2 Hq=6 S=3 C=12")
    pair = h.Pair(wl, S=3, C=12)
    for f in range(wl.frames):
        pair.step()
        if f == wl.window_frames:
            pair.check_bank(bitwise=True)
    pair.check_bank(bitwise=True)
    pair.check_near_tie_counter()
    pseudo = pair.synthesize()
    for tq in (5, 1):
        pair.attend(pair.query(np.random.default_rng(3), tq=tq), pseudo)


@pytest.mark.parametrize("S", [5, 7, 16])
def test_formed_rows_across_s(S):
    """bf16 readout forming pseudo-token rows in LDS, S in {5, 7, 16}: T=49,
    W=3 (147 near rows, the near/pseudo boundary inside a 64-row tile), K=40,
    2 kv heads (several context splits, some holding one tile); readout with
    formed rows, then with the rows written back, both against the oracle."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=7, grid_w=7,
                                 frames=12, window_frames=3, capacity=40, query_tokens=6)
    h.log(f"case: formed rows S={S} T=49 W=3 K=40")
    pair = h.Pair(wl, S=S, B=max(32, S))
    for f in range(wl.frames):
        pair.step()
    pseudo = pair.synthesize()
    rng = np.random.default_rng(40 + S)
    q = pair.query(rng)
    w1, o1, _ = pair.attend(q, pseudo)      # formed rows
    w2, o2, _ = pair.attend(q, pseudo)      # rows written by read_pseudo
    h.log(f"readout err formed {w1:.2e} written {w2:.2e}, max diff {np.abs(o1 - o2).max():.2e}")


@pytest.mark.parametrize("grp,tq", [(8, 5), (7, 13), (4, 32), (3, 43)])
def test_readout_row_blocks(grp, tq):
    """bf16 readout over 40, 91, 128 and 129 query rows per kv head: up to
    128 rows two waves share each 32-row block (one per 32-key half of every
    tile) and merge at the end, partial blocks included; 129 rows take one
    wave per block.  T=49, W=3, K=40, S=8 (rows formed in LDS), 2 kv heads;
    readout against the oracle, formed and written rows."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=2 * grp, grid_h=7, grid_w=7,
                                 frames=12, window_frames=3, capacity=40, query_tokens=tq)
    h.log(f"case: readout rows {grp * tq} (grp {grp}, tq {tq})")
    pair = h.Pair(wl)
    for f in range(wl.frames):
        pair.step()
    pseudo = pair.synthesize()
    q = pair.query(np.random.default_rng(70 + grp))
    w1, o1, _ = pair.attend(q, pseudo)      # formed rows
    w2, o2, _ = pair.attend(q, pseudo)      # rows written by read_pseudo
    h.log(f"readout err formed {w1:.2e} written {w2:.2e}")


# K = 48: one row block, the exactly tested pairs all listed, 16-dim filter;
# K = 600: 8-dim filter, more filter pairs than the list holds (rows scanned);
# K = 1100: 4-dim filter, two row blocks (the first overflows, the second
# merges from its bitmask)
@pytest.mark.parametrize("eps_k,eps_v,grid,cap", [(1.0, 12.0, 6, 48), (1.5, 14.0, 6, 48),
                                                  (1.0, 12.0, 4, 600), (1.5, 14.0, 5, 1100)])
def test_maintenance_aging_merging_recycling(eps_k, eps_v, grid, cap):
    """Prototype maintenance after every fold (T_idle = 2 frames, gamma =
    0.3, merge thresholds that let same-cluster prototypes merge): banks
    bitwise equal to the oracle's after every fold, then the readout."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=grid, grid_w=grid,
                                 frames=14, window_frames=2, capacity=cap, query_tokens=4)
    h.log(f"case: maintenance eps_k={eps_k} eps_v={eps_v} T={grid * grid} K={cap} W=2")
    pair = h.Pair(wl, maintenance=True, t_idle=2, gamma=0.3, eps_k=eps_k, eps_v=eps_v)
    for f in range(wl.frames):
        pair.step()
        if f >= wl.window_frames:
            pair.check_bank(bitwise=True)
    c = pair.gpu.counters()
    h.log(f"aged {c.aged} merged {c.merged} recycled {c.recycled}, near ties {pair.near_ties}")
    assert c.aged > 0 and c.merged > 0 and c.recycled > 0
    pseudo = pair.synthesize()
    pair.attend(pair.query(np.random.default_rng(11)), pseudo)


@pytest.mark.parametrize("wl_name,alpha,beta", [("7b", 0.05, 0.05), ("tiny", 0.3, 0.7)])
def test_ema_centres(wl_name, alpha, beta):
    """Fixed-rate EMA centres (Alg. "ProtoKV Streaming Update" literally):
    banks bitwise equal to the oracle's after every fold (centres, squared
    sums, histograms of the residuals coded after each token's update,
    masses, spatial state), then the synthesized rows and the readout."""
    h = H()
    if wl_name == "7b":
        wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=6, grid_w=6,
                                     frames=14, window_frames=2, capacity=48, query_tokens=4)
    else:
        wl = W.WORKLOADS["tiny"].with_(frames=12)
    h.log(f"case: EMA centres {wl.name} alpha={alpha} beta={beta} T={wl.tokens_per_frame} K={wl.capacity}")
    pair = h.Pair(wl, ema=True, alpha=alpha, beta=beta)
    for f in range(wl.frames):
        pair.step()
        if f >= wl.window_frames:
            pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    pair.attend(pair.query(np.random.default_rng(13)), pseudo)


@pytest.mark.parametrize("wl_name,theta,grid", [("7b", 1e4, 6), ("7b", 1e6, 6), ("7b", 1e4, 24), ("tiny", 1e4, 8)])
def test_rope_readout(wl_name, theta, grid):
    """Rotary positions in the readout: near keys at their stream positions,
    the pseudo-keys of prototype k at tau_k, query token t at frames*T + t.
    Rows (rotated keys within one unit in the last place) and readout
    (abs 2e-2) against the oracle's float64 rotation."""
    h = H()
    if wl_name == "7b":
        wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=grid, grid_w=grid,
                                     frames=12, window_frames=2, capacity=48, query_tokens=4)
    else:
        wl = W.WORKLOADS["tiny"].with_(frames=10)
    h.log(f"case: RoPE {wl.name} theta={theta} T={wl.tokens_per_frame} K={wl.capacity}")
    pair = h.Pair(wl, rope_theta=theta)
    for f in range(wl.frames):
        pair.step()
    pseudo = pair.synthesize()
    q = pair.query(np.random.default_rng(17))
    # bf16 KV: the first readout forms the pseudo-keys in LDS and turns them
    # at tau_k there; the rows are then written (and checked against the
    # oracle) and the second readout reads them.  Both are checked against
    # the oracle; the written keys carry the same roundings as the formed
    # ones, so the two readouts differ only by their context splits.
    worst, go, _ = pair.attend(q, pseudo)
    w2, go2, _ = pair.attend(q, pseudo)
    h.log(f"readout err formed {worst:.2e} written {w2:.2e}, max diff {np.abs(go - go2).max():.2e}")
    # the rotation is visible at this tolerance: the unrotated readout of
    # the same bank is far from the GPU's
    st = pair.oracle[0]
    st.p.rope_theta = 0.0
    try:
        plain, _ = st.attend(q, wl.num_kv_heads, pseudo)
    finally:
        st.p.rope_theta = theta
    gap = max(float(np.abs(go[u // wl.num_kv_heads] - plain[u // wl.num_kv_heads]).max()) for u in pair.sample)
    h.log(f"readout abs err {worst:.2e}, distance from the unrotated readout {gap:.2e}")
    assert gap > 3 * h.READOUT_ATOL


@pytest.mark.parametrize("wl_name", ["7b", "tiny"])
def test_codebook_warmup(wl_name):
    """PQ codebook warm-up: the warm-up folds count no codes (banks bitwise
    equal to the oracle's after every fold), the codebooks learned from the
    reservoir are bitwise the oracle's, and the later folds code with them
    (banks bitwise), then the readout.  The bf16 case caps the reservoir
    below the residuals offered."""
    h = H()
    if wl_name == "7b":
        wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=6, grid_w=6,
                                     frames=12, window_frames=2, capacity=48, query_tokens=4)
        kw = dict(warm_frames=4, warm_tokens=64, kmeans_epochs=3, kmeans_batch=16)
    else:
        wl = W.WORKLOADS["tiny"].with_(frames=10)
        kw = dict(warm_frames=3, warm_tokens=1024, kmeans_epochs=2, kmeans_batch=64)
    h.log(f"case: codebook warm-up {wl.name} {kw}")
    pair = h.Pair(wl, **kw)
    given = pair.gpu.read_codebooks(0)
    learned = False
    for f in range(wl.frames):
        pair.step()
        if f >= wl.window_frames:
            pair.check_bank(bitwise=True)
            st = pair.oracle[0]
            if st.folds >= kw["warm_frames"]:
                cb = pair.gpu.read_codebooks(0)
                for i, u in enumerate(pair.sample):
                    assert np.array_equal(cb[u], st.codebooks[i]), f"unit {u}: learned codebooks differ"
                    assert not np.array_equal(cb[u], given[u])
                learned = True
    assert learned
    pseudo = pair.synthesize()
    pair.attend(pair.query(np.random.default_rng(19)), pseudo)


@pytest.mark.parametrize("case", ["maintenance+warmup+rope", "ema+rope"])
def test_combined_options(case):
    """The optional paths together: banks bitwise equal to the oracle's after
    every fold (through the warm-up, its k-means and maintenance merges), then
    the rows and the rotated readout."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=6, grid_w=6,
                                 frames=14, window_frames=2, capacity=48, query_tokens=4)
    if case == "ema+rope":
        kw = dict(ema=True, alpha=0.1, beta=0.2, rope_theta=1e4)
    else:
        kw = dict(maintenance=True, t_idle=2, gamma=0.3, eps_k=1.0, eps_v=12.0,
                  warm_frames=3, warm_tokens=200, kmeans_epochs=2, kmeans_batch=32, rope_theta=1e6)
    h.log(f"case: combined {case} {kw}")
    pair = h.Pair(wl, **kw)
    for f in range(wl.frames):
        pair.step()
        if f >= wl.window_frames:
            pair.check_bank(bitwise=True)
    if case != "ema+rope":
        c = pair.gpu.counters()
        assert c.merged > 0 and c.recycled > 0
        cb = pair.gpu.read_codebooks(0)
        for i, u in enumerate(pair.sample):
            assert np.array_equal(cb[u], pair.oracle[0].codebooks[i])
    pseudo = pair.synthesize()
    pair.attend(pair.query(np.random.default_rng(23)), pseudo)


def test_capacity_limit_gives_exact_attention():
    """K >= evicted tokens: every token keeps its own slot, and the readout is
    exact attention over the full history with far logits shifted by ln S
    (checked against torch SDPA on the CPU, independent of the oracle)."""
    import torch
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=4, grid_w=8,
                                 frames=10, window_frames=3, capacity=7 * 32, query_tokens=6)
    h.log("case: capacity limit T=32 K=224 frames=10 W=3")
    pair = h.Pair(wl)
    hist = []
    for f in range(wl.frames):
        gen = pair.host[0]
        pair.step()
    # rebuild the full history from the oracle's record of appended frames
    pseudo = pair.synthesize()
    q = pair.query(np.random.default_rng(4))
    worst, go, _ = pair.attend(q, pseudo)
    S = pair.p.S
    for i, u in enumerate(pair.sample):
        st = pair.oracle[0]
        b = st.banks[i]
        assert np.all(b.n[: (wl.frames - wl.window_frames) * 32] == 1)
        far_k = b.sum_k[b.n > 0]
        far_v = b.sum_v[b.n > 0]
        kn, vn = st.near(i)
        keys = np.concatenate([far_k, kn]).astype(np.float64)
        vals = np.concatenate([far_v, vn]).astype(np.float64)
        mask = np.concatenate([np.full(len(far_k), math.log(S)), np.zeros(len(kn))])
        l, hk = divmod(u, wl.num_kv_heads)
        grp = wl.num_q_heads // wl.num_kv_heads
        for g in range(grp):
            qh = torch.tensor(q[l][:, hk * grp + g].astype(np.float64))[None, None]
            ref = torch.nn.functional.scaled_dot_product_attention(
                qh, torch.tensor(keys)[None, None], torch.tensor(vals)[None, None],
                attn_mask=torch.tensor(mask)[None, None, None, :])[0, 0].numpy()
            assert np.abs(go[l][:, hk * grp + g] - ref).max() <= 2e-2


def test_duplicate_tokens_force_exact_ties():
    """All tokens of every frame share one key and value (lambda_sp = 0), so
    in the first assigning fold every slot has the same cost: the exact tie
    goes to the lowest slot on both sides.  Later folds stay in parity up to
    counted near ties."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=1, num_q_heads=1, grid_h=4, grid_w=4,
                                 frames=9, window_frames=2, capacity=8, query_tokens=4)
    h.log("case: forced ties T=16 K=8")
    pair = h.Pair(wl, lambda_sp=0.0)
    orig = pair.host[0].next_frame

    def dup_frame():
        k, v = orig()
        k[:] = k[:, :1]
        v[:] = v[:, :1]
        return k, v
    pair.host[0].next_frame = dup_frame
    for f in range(wl.window_frames + 1):
        pair.step()
    ga = pair.gpu.read_assignments(0)
    assert ga[0][:8].tolist() == list(range(8))   # seeds
    assert np.all(ga[0][8:] == 0)                 # exact tie -> lowest slot
    for f in range(wl.frames - wl.window_frames - 1):
        pair.step()
    pair.check_bank()
    h.log(f"near ties {pair.near_ties}, gpu counter {pair.gpu.counters().near_ties}, resyncs {pair.resyncs}")
    assert pair.near_ties > 0
    pair.check_near_tie_counter()


@pytest.mark.parametrize("use_pq,mass_bias", [(False, True), (True, False)])
def test_ablation_switches(use_pq, mass_bias):
    """'w/o residual stats' (PQ off) and 'b_k = 0' (mass bias off)."""
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=7, grid_w=7,
                                 frames=16, window_frames=3, capacity=64, query_tokens=8)
    h.log(f"case: ablation use_pq={use_pq} mass_bias={mass_bias}")
    pair = h.Pair(wl, use_pq=use_pq, mass_bias=mass_bias)
    for f in range(wl.frames):
        pair.step()
    pair.check_bank(bitwise=True)
    pseudo = pair.synthesize()
    pair.attend(pair.query(np.random.default_rng(5)), pseudo)


def test_multi_stream_round_robin():
    """3 independent streams appended in one batched call per round, plus a
    round where only stream 1 advances; per-stream parity."""
    h = H()
    wl = W.WORKLOADS["multi"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=6, grid_w=6,
                                    frames=12, window_frames=2, capacity=48, query_tokens=4, streams=3)
    h.log("case: 3 streams T=36 K=48")
    pair = h.Pair(wl, streams=3)
    for f in range(8):
        pair.step()
    pair.step(streams=[1])
    pair.step(streams=[2, 0])
    pair.check_near_tie_counter()
    for s in range(3):
        pair.check_bank(stream=s, bitwise=True)
        pseudo = pair.synthesize(stream=s)
        pair.attend(pair.query(np.random.default_rng(6 + s)), pseudo, stream=s)


def test_state_machine_errors():
    import torch
    from paper_2606_26762_amd import protokv as pk
    h = H()
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=1, num_q_heads=1, grid_h=2, grid_w=2,
                                 frames=4, window_frames=1, capacity=4, query_tokens=2)
    h.log("case: state machine errors")
    pair = h.Pair(wl)
    g = pair.gpu
    q = torch.zeros((1, 2, 1, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(pk.ProtoKVError) as e:
        g.attend(0, q)                         # nothing appended
    assert e.value.status == 4
    pair.step()
    pair.step()                                # frame 1 evicts frame 0 -> folded by step
    k = torch.zeros((1, 1, 1, 4, 128), dtype=torch.bfloat16, device="cuda")
    g.append_frame([0], k, k)                  # pending eviction
    with pytest.raises(pk.ProtoKVError) as e:
        g.append_frame([0], k, k)
    assert e.value.status == 4
    with pytest.raises(pk.ProtoKVError) as e:
        g.synthesize(0)
    assert e.value.status == 4
    g.fold()
    with pytest.raises(pk.ProtoKVError) as e:
        g.attend(0, q)                         # no synthesis since the fold
    assert e.value.status == 4
    g.synthesize(0)
    g.attend(0, q)
    with pytest.raises(pk.ProtoKVError) as e:
        g.attend(0, torch.zeros((1, 3, 1, 128), dtype=torch.bfloat16, device="cuda"))  # tq > max
    assert e.value.status == 1
    with pytest.raises(pk.ProtoKVError) as e:
        g.append_frame([3], k, k)
    assert e.value.status == 1
    info = g.stream_info(0)
    assert (info.frames, info.pending, info.active_slots) == (3, 0, 4)
