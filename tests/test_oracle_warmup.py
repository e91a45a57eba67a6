"""Pins of the oracle's PQ codebook warm-up (appendix "PQ codebook
initialization": mini-batch k-means on a reservoir of residuals collected
during the first T_warm steps, per subspace and per key / value).

Each test checks against something other than the code under test: the
running mean that a per-centre rate 1/count must reproduce, cluster means
of well-separated data, a two-row batch where updating inside the batch
would change the second assignment, residuals rebuilt from a copy of the
bank taken before each fold, and the mass bookkeeping of the warm-up
folds.  No GPU is needed.
"""
import numpy as np
import pytest

from oracle import protokv_oracle as O
from paper_2606_26762_amd import workloads as W
from tests.test_oracle_pins import tiny_params, tiny_stream

F32 = np.float32


def test_single_centre_tracks_the_running_mean():
    """One centre: every row joins it, eta = 1/count makes it the running
    mean (the first row replaces the start value exactly); a second epoch
    presents every row again, so the mean is unchanged."""
    rng = np.random.default_rng(0)
    x = (rng.standard_normal((300, 16)) * 3 + 1).astype(F32)
    start = np.full((1, 16), 100.0, F32)
    for epochs in (1, 2):
        c = O.minibatch_kmeans(x, start, epochs, 64)
        assert np.all(np.abs(c[0] - x.astype(np.float64).mean(0)) <= 1e-4)
    one = O.minibatch_kmeans(x[:1], start, 1, 64)
    assert np.array_equal(one[0], x[0])


def test_separated_clusters_are_recovered():
    """C tight clusters far apart, stored cluster by cluster so that rows
    i * floor(N / C) start one centre in each: the centres end at the
    cluster means."""
    rng = np.random.default_rng(1)
    C, per = 16, 40
    means = rng.standard_normal((C, 16)) * 20
    x = np.concatenate([means[c] + 0.01 * rng.standard_normal((per, 16)) for c in range(C)]).astype(F32)
    init = x[np.arange(C) * (len(x) // C)]
    c = O.minibatch_kmeans(x, init, 3, 64)
    for k in range(C):
        assert np.all(np.abs(c[k] - x[k * per:(k + 1) * per].astype(np.float64).mean(0)) <= 1e-4)


def test_batch_rows_are_assigned_with_the_centres_at_batch_start():
    """Centres 0 and 10 (dim 0), one batch of rows 4.9 then 7.4: as the batch
    starts, 7.4 is nearer 10 (2.6 < 7.4), although after 4.9 has moved
    centre 0 to 4.9 it would be nearer centre 0 (2.5)."""
    c0 = np.zeros((2, 16), F32)
    c0[1, 0] = 10.0
    x = np.zeros((2, 16), F32)
    x[0, 0], x[1, 0] = 4.9, 7.4
    c = O.minibatch_kmeans(x, c0, 1, 2)
    assert c[0, 0] == F32(4.9) and c[1, 0] == F32(7.4)


def test_learned_codebooks_recover_each_subspace_and_side():
    """A reservoir whose every subspace holds C tight clusters stored block
    by block (different clusters per subspace and for keys and values):
    each learned codeword is its block's mean in that subspace and side."""
    p = tiny_params()
    rng = np.random.default_rng(2)
    C, per, G, Dp = p.C, 30, p.G, 16
    res = []
    for side in range(2):
        means = rng.standard_normal((G, C, Dp)) * 20
        rows = [np.concatenate([means[g, k] for g in range(G)]) + 0.01 * rng.standard_normal(G * Dp)
                for k in range(C) for _ in range(per)]
        res.append(np.array(rows, dtype=F32))
    cb = O.learn_codebooks(res[0], res[1], np.zeros((2, G, C, Dp), F32), p)
    for side in range(2):
        for g in range(G):
            for k in range(C):
                blk = res[side][k * per:(k + 1) * per, g * Dp:(g + 1) * Dp].astype(np.float64)
                assert np.all(np.abs(cb[side, g, k] - blk.mean(0)) <= 1e-4)


def _warm_stream(p, frames, seed=5):
    wl = tiny_stream(p, frames, seed=seed)
    cb = W.make_codebooks(wl, units=[0], samples=128, iters=2, G=p.G, C=p.C)
    return wl, cb, W.HostStream(wl, units=[0]), O.OracleStream(p, [0], cb)


def test_warmup_folds_count_no_codes_and_fill_the_reservoir():
    """During the warm-up folds histograms and n_res stay 0 and every
    non-seed token's residual joins the reservoir; afterwards n_res counts
    only the later folds' tokens and the codebooks have changed."""
    p = tiny_params(capacity=20, warm_frames=3, warm_tokens=10 ** 6)
    frames = 8
    wl, cb, gen, st = _warm_stream(p, frames)
    warm_tokens, post_tokens = 0, 0
    for _ in range(frames):
        folds_before = st.folds
        res = st.append_frame(*gen.next_frame())
        if res is None:
            continue
        r = res[0]
        n_rest = len(r.assign) - r.n_seed
        if folds_before < p.warm_frames:
            assert not st.banks[0].hist_k.any() and not st.banks[0].n_res.any()
            warm_tokens += n_rest
        else:
            post_tokens += n_rest
    assert warm_tokens > 0 and post_tokens > 0
    assert int(st.banks[0].n_res.sum()) == post_tokens
    assert len(st.reservoir[0][0]) == len(st.reservoir[0][1]) == warm_tokens
    assert not np.array_equal(st.codebooks[0], cb[0])


def test_reservoir_residuals_use_the_pre_fold_centres():
    """One warm-up fold into a bank whose slots are all taken: every residual
    equals the evicted key minus float32(sum / n) of its slot as it stood
    before the fold, not after it."""
    p = tiny_params(capacity=16, warm_frames=50, warm_tokens=10 ** 6)
    wl, cb, gen, st = _warm_stream(p, 12, seed=7)
    for _ in range(p.window_frames + 2):          # seeds fill the bank
        st.append_frame(*gen.next_frame())
    ring_oldest = st.rings[0][0]
    before = st.banks[0].copy()
    n0 = len(st.reservoir[0][0])
    r = st.append_frame(*gen.next_frame())[0]
    fe, ke, _ = ring_oldest
    got = st.reservoir[0][0][n0:]
    rest = np.arange(r.n_seed, len(r.assign))
    assert len(got) == len(rest) > 0
    for i, j in enumerate(rest):
        slot = r.assign[j]
        c = (before.sum_k[slot] / F32(before.n[slot])).astype(F32)
        assert np.array_equal(got[i], (ke[j] - c).astype(F32))


def test_too_few_residuals_keep_the_given_codebooks():
    p = tiny_params(capacity=20, warm_frames=2, warm_tokens=10)   # 10 < C = 16
    frames = 6
    wl, cb, gen, st = _warm_stream(p, frames)
    for _ in range(frames):
        st.append_frame(*gen.next_frame())
    assert len(st.reservoir[0][0]) <= 10
    assert np.array_equal(st.codebooks[0], cb[0])


def test_warmup_is_refused_with_ema_centres():
    with pytest.raises(ValueError):
        O.OracleStream(tiny_params(ema=True, warm_frames=2), [0], np.zeros((1, 2, 8, 16, 16), F32))
