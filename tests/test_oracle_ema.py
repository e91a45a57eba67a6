"""Pins of the oracle's fixed-rate EMA centres (Alg. "ProtoKV Streaming
Update": c <- (1 - alpha) c + alpha K, p <- (1 - beta) p + beta V, then the
residual statistics from K - c, V - p with the updated centres).

Each test checks the EMA mode against something other than its own code:
the geometric closed form of repeated updates, the exact limits alpha = 1
(the centre becomes the last token) and alpha = 0 (the centre stays), the
order dependence that distinguishes an EMA from a mean, a codebook built so
that the residual before and after the centre update fall on different
codewords, and synthesis from the stored centres.  No GPU is needed.
"""
import math

import numpy as np
import pytest

from oracle import protokv_oracle as O
from tests.test_oracle_pins import run_stream, tiny_params, tiny_stream

F32 = np.float32
D = 128


def _params(**kw):
    base = dict(head_dim=D, grid_h=2, grid_w=4, window_frames=1, capacity=1, kv_dtype="fp32", ema=True)
    base.update(kw)
    return O.Params(**base)


def _codebooks(p, rng=None):
    """Codebooks [2][G][C][D/G] with no special structure (fixed seed)."""
    rng = rng or np.random.default_rng(7)
    return rng.standard_normal((2, p.G, p.C, D // p.G)).astype(F32)


def _fold_one_slot(p, first, rest_k, rest_v, first_v=None, cb=None):
    """Capacity 1: token 0 seeds the slot, tokens 1.. are absorbed into it in
    eviction order.  Returns the bank."""
    T = p.tokens_per_frame
    keys = np.stack([first] + list(rest_k)).astype(F32)
    values = np.stack([first if first_v is None else first_v] + list(rest_v)).astype(F32)
    assert keys.shape == (T, D)
    b = O.Bank(p)
    O.fold_frame(b, keys, values, 0, 1, p, _codebooks(p) if cb is None else cb)
    return b


def test_repeated_token_follows_the_geometric_closed_form():
    """Seed K0, then m = T - 1 copies of x: c_m = (1-a)^m K0 + (1 - (1-a)^m) x
    (values with beta).  float32 rounding stays within m * 2^-22 relative."""
    p = _params(alpha=0.05, beta=0.2)
    rng = np.random.default_rng(1)
    k0, x = rng.standard_normal(D).astype(F32), rng.standard_normal(D).astype(F32)
    v0, y = rng.standard_normal(D).astype(F32), rng.standard_normal(D).astype(F32)
    m = p.tokens_per_frame - 1
    b = _fold_one_slot(p, k0, [x] * m, [y] * m, first_v=v0)
    for got, start, tok, rate in ((b.sum_k[0], k0, x, 0.05), (b.sum_v[0], v0, y, 0.2)):
        q = (1.0 - rate) ** m
        want = q * start.astype(np.float64) + (1.0 - q) * tok.astype(np.float64)
        scale = np.abs(start).astype(np.float64) + np.abs(tok)
        assert np.all(np.abs(got - want) <= m * 2.0 ** -22 * scale + 1e-30)
    assert b.n[0] == m + 1 and b.n_res[0] == m


def test_alpha_one_keeps_the_last_token_and_alpha_zero_keeps_the_seed():
    """alpha = 1: (1 - 1) c + 1 K = K exactly, so the centre is the last
    absorbed token; alpha = 0: 1 c + 0 K = c, so the centre is the seed."""
    rng = np.random.default_rng(2)
    toks = rng.standard_normal((8, D)).astype(F32)
    b1 = _fold_one_slot(_params(alpha=1.0, beta=1.0), toks[0], toks[1:], toks[1:][::-1])
    assert np.array_equal(b1.sum_k[0], toks[7])
    assert np.array_equal(b1.sum_v[0], toks[1])   # values absorbed in reverse here
    b0 = _fold_one_slot(_params(alpha=0.0, beta=0.0), toks[0], toks[1:], toks[1:])
    assert np.array_equal(b0.sum_k[0], toks[0]) and np.array_equal(b0.sum_v[0], toks[0])


def test_updates_follow_eviction_order():
    """An EMA depends on order: the centre equals the float64 recursion in
    eviction order (within rounding) and differs from the reversed order."""
    p = _params()
    rng = np.random.default_rng(3)
    toks = rng.standard_normal((8, D)).astype(F32) * F32(4)
    b = _fold_one_slot(p, toks[0], toks[1:], toks[1:])
    c = toks[0].astype(np.float64)
    for x in toks[1:]:
        c = 0.95 * c + 0.05 * x
    r = toks[0].astype(np.float64)
    for x in toks[1:][::-1]:
        r = 0.95 * r + 0.05 * x
    tol = 1e-5 * (np.abs(c) + 1)
    assert np.all(np.abs(b.sum_k[0] - c) <= tol)
    assert np.max(np.abs(c - r)) > 100 * np.max(tol)


def test_residual_is_taken_after_the_centre_update():
    """Two tokens: 0 seeds the slot, then x = e_0 is absorbed.  The key centre
    becomes alpha x, so the key residual is (1 - alpha) x = 0.95 e_0, not x;
    the value centre (beta = 0.5) becomes 0.5 x, residual 0.5 e_0.  In every
    subspace codeword 0 is e_0 (restricted) and 1 is 0.95 e_0; 0.5 e_0 is
    codeword 2 of the key codebook and 3 of the value codebook: subspace 0
    must count codeword 1 for the key and 3 for the value."""
    p = _params(beta=0.5, grid_h=1, grid_w=2)
    cb = np.full((2, p.G, p.C, D // p.G), 50.0, dtype=F32)
    for kv, c, x0 in ((0, 0, 1.0), (0, 1, 0.95), (0, 2, 0.5), (1, 0, 1.0), (1, 1, 0.95), (1, 3, 0.5)):
        cb[kv, :, c, :] = 0.0
        cb[kv, :, c, 0] = x0
    x = np.zeros(D, F32)
    x[0] = 1.0
    zero = np.zeros(D, F32)
    b = O.Bank(p)
    O.fold_frame(b, np.stack([zero, x]), np.stack([zero, x]), 0, 1, p, cb)
    assert b.n[0] == 2 and b.n_res[0] == 1
    assert b.sum_k[0, 0] == F32(0.05) and b.sum_v[0, 0] == F32(0.5)
    assert b.hist_k[0, 0, 1] == 1 and b.hist_k[0, 0].sum() == 1
    assert b.hist_v[0, 0, 3] == 1 and b.hist_v[0, 0].sum() == 1


def test_synthesis_uses_the_stored_centres():
    """With EMA centres the row fields are the centres: a slot of mass 5
    without residuals gives S pseudo-keys equal to c (not c / 5) and the
    bias ln 5; the running-mean reading of the same bank divides by 5."""
    p = _params(capacity=2)
    b = O.Bank(p)
    c = np.linspace(-1, 1, D).astype(F32)
    b.n[0] = 5
    b.sum_k[0] = c
    b.sum_v[0] = c[::-1].copy()
    ps = O.synthesize(b, _codebooks(p), p)
    assert len(ps.keys) == p.S
    assert np.all(ps.keys == c) and np.all(ps.values == c[::-1])
    assert np.allclose(ps.bias, math.log(5))
    pm = _params(capacity=2, ema=False)
    assert np.array_equal(O.synthesize(b, _codebooks(pm), pm).keys[0], (c / F32(5)).astype(F32))


def test_stream_conserves_mass_and_squared_sums():
    """A short stream with EMA centres: masses count the evicted tokens,
    residual counts the absorbed ones, and the squared sums stay the sums of
    the squared members (the EMA changes the centres only)."""
    p = tiny_params(ema=True, capacity=6)
    frames = 8
    st, log, _ = run_stream(p, tiny_stream(p, frames), frames)
    b = st.banks[0]
    evicted = sum(len(res.assign) for _, _, _, res in log)
    assert int(b.n.sum()) == evicted
    seeded = sum(res.n_seed for _, _, _, res in log)
    assert int(b.n_res.sum()) == evicted - seeded
    sq = np.zeros_like(b.sq_k, dtype=np.float64)
    for _, ke, _, res in log:
        for j, k in enumerate(res.assign):
            sq[k] += ke[j].astype(np.float64) ** 2
    assert np.allclose(b.sq_k, sq, rtol=1e-5, atol=1e-5)
    assert np.all(b.hist_k.sum(axis=2) == b.n_res[:, None])


def test_maintenance_is_refused_with_ema_centres():
    with pytest.raises(ValueError):
        O.OracleStream(tiny_params(ema=True, maintenance=True), [0], np.zeros((1, 2, 8, 16, 16), F32))
