"""Pins of the oracle's variance-aware pseudo-token allocation (appendix
"Dynamic Pseudo-Token Allocation": S_k = S_tot Var(H_k) / sum_j Var(H_j)
under the fixed total S_tot = K_max S).

Var(H_k) is checked against numpy's weighted mean and variance of the
codewords, per subspace, and against closed forms; the allocation against
exact rational arithmetic, its fixed total, its bounds and the special
cases the passage fixes (equal variances give every prototype S).  No GPU.
"""
import fractions
import math

import numpy as np
import pytest

from oracle import protokv_oracle as O

F32 = np.float32


def _bank(p, rng, n_active, nres_max=40, zero_every=0):
    b = O.Bank(p)
    for k in range(n_active):
        b.n[k] = int(rng.integers(1, 60))
        nres = 0 if (zero_every and k % zero_every == 0) else int(rng.integers(1, nres_max))
        b.n_res[k] = nres
        for h in (b.hist_k, b.hist_v):
            for g in range(p.G):
                # concentrated or spread code distributions
                conc = rng.random() < 0.5
                w = rng.dirichlet(np.full(p.C, 0.2 if conc else 2.0))
                h[k, g] = rng.multinomial(nres, w) if nres else 0
    return b


def _params(**kw):
    base = dict(head_dim=128, grid_h=2, grid_w=2, window_frames=1, capacity=40, kv_dtype="fp32")
    base.update(kw)
    return O.Params(**base)


def test_residual_variance_is_numpys_weighted_variance_of_the_codewords():
    p = _params()
    rng = np.random.default_rng(0)
    cb = rng.standard_normal((2, p.G, p.C, 16)).astype(F32)
    b = _bank(p, rng, 33, zero_every=7)
    var = O.residual_variance(b, cb)
    for k in range(p.capacity):
        if b.n_res[k] == 0:
            assert var[k] == 0.0
            continue
        ref = 0.0
        for side, h in ((0, b.hist_k), (1, b.hist_v)):
            for g in range(p.G):
                cw = cb[side, g].astype(np.float64)
                wts = h[k, g].astype(np.float64)
                mean = np.average(cw, axis=0, weights=wts)
                ref += float(np.average((cw - mean) ** 2, axis=0, weights=wts).sum())
        assert abs(var[k] - ref) <= 1e-12 * max(ref, 1.0), (k, var[k], ref)


def test_residual_variance_closed_forms():
    """All residual mass on one codeword per subspace: no variance.  Half on
    codeword a, half on b in one subspace of one side: |a - b|^2 / 4."""
    p = _params(capacity=3)
    rng = np.random.default_rng(1)
    cb = rng.standard_normal((2, p.G, p.C, 16)).astype(F32)
    b = O.Bank(p)
    b.n[:2] = 10
    b.n_res[:2] = 8
    b.hist_k[0, :, 3] = 8
    b.hist_v[0, :, 5] = 8
    b.hist_k[1, :, 0] = 8
    b.hist_v[1, :, 0] = 8
    b.hist_v[1, 2, 0] = 4
    b.hist_v[1, 2, 7] = 4
    var = O.residual_variance(b, cb)
    assert var[0] == 0.0
    d = cb[1, 2, 0].astype(np.float64) - cb[1, 2, 7].astype(np.float64)
    assert abs(var[1] - float(d @ d) / 4.0) < 1e-12
    assert var[2] == 0.0


def _exact_shares(var, S, s_max):
    """Real shares by water-filling in exact rationals (the reading without
    any rounding)."""
    A = len(var)
    total = A * S
    capped = set()
    while True:
        rest = fractions.Fraction(total - A - len(capped) * (s_max - 1))
        w = sum(fractions.Fraction(float(var[k])) for k in range(A) if k not in capped)
        nunc = A - len(capped)
        x = [fractions.Fraction(s_max) if k in capped else
             (1 + rest * fractions.Fraction(float(var[k])) / w if w > 0 else 1 + rest / nunc) for k in range(A)]
        over = [k for k in range(A) if k not in capped and x[k] > s_max]
        if not over:
            return x
        capped.update(over)


@pytest.mark.parametrize("seed,S,s_max", [(2, 8, 16), (3, 8, 8 + 3), (4, 3, 16), (5, 8, 9)])
def test_allocation_keeps_the_total_and_follows_the_exact_shares(seed, S, s_max):
    rng = np.random.default_rng(seed)
    A = 57
    var = rng.gamma(0.5, 1.0, A)
    var[::9] = 0.0
    out = O.allocate_pseudo(var, S, s_max)
    assert sum(out) == A * S
    assert all(1 <= s <= s_max for s in out)
    x = _exact_shares(var, S, s_max)
    cum, prev = fractions.Fraction(0), 0
    for k in range(A):
        assert abs(out[k] - x[k]) < 1, (k, out[k], float(x[k]))
        cum += x[k]
        # cumulative rounding: the running total stays within 1/2 of the shares'
        assert abs(prev + out[k] - cum) <= fractions.Fraction(1, 2) + fractions.Fraction(1, 10 ** 9)
        prev += out[k]
    # a prototype capped in the exact shares is at s_max
    for k in range(A):
        if x[k] == s_max:
            assert out[k] == s_max


def test_allocation_special_cases():
    # equal variances: the fixed allocation, S for every prototype
    assert O.allocate_pseudo([0.7] * 11, 8, 16) == [8] * 11
    # no variance at all: S for every prototype
    assert O.allocate_pseudo([0.0] * 5, 8, 16) == [8] * 5
    # one prototype holds all the variance: capped, the rest share equally
    out = O.allocate_pseudo([0.0, 5.0, 0.0, 0.0], 8, 16)
    assert out[1] == 16 and sum(out) == 32 and sorted(out[::2] + [out[3]])[0] >= 5
    assert O.allocate_pseudo([], 8, 16) == []
    # a share of 1 + 28 * 5 / 8 = 18.5 is capped at 16; the 13 left go equally
    # to the three others (5.33 each), cumulatively rounded to 5, 6, 5
    assert O.allocate_pseudo([1.0, 1.0, 1.0, 5.0], 8, 16) == [5, 6, 5, 16]
    # two prototypes, variances 1 : 3, S = 4: shares 1 + 6/4 = 2.5 and 1 + 18/4 = 5.5
    assert O.allocate_pseudo([1.0, 3.0], 4, 16) == [3, 5]


def test_synthesis_gives_each_prototype_its_top_sk_modes():
    """With the allocation each slot's rows are its top-S_k tuples (the first
    S_k of its top-s_max list), all with bias ln n_k; the total row count is
    A * S; with equal variances the rows are those of the fixed S."""
    p = _params(capacity=30, var_alloc=True, s_max=12, S=6)
    rng = np.random.default_rng(6)
    cb = rng.standard_normal((2, p.G, p.C, 16)).astype(F32)
    b = _bank(p, rng, 30, zero_every=11)
    b.sum_k[:30] = rng.standard_normal((30, 128)).astype(F32)
    b.sum_v[:30] = rng.standard_normal((30, 128)).astype(F32)
    ps = O.synthesize(b, cb, p)
    counts = O.pseudo_counts(b, cb, p)
    assert len(ps.keys) == 30 * p.S == int(counts.sum())
    full = O.synthesize(b, cb, O.dataclasses.replace(p, var_alloc=False, S=p.s_max))
    row = 0
    for k in range(30):
        n = int(counts[k])
        assert np.array_equal(ps.slots[row:row + n], np.full(n, k))
        assert np.array_equal(ps.keys[row:row + n], full.keys[k * p.s_max:k * p.s_max + n])
        assert np.array_equal(ps.values[row:row + n], full.values[k * p.s_max:k * p.s_max + n])
        assert np.allclose(ps.bias[row:row + n], math.log(b.n[k]))
        row += n
    assert len(set(counts[:30].tolist())) > 2
    # equal variances: every slot with the same histograms
    b2 = O.Bank(p)
    b2.n[:30], b2.n_res[:30] = b.n[:30], 7
    b2.hist_k[:30] = b.hist_k[1]
    b2.hist_v[:30] = b.hist_v[1]
    b2.hist_k[:30] = 0
    b2.hist_k[:30, :, 2] = 5
    b2.hist_k[:30, :, 4] = 2
    b2.hist_v[:30] = b2.hist_k[:30]
    b2.sum_k[:30], b2.sum_v[:30] = b.sum_k[:30], b.sum_v[:30]
    a = O.synthesize(b2, cb, p)
    f = O.synthesize(b2, cb, O.dataclasses.replace(p, var_alloc=False))
    assert np.array_equal(a.keys, f.keys) and np.array_equal(a.values, f.values)
