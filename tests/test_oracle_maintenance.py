"""Pins of the oracle's prototype maintenance (Alg. "Prototype Maintenance").

Each test checks the maintenance pass against something other than its own
code: a parameter choice under which the algorithm does nothing, numbers
worked out by hand for a few slots, conservation of what a merge adds, the
strictness of the thresholds, and the order in which recycling takes the
near window's tokens.  No GPU is needed.
"""
import numpy as np
import pytest

from oracle import protokv_oracle as O
from tests.test_oracle_pins import run_stream, tiny_params, tiny_stream

F32 = np.float32
D = 128


def _params(**kw):
    base = dict(head_dim=D, grid_h=2, grid_w=2, window_frames=1, capacity=6, kv_dtype="fp32",
                maintenance=True, t_idle=3)
    base.update(kw)
    return O.Params(**base)


def _bank_with(p, rows):
    """A bank whose slots 0..len(rows)-1 hold (n, key centre, value centre,
    mu, tau): sums are n times the centres (exact for the small integers
    and binary fractions used here)."""
    b = O.Bank(p)
    for k, (n, ck, cv, mu, tau) in enumerate(rows):
        b.n[k] = n
        b.sum_k[k] = (np.asarray(ck, F32) * F32(n)).astype(F32)
        b.sum_v[k] = (np.asarray(cv, F32) * F32(n)).astype(F32)
        b.sq_k[k] = (np.asarray(ck, F32) ** 2 * F32(n)).astype(F32)
        b.sq_v[k] = (np.asarray(cv, F32) ** 2 * F32(n)).astype(F32)
        b.mu[k] = np.asarray(mu, F32)
        b.sigma[k] = np.array([1.0, 0.0, 1.0], F32)
        b.tau[k] = tau
        b.n_res[k] = n - 1
        b.hist_k[k, :, 0] = n - 1
        b.hist_v[k, :, 1] = n - 1
    return b


def _vec(*pairs):
    """A D-vector with the given (index, value) entries, zeros elsewhere."""
    v = np.zeros(D, F32)
    for i, x in pairs:
        v[i] = x
    return v


def _near(p, frame, seed=0):
    rng = np.random.default_rng(seed)
    T = p.tokens_per_frame
    return [(frame, rng.standard_normal((T, D)).astype(F32), rng.standard_normal((T, D)).astype(F32))]


def test_no_op_parameters_leave_the_stream_unchanged():
    """gamma = 0 (floor(n) = n) and eps = 0 (no distance is below 0): the
    pass changes nothing, so a stream with maintenance equals one without."""
    p_off = tiny_params(capacity=20, t_idle=1)
    p_on = tiny_params(capacity=20, t_idle=1, maintenance=True, gamma=0.0, eps_k=0.0, eps_v=0.0)
    frames = 10
    st_off, _, _ = run_stream(p_off, tiny_stream(p_off, frames), frames)
    st_on, _, _ = run_stream(p_on, tiny_stream(p_on, frames), frames)
    for name in ("n", "sum_k", "sum_v", "sq_k", "sq_v", "hist_k", "hist_v", "n_res", "mu", "sigma", "tau"):
        assert np.array_equal(getattr(st_off.banks[0], name), getattr(st_on.banks[0], name)), name


def test_aging_floors_the_mass_and_keeps_the_centre():
    """Idle means (t - frame(tau)) > T_idle.  With gamma = 0.05:
    floor(0.95 * 40) = 38 and floor(0.95 * 19) = 18; a slot idle by exactly
    T_idle frames is not aged.  Sums are scaled by n'/n, so the centre stays
    (here exactly: 38/40 and 18/19 times a multiple of n)."""
    p = _params(capacity=4, grid_h=2, grid_w=2)
    T = p.tokens_per_frame
    t = 10
    far = 5 * T                  # frame 5: 10 - 5 = 5 > 3, idle
    edge = (t - p.t_idle) * T    # frame 7: 10 - 7 = 3, not idle
    rows = [(40, _vec((0, 0.5)), _vec((1, 0.25)), (0.25, 0.25), far),
            (19, _vec((2, 1.0)), _vec((3, 2.0)), (0.75, 0.25), far),
            (7, _vec((4, 3.0)), _vec((5, 3.0)), (0.25, 0.75), edge)]
    b = _bank_with(p, rows)
    before = b.copy()
    st = O.maintain(b, _near(p, t), t, p)
    assert st["aged"] == 2 and st["merged"] == 0 and st["recycled"] == 0
    assert (b.n[0], b.n[1], b.n[2]) == (38, 18, 7)
    for k, n in ((0, 38), (1, 18)):
        assert np.allclose(b.sum_k[k] / F32(n), before.sum_k[k] / F32(before.n[k]), rtol=2e-7, atol=0)
        assert np.allclose(b.sum_v[k] / F32(n), before.sum_v[k] / F32(before.n[k]), rtol=2e-7, atol=0)
        assert np.array_equal(b.hist_k[k], before.hist_k[k]) and b.n_res[k] == before.n_res[k]
        assert np.array_equal(b.mu[k], before.mu[k]) and b.tau[k] == before.tau[k]
    for name in ("sum_k", "sum_v", "sq_k", "mu", "hist_k"):
        assert np.array_equal(getattr(b, name)[2], getattr(before, name)[2])


def test_aging_to_zero_recycles_from_the_newest_near_token():
    """n = 1 idle -> floor(0.95) = 0: the slot is empty and is reseeded from
    the newest near frame's first token (n = 1, sums = the token, Sigma = I,
    tau = its position, no residual statistics)."""
    p = _params(capacity=3)
    T = p.tokens_per_frame
    t = 9
    rows = [(1, _vec((0, 1.0)), _vec((0, 1.0)), (0.25, 0.25), 0),
            (5, _vec((1, 1.0)), _vec((1, 1.0)), (0.75, 0.75), t * T)]
    b = _bank_with(p, rows)
    near = _near(p, t - 1, seed=1) + _near(p, t, seed=2)   # oldest first
    st = O.maintain(b, near, t, p)
    assert st == {"aged": 1, "merged": 0, "recycled": 1, "near_threshold": 0}
    _, kt, vt = near[-1]
    assert b.n[0] == 1 and b.n_res[0] == 0 and b.tau[0] == t * T
    assert np.array_equal(b.sum_k[0], kt[0]) and np.array_equal(b.sum_v[0], vt[0])
    assert np.array_equal(b.sq_k[0], kt[0] * kt[0])
    assert np.array_equal(b.mu[0], np.array([0.25, 0.25], F32))   # cell (0, 0) centre on 2x2
    assert np.array_equal(b.sigma[0], np.array([1.0, 0.0, 1.0], F32))
    assert not b.hist_k[0].any() and not b.hist_v[0].any()
    assert b.n[2] == 0   # past the active prefix: left for seeding


def test_merge_adds_statistics_and_weights_the_spatial_mean():
    """Two slots with equal centres merge into the lower one: n, sums, squared
    sums, histograms and n_res add (conservation); mu = (3 mu_0 + 2 mu_1) / 5
    by hand; Sigma and tau of slot 0 stay; slot 1 is recycled."""
    p = _params(capacity=2, t_idle=1000)
    t = 4
    ck, cv = _vec((0, 0.5), (7, -0.25)), _vec((3, 0.5))
    rows = [(3, ck, cv, (0.25, 0.25), 4 * p.tokens_per_frame),
            (2, ck, cv, (0.75, 0.75), 4 * p.tokens_per_frame + 1)]
    b = _bank_with(p, rows)
    before = b.copy()
    b.sigma[0] = np.array([0.5, 0.125, 0.25], F32)
    st = O.maintain(b, _near(p, t), t, p)
    assert st == {"aged": 0, "merged": 1, "recycled": 1, "near_threshold": 0}
    assert b.n[0] == 5 and b.n_res[0] == before.n_res[0] + before.n_res[1]
    assert np.array_equal(b.sum_k[0], before.sum_k[0] + before.sum_k[1])
    assert np.array_equal(b.sq_v[0], before.sq_v[0] + before.sq_v[1])
    assert np.array_equal(b.hist_k[0], before.hist_k[0] + before.hist_k[1])
    assert np.array_equal(b.hist_v[0], before.hist_v[0] + before.hist_v[1])
    assert np.array_equal(b.mu[0], np.array([0.45, 0.45], F32))   # (3*0.25 + 2*0.75) / 5
    assert np.array_equal(b.sigma[0], np.array([0.5, 0.125, 0.25], F32)) and b.tau[0] == before.tau[0]
    assert b.n[1] == 1 and b.n_res[1] == 0   # recycled


@pytest.mark.parametrize("x2,merged", [(0.3, 1), (0.25, 2)])
def test_merge_uses_the_centre_updated_by_earlier_merges(x2, merged):
    """Key centres 0, 0.125 and x2 on one axis, masses 1, equal values:
    slot 0 absorbs slot 1 (0.125 < 0.2) and moves to 0.0625; slot 2 is then
    0.3 - 0.0625 = 0.2375 away (no merge) or 0.25 - 0.0625 = 0.1875 away
    (merge), although both are more than 0.2 from the original centre 0."""
    p = _params(capacity=3, t_idle=1000)
    t = 2
    tau = t * p.tokens_per_frame
    cv = _vec((1, 1.0))
    rows = [(1, _vec((0, 0.0)), cv, (0.25, 0.25), tau),
            (1, _vec((0, 0.125)), cv, (0.25, 0.25), tau),
            (1, _vec((0, x2)), cv, (0.25, 0.25), tau)]
    b = _bank_with(p, rows)
    st = O.maintain(b, _near(p, t), t, p)
    assert st["merged"] == merged
    assert b.n[0] == 1 + merged
    if merged == 1:
        assert b.n[2] == 1 and b.sum_k[2][0] == F32(0.3)   # untouched
    assert np.isclose(b.sum_k[0][0] / b.n[0], (0.125 + (x2 if merged == 2 else 0.0)) / b.n[0])


def test_merge_thresholds_are_strict_and_need_both_centres():
    """A key distance of exactly eps_K (0.25 with eps_K = 0.25 here, an exact
    binary value) does not merge; a close key with a value distance of 1 does
    not merge either."""
    p = _params(capacity=4, t_idle=1000, eps_k=0.25, eps_v=0.25)
    t = 2
    tau = t * p.tokens_per_frame
    rows = [(1, _vec((0, 0.0)), _vec((1, 0.0)), (0.25, 0.25), tau),
            (1, _vec((0, 0.25)), _vec((1, 0.0)), (0.25, 0.25), tau),   # key distance exactly 0.25
            (1, _vec((5, 2.0)), _vec((6, 0.0)), (0.25, 0.25), tau),
            (1, _vec((5, 2.0)), _vec((6, 1.0)), (0.25, 0.25), tau)]    # keys equal, values 1 apart
    b = _bank_with(p, rows)
    st = O.maintain(b, _near(p, t), t, p)
    assert st["merged"] == 0 and list(b.n[:4]) == [1, 1, 1, 1]


def test_recycling_takes_near_tokens_newest_frame_first_in_raster_order():
    """Three empty prefix slots (merged away) take tokens 0, 1, 2 of the
    newest near frame, in slot order."""
    p = _params(capacity=4, t_idle=1000)
    t = 3
    tau = t * p.tokens_per_frame
    c = _vec((0, 1.0))
    rows = [(1, c, c, (0.25, 0.25), tau)] * 4
    b = _bank_with(p, rows)
    near = _near(p, t - 1, seed=5) + _near(p, t, seed=6)
    st = O.maintain(b, near, t, p)
    assert st == {"aged": 0, "merged": 3, "recycled": 3, "near_threshold": 0}
    _, kt, vt = near[-1]
    T = p.tokens_per_frame
    for e, k in enumerate((1, 2, 3)):
        assert np.array_equal(b.sum_k[k], kt[e]) and b.tau[k] == t * T + e
    assert b.n[0] == 4


def test_merge_distance_is_the_squared_euclidean_distance():
    """The merge test's ||a - b||^2 against scipy's sqeuclidean on random float32
    centres (float64 sums agree to rounding), and a 3-4-5 case exactly."""
    import scipy.spatial.distance as ssd
    rng = np.random.default_rng(5)
    for _ in range(200):
        scale = 10.0 ** rng.uniform(-3, 2)
        a = (rng.standard_normal(D) * scale).astype(F32)
        b = (a + rng.standard_normal(D) * scale * rng.uniform(0, 1)).astype(F32)
        ref = ssd.sqeuclidean(a.astype(np.float64), b.astype(np.float64))
        assert abs(O._dist2(a, b) - ref) <= 1e-13 * ref
    assert O._dist2(_vec((0, 3.0)), _vec((1, 4.0))) == 25.0
    assert O._dist2(_vec((127, 0.5)), _vec()) == 0.25


def test_pair_on_the_threshold_is_counted_and_not_merged():
    """Key centres exactly eps_K apart (0.25^2 = 0.0625 is exact): the strict
    test keeps them apart, and the pair is counted as near-threshold."""
    p = _params(eps_k=0.25, eps_v=10.0, t_idle=100)
    rows = [(2, _vec((0, 0.5)), _vec((0, 1.0)), (0.25, 0.25), 0),
            (2, _vec((0, 0.75)), _vec((0, 1.0)), (0.25, 0.25), 0)]
    b = _bank_with(p, rows)
    st = O.maintain(b, _near(p, 1), 1, p)
    assert st["merged"] == 0 and st["near_threshold"] == 1
    assert b.n[0] == 2 and b.n[1] == 2
