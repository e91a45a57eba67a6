"""Host check of the screen's float32 spatial-term error bound (Eq. 1's
Mahalanobis distance).

The screen writes the quadratic form of (Sigma + rho I)^-1 as
q = (la dx + lb dy)^2 + (lc dy)^2, evaluates it in float32 as
u = fma(lb, dy, la * dx), q' = fma(u, u, (lc * dy)^2), d' = sqrt(q') (raw, ~1 ulp),
and bounds the error by eps_k * d + 2e-15 with
eps_k = 1.02 (8 + 5 rho) 2^-24 + 2.5e-7 (squared distances:
1.02 (16 + 10 rho) 2^-24 on q), rho = |B| / sqrt(det), stored rounded up by
0.1%.  This test replays that float32 sequence in numpy (a fused multiply-add
as one rounding of the exact float64 value, the hardware square root as the
correctly rounded one moved one ulp either way) on random
covariances from isotropic to nearly singular and positions from the centre
itself to far away, and checks every result against the float64 distance
from the same float32 positions.  It pins the derivation, not the kernel: the
GPU parity tests check the kernel's assignments against the oracle.
"""
import numpy as np

U = 2.0 ** -24


def f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def fma32(a, b, c):
    # a * b is exact in float64 for float32 operands; one rounding to float32
    # of the float64 sum stands in for the fused operation (the double
    # rounding it can add is far inside the bound's 2% margin)
    return f32(a.astype(np.float64) * b.astype(np.float64) + c.astype(np.float64))


def meta(sxx, sxy, syy, ridge, squared):
    """Float64 factors and error bound of one slot, as the screening meta holds them."""
    A, B, Cc = sxx + ridge, sxy, syy + ridge
    det = A * Cc - B * B
    rd, rc = 1.0 / np.sqrt(det), 1.0 / np.sqrt(Cc)
    rho = np.abs(B) * rd
    eq = (16.0 + 10.0 * rho) * U * 1.02
    eps = (eq if squared else 0.5 * eq + 2.5e-7) * 1.001
    return f32(Cc * rc * rd), f32(-B * rc * rd), f32(rc), f32(eps), (A, B, Cc, det)


def screen_term(tx, ty, mx, my, la, lb, lc, squared, sqrt_shift):
    dx = f32(tx - mx)  # float32 subtraction: exact difference, one rounding
    dy = f32(ty - my)
    u = fma32(lb, dy, f32(la * dx))
    v = f32(lc * dy)
    q = fma32(u, u, f32(v * v))
    if squared:
        return q
    d = f32(np.sqrt(q.astype(np.float64)))
    return np.where(sqrt_shift > 0, np.nextafter(d, np.float32(np.inf)),
                    np.where((sqrt_shift < 0) & (d > 0), np.nextafter(d, np.float32(0)), d)).astype(np.float32)


def exact_term(tx, ty, mx, my, A, B, Cc, det, squared):
    dx = tx.astype(np.float64) - mx.astype(np.float64)
    dy = ty.astype(np.float64) - my.astype(np.float64)
    q = (Cc * dx * dx - 2.0 * B * dx * dy + A * dy * dy) / det
    q = np.maximum(q, 0.0)
    return q if squared else np.sqrt(q)


def _cases(rng, n):
    # covariance with eigenvalues spread over five decades and any orientation,
    # correlations up to 1 - 1e-9, plus axis-aligned and isotropic ones
    l1 = 10.0 ** rng.uniform(-5, 0, n)
    l2 = l1 * 10.0 ** -rng.uniform(0, 5, n)
    th = rng.uniform(0, np.pi, n)
    c, s = np.cos(th), np.sin(th)
    sxx = l1 * c * c + l2 * s * s
    syy = l1 * s * s + l2 * c * c
    sxy = (l1 - l2) * c * s
    k = n // 8
    sxy[:k] = 0.0
    syy[k:2 * k] = sxx[k:2 * k]
    sxy[k:2 * k] = 0.0
    ridge = 10.0 ** rng.uniform(-9, -3, n)
    # token positions on the unit square, centres near or at them
    tx = f32(rng.uniform(0, 1, n))
    ty = f32(rng.uniform(0, 1, n))
    off = 10.0 ** rng.uniform(-8, 0, n)
    ang = rng.uniform(0, 2 * np.pi, n)
    mx = f32(tx + off * np.cos(ang))
    my = f32(ty + off * np.sin(ang))
    mx[:k // 4] = tx[:k // 4]
    my[:k // 4] = ty[:k // 4]
    return sxx, sxy, syy, ridge, tx, ty, mx, my


def test_spatial_term_within_bound():
    rng = np.random.default_rng(2606)
    n = 400_000
    sxx, sxy, syy, ridge, tx, ty, mx, my = _cases(rng, n)
    for squared in (False, True):
        la, lb, lc, eps, (A, B, Cc, det) = meta(sxx, sxy, syy, ridge, squared)
        exact = exact_term(tx, ty, mx, my, A, B, Cc, det, squared)
        for shift in (-1, 0, 1):
            got = screen_term(tx, ty, mx, my, la, lb, lc, squared, np.full(n, shift))
            assert np.all(np.isfinite(got)) and np.all(got >= 0)
            err = np.abs(got.astype(np.float64) - exact)
            bound = eps.astype(np.float64) * exact + (0.0 if squared else 2e-15) + 1e-300
            worst = np.max(err / bound)
            assert worst <= 1.0, (squared, shift, worst)


def test_bound_is_not_vacuous():
    # the bound is tight to within a small factor on the worst cases: a plain
    # float32 evaluation of the expanded form on nearly singular covariances
    # breaks it, so the test above can fail
    rng = np.random.default_rng(7)
    n = 200_000
    sxx, sxy, syy, ridge, tx, ty, mx, my = _cases(rng, n)
    la, lb, lc, eps, (A, B, Cc, det) = meta(sxx, sxy, syy, ridge, False)
    exact = exact_term(tx, ty, mx, my, A, B, Cc, det, False)
    qa, qb, qc = f32(Cc / det), f32(-B / det), f32(A / det)
    dx, dy = f32(tx - mx), f32(ty - my)
    q = f32(f32(f32(qa * dx) * dx) + f32(f32(f32(2 * qb) * dx) * dy) + f32(f32(qc * dy) * dy))
    naive = np.sqrt(np.maximum(q, 0).astype(np.float64))
    bound = eps.astype(np.float64) * exact + 2e-15
    assert np.max(np.abs(naive - exact) / bound) > 1.0
    got = screen_term(tx, ty, mx, my, la, lb, lc, False, np.zeros(n))
    ratio = np.abs(got.astype(np.float64) - exact) / bound
    assert np.max(ratio) > 0.05
    # and the correlation term of eps is needed: without it the sum-of-squares
    # evaluation itself leaves the bound on nearly singular covariances
    no_rho = 0.5 * 16.0 * U * 1.02 + 2.5e-7
    assert np.max(np.abs(got.astype(np.float64) - exact) / (no_rho * exact + 2e-15)) > 1.0
