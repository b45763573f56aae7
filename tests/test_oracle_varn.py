"""Pins of the oracle's VarN (App. H, Algorithm 1): alternating log-domain dual-scale
variance normalisation, rows = tokens, columns = channels.

Each test checks a property that Algorithm 1 fixes mathematically, with variances taken by
numpy (not by the oracle):
  * a column update leaves every unclamped column with variance exactly 1, a row update
    every unclamped row (closed form of the half steps);
  * K = 0 returns unit scales and B = T;
  * scale and permutation equivariance;
  * convergence of Imb(.) to 2 when nothing is clamped;
  * best-scale tracking: the returned balanced tile has the smallest imbalance of all
    iterations, the latest iteration winning ties.
"""
import numpy as np
import pytest

from tiles import tile

UNCLAMPED = dict(log_lo=-np.inf, log_hi=np.inf, c_min=0.0, c_max=np.inf)


def np_imb(X, floor=1e-8):
    vr = X.var(axis=1, ddof=1)
    vc = X.var(axis=0, ddof=1)
    return vr.max() / max(vr.min(), floor) + vc.max() / max(vc.min(), floor)


def cur(T, Lc, Lr):
    return T / np.exp(Lc)[None, :] / np.exp(Lr)[:, None]


@pytest.mark.parametrize("kind", ["tinyK", "tinyV", "stressK"])
def test_half_steps_unclamped(orc, kind):
    T = orc.hadamard128(tile(kind, 11))
    r = orc.varn(T, orc.Params(varn_iters=6, **UNCLAMPED))
    for k in range(1, 7):
        after_col = cur(T, r.Lc[k], r.Lr[k - 1])
        np.testing.assert_allclose(after_col.var(axis=0, ddof=1), 1.0, rtol=0, atol=1e-12)
        after_row = cur(T, r.Lc[k], r.Lr[k])
        np.testing.assert_allclose(after_row.var(axis=1, ddof=1), 1.0, rtol=0, atol=1e-12)


@pytest.mark.parametrize("kind", ["tinyK", "tinyV", "stressK"])
def test_half_steps_clamped(orc, kind):
    """With Algorithm 1's clamp [-0.3, 10], rows whose log-scale is strictly inside it are
    exactly unit-variance after the row step; the rest sit on a bound."""
    T = orc.hadamard128(tile(kind, 12))
    p = orc.Params()
    r = orc.varn(T, p)
    for k in range(1, p.varn_iters + 1):
        inside = (r.Lr[k] > p.log_lo + 1e-15) & (r.Lr[k] < p.log_hi - 1e-15)
        v = cur(T, r.Lc[k], r.Lr[k]).var(axis=1, ddof=1)
        np.testing.assert_allclose(v[inside], 1.0, rtol=0, atol=1e-12)
        on_bound = ~inside
        np.testing.assert_array_equal(np.isclose(r.Lr[k][on_bound], p.log_lo) | np.isclose(r.Lr[k][on_bound], p.log_hi),
                                      True)
        # a row pinned at the lower bound had variance below exp(2 * lo) relative to its scale
        assert np.all(r.Lc[k] >= p.log_lo) and np.all(r.Lc[k] <= p.log_hi)


def test_zero_iterations(orc):
    T = orc.hadamard128(tile("tinyK", 3))
    r = orc.varn(T, orc.Params(varn_iters=0))
    np.testing.assert_array_equal(r.Sc, 1.0)
    np.testing.assert_array_equal(r.Sr, 1.0)
    np.testing.assert_array_equal(r.B, T)
    assert r.best_iter == 0
    np.testing.assert_allclose(r.imb[0], np_imb(T), rtol=1e-12)


@pytest.mark.parametrize("alpha", [2.5, 40.0])
def test_scale_equivariance(orc, alpha):
    """The first column update absorbs a global factor: same B and S_r*, S_c* times alpha."""
    T = orc.hadamard128(tile("tinyV", 4))
    p = orc.Params(**UNCLAMPED)
    r1, r2 = orc.varn(T, p), orc.varn(alpha * T, p)
    assert r1.best_iter == r2.best_iter
    np.testing.assert_allclose(r2.Sc, alpha * r1.Sc, rtol=1e-12)
    np.testing.assert_allclose(r2.Sr, r1.Sr, rtol=1e-12)
    np.testing.assert_allclose(r2.B, r1.B, rtol=1e-11, atol=1e-12)


def test_scale_equivariance_with_clamp(orc):
    """Also under the printed clamp [-0.3, 10], for a tile on which the clamp never binds in
    any iteration (so that every update is the unclamped one)."""
    rng = np.random.default_rng(5)  # rows of nearly equal spread: no row scale nears e^-0.3
    T = 3.0 * orc.hadamard128(rng.standard_normal((128, 128)))
    p = orc.Params()
    r1 = orc.varn(T, p)
    alpha = 50.0
    r2 = orc.varn(alpha * T, p)
    for r in (r1, r2):  # precondition: no log-scale ever reached a bound
        assert np.all((r.Lc[1:] > p.log_lo) & (r.Lc[1:] < p.log_hi))
        assert np.all((r.Lr[1:] > p.log_lo) & (r.Lr[1:] < p.log_hi))
    np.testing.assert_allclose(r2.Sc, alpha * r1.Sc, rtol=1e-12)
    np.testing.assert_allclose(r2.Sr, r1.Sr, rtol=1e-12)
    np.testing.assert_allclose(r2.B, r1.B, rtol=1e-11, atol=1e-12)


def test_permutation_equivariance(orc):
    T = orc.hadamard128(tile("stressK", 6))
    rng = np.random.default_rng(7)
    pr, pc = rng.permutation(128), rng.permutation(128)
    p = orc.Params()
    r1 = orc.varn(T, p)
    r2 = orc.varn(T[pr][:, pc], p)
    np.testing.assert_allclose(r2.Sc, r1.Sc[pc], rtol=1e-12)
    np.testing.assert_allclose(r2.Sr, r1.Sr[pr], rtol=1e-12)
    np.testing.assert_allclose(r2.B, r1.B[pr][:, pc], rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("kind,iters,bound", [("tinyK", 8, 1e-6), ("tinyV", 8, 1e-6), ("stressK", 16, 1e-9)])
def test_converges_to_balanced(orc, kind, iters, bound):
    """Unclamped, the alternating normalisation drives Imb to its minimum 2 (all row
    variances equal and all column variances equal); row variances are exactly 1."""
    for seed in range(8):
        T = orc.hadamard128(tile(kind, 100 + seed))
        r = orc.varn(T, orc.Params(varn_iters=iters, **UNCLAMPED))
        assert r.imb[-1] - 2.0 <= bound
        C = cur(T, r.Lc[-1], r.Lr[-1])
        np.testing.assert_allclose(C.var(axis=1, ddof=1), 1.0, atol=1e-12)
        vc = C.var(axis=0, ddof=1)
        assert vc.max() / vc.min() - 1.0 <= bound
        # The common column variance is fixed by the means: the tile's sum of squares counted
        # by rows (each row: unit variance, plus its mean) equals the count by columns (each
        # column: variance kappa^2, plus its mean), so with R = C = 128
        #   kappa^2 = (R (C - 1) + C sum_r m_r^2 - R sum_c mu_c^2) / (C (R - 1)).
        # Mean-centring makes unit rows and unit columns jointly inconsistent unless the two
        # sums of squared means agree, which is why kappa is not 1 in general.
        R, Cn = C.shape
        kappa2 = (R * (Cn - 1) + Cn * (C.mean(axis=1) ** 2).sum() - R * (C.mean(axis=0) ** 2).sum()) / (Cn * (R - 1))
        np.testing.assert_allclose(vc, kappa2, rtol=2 * bound + 1e-12)
        if kind == "tinyV":  # value-like tiles: small means, kappa within 1 % of 1
            assert abs(np.sqrt(kappa2) - 1.0) < 1e-2


@pytest.mark.parametrize("kind", ["tinyK", "tinyV", "stressK"])
def test_best_tracking(orc, kind):
    T = orc.hadamard128(tile(kind, 21))
    p = orc.Params()
    r = orc.varn(T, p)
    # every recorded imbalance is Imb of the state it belongs to
    for k in range(p.varn_iters + 1):
        np.testing.assert_allclose(r.imb[k], np_imb(cur(T, r.Lc[k], r.Lr[k])), rtol=1e-10)
    # kept iteration: smallest imbalance, latest on ties
    m = r.imb.min()
    assert r.best_iter == max(k for k in range(p.varn_iters + 1) if r.imb[k] == m)
    np.testing.assert_allclose(r.Sc, np.exp(r.Lc[r.best_iter]), rtol=1e-15)
    np.testing.assert_allclose(r.Sr, np.exp(r.Lr[r.best_iter]), rtol=1e-15)
    np.testing.assert_allclose(np_imb(r.B), m, rtol=1e-10)
    np.testing.assert_allclose(r.B, T / r.Sc[None, :] / r.Sr[:, None], rtol=1e-15)


def test_best_tracking_keeps_earlier_iteration(orc):
    """When later iterations get worse, the earlier scales are kept (constructed case: a tile
    whose rows already have equal variance and whose columns do not converge under a tight
    clamp)."""
    T = orc.hadamard128(tile("stressK", 22))
    # a clamp that lets the first step move but then pins every scale: I stays constant,
    # so "<=" keeps the latest iteration
    p = orc.Params(log_lo=-0.05, log_hi=0.05)
    r = orc.varn(T, p)
    m = r.imb.min()
    assert r.best_iter == max(k for k in range(p.varn_iters + 1) if r.imb[k] == m)
    # and if the initial state is the best, nothing is kept but the unit scales
    p0 = orc.Params(varn_iters=3, log_lo=0.0, log_hi=0.0)
    r0 = orc.varn(T, p0)
    np.testing.assert_array_equal(r0.Sc, 1.0)
    np.testing.assert_array_equal(r0.Sr, 1.0)
    assert r0.best_iter == 3  # all iterations equal the initial state; the latest wins


def test_degenerate_tiles(orc):
    """Zero and constant tiles: every variance is below c_min and gets clamped; Imb uses the
    1e-8 floor; nothing becomes NaN."""
    p = orc.Params()
    for T in (np.zeros((128, 128)), np.full((128, 128), 3.25)):
        r = orc.varn(T, p)
        assert np.all(np.isfinite(r.Sc)) and np.all(np.isfinite(r.Sr)) and np.all(np.isfinite(r.B))
        np.testing.assert_allclose(r.Lc[1], p.log_lo)  # 0.5*log(1e-8) = -9.2 clamps to -0.3


def test_force_best_keeps_the_named_iteration(orc):
    """The test-only force_best knob returns the scales recorded for that iteration, and -1 is
    Algorithm 1's own selection."""
    from tiles import tile
    T = orc.hadamard128(tile("tinyK", 4))
    base = orc.varn(T, orc.Params())
    for k in (0, 3, 8):
        r = orc.varn(T, orc.Params(force_best=k))
        assert r.best_iter == k
        assert np.allclose(np.log(r.Sc), base.Lc[k], rtol=0, atol=1e-12)
        assert np.allclose(np.log(r.Sr), base.Lr[k], rtol=0, atol=1e-12)
