"""Pins of the oracle's ternarization variants (Sec. 3.1): the asymmetric
thresholds of Eq. (3)-(4), the Gaussian-optimal threshold, and the
Kolmogorov-Smirnov choice between the Gaussian and exponential references.

Each check ties the oracle to something other than itself: enumeration of
every ternary assignment, the Eq. (5) solution, a root of the defining
equation found by scipy, scipy's own K-S statistic, and large-sample limits.
"""
import itertools

import numpy as np
import pytest
from scipy import optimize, stats

import oracle


def brute_force_error(w):
    """min over T in {-1,0,1}^n of ||w - alpha_T T||^2 with the best alpha_T >= 0."""
    w = w.astype(np.float64)
    best = float(np.dot(w, w))
    for T in itertools.product((-1, 0, 1), repeat=w.size):
        T = np.array(T, np.float64)
        tt = float(np.dot(T, T))
        if tt == 0:
            continue
        a = max(0.0, float(np.dot(w, T)) / tt)
        best = min(best, float(np.sum((w - a * T) ** 2)))
    return best


def error_of(w, t, alpha):
    w = w.astype(np.float64)
    return float(np.sum((w - float(alpha) * t.astype(np.float64)) ** 2))


# ---------------------------------------------------------------------------
# Eq. (3)-(4): asymmetric thresholds
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(40))
def test_asym_matches_enumeration(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 8))
    w = rng.standard_normal(n).astype(np.float32)
    if seed % 5 == 0:
        w[rng.integers(0, n)] = 0.0                       # zeros are never kept
    if seed % 7 == 0 and n > 2:
        w[1] = -w[0]                                      # a magnitude tie across signs
    t, a, dp, dn = oracle.ternarize_group_asym(w)
    assert error_of(w, t, a) <= brute_force_error(w) * (1 + 1e-9) + 1e-12


@pytest.mark.parametrize("seed", range(30))
def test_asym_reaches_the_symmetric_optimum(seed):
    # the optimum over (Dp, Dn) is the optimum of Eq. (5): for a given kept
    # count the largest kept sum is the top magnitudes whatever their sign
    rng = np.random.default_rng(100 + seed)
    w = rng.laplace(0, 1, 64).astype(np.float32)
    t, a, dp, dn = oracle.ternarize_group_asym(w)
    ts, as_, _ = oracle.ternarize_group(w)
    assert np.array_equal(t, ts)
    assert abs(float(a) - float(as_)) <= np.spacing(np.float32(as_))


def test_asym_thresholds_bracket_the_kept_sets():
    rng = np.random.default_rng(7)
    w = (rng.standard_normal(64) + 0.4).astype(np.float32)   # skewed: different thresholds
    t, a, dp, dn = oracle.ternarize_group_asym(w)
    assert np.all(w[t == 1] > dp) and np.all(w[(t == 0) & (w > 0)] <= dp)
    assert np.all(-w[t == -1] > dn) and np.all(-w[(t == 0) & (w < 0)] <= dn)
    kept = np.abs(w[t != 0]).astype(np.float64)
    assert np.float32(kept.sum() / kept.size) == a


def test_asym_all_zero_and_one_sided():
    t, a, dp, dn = oracle.ternarize_group_asym(np.zeros(8, np.float32))
    assert not t.any() and a == 0 and dp == 0 and dn == 0
    t, a, dp, dn = oracle.ternarize_group_asym(np.array([3, 1, 2, 0], np.float32))
    # f(1) = 9, f(2) = 12.5, f(3) = 12: keep {3, 2}, Dp = 1, no negatives
    assert list(t) == [1, 0, 1, 0] and a == np.float32(2.5) and dp == 1 and dn == 0


def test_asym_tie_keeps_first_maximum():
    # f(1, 0) = 3^2/1 = 9 and f(1, 3) = (3+1+1+1)^2/4 = 9 tie exactly (every
    # other pair scores less); the first maximum in (a, then b) order wins
    t, a, dp, dn = oracle.ternarize_group_asym(np.array([3, -1, -1, -1], np.float32))
    assert list(t) == [1, 0, 0, 0] and a == 3 and dp == 0 and dn == 1


def test_asym_layer_grouping_matches_groups():
    rng = np.random.default_rng(3)
    w = rng.standard_normal((3, 8, 2, 2)).astype(np.float32)
    t, a, dp, dn = oracle.ternarize_asym(w, 4)
    for o in range(3):
        for r in range(2):
            for s in range(2):
                for cb in range(2):
                    g = ((r * 2 + s) * 8 + cb * 4) // 4
                    tg, ag, dpg, dng = oracle.ternarize_group_asym(w[o, cb * 4:(cb + 1) * 4, r, s])
                    k0 = (r * 2 + s) * 8 + cb * 4
                    assert np.array_equal(t[o, k0:k0 + 4], tg)
                    assert (a[o, g], dp[o, g], dn[o, g]) == (ag, dpg, dng)


# ---------------------------------------------------------------------------
# Gaussian-optimal threshold
# ---------------------------------------------------------------------------

def test_gauss_u_is_the_root_of_its_equation():
    u = optimize.brentq(lambda x: 2 * x * stats.norm.sf(x) - stats.norm.pdf(x), 0.1, 2.0,
                        xtol=1e-17, rtol=1e-15)
    assert abs(oracle.gauss_u() - u) <= 1e-15


def test_gauss_u_is_the_large_sample_optimum_of_eq5():
    # the exact Eq. (5) solver on one large Gaussian group: Delta / sigma -> u*
    rng = np.random.default_rng(11)
    w = rng.standard_normal(1_000_000).astype(np.float32)
    _, a, d = oracle.ternarize_group(w, oracle.EXACT)
    assert abs(float(d) - oracle.gauss_u()) < 4e-3
    # and the rule's alpha approaches the exact one
    _, ag, dg = oracle.ternarize_group(w, oracle.GAUSS)
    assert abs(float(dg) - oracle.gauss_u() * float(np.sqrt(np.mean(w.astype(np.float64) ** 2)))) < 1e-6
    assert abs(float(ag) - float(a)) < 4e-3


def test_gauss_rule_on_a_worked_group():
    w = np.array([2, -2, 2, -2, 0.5, -1.0, 1.3, 0.0], np.float32)
    rms = np.sqrt(np.sum(w.astype(np.float64) ** 2) / 8)
    t, a, d = oracle.ternarize_group(w, oracle.GAUSS)
    assert d == np.float32(oracle.gauss_u() * rms)
    keep = np.abs(w) > d
    assert np.array_equal(t, (np.sign(w) * keep).astype(np.int8))
    assert a == np.float32(np.abs(w[keep]).astype(np.float64).sum() / keep.sum())


# ---------------------------------------------------------------------------
# K-S distances and the per-layer choice
# ---------------------------------------------------------------------------

def _sample(w):
    w = np.ascontiguousarray(w, np.float32).ravel()
    step = -(-w.size // oracle.KS_SAMPLE)
    return np.abs(w[::step]).astype(np.float64)


@pytest.mark.parametrize("n,dist", [(1000, "normal"), (5000, "laplace"), (100_000, "normal"),
                                    (70_001, "laplace")])
def test_ks_distances_match_scipy(n, dist):
    rng = np.random.default_rng(n)
    w = (rng.standard_normal(n) if dist == "normal" else rng.laplace(0, 1, n)).astype(np.float32)
    dg, de = oracle.ks_distances(w)
    m = _sample(w)
    sig = np.sqrt(np.mean(m ** 2))
    mu = np.mean(m)
    assert abs(dg - stats.kstest(m, "halfnorm", args=(0, sig)).statistic) < 1e-12
    assert abs(de - stats.kstest(m, "expon", args=(0, mu)).statistic) < 1e-12


def test_ks_picks_the_generating_law():
    rng = np.random.default_rng(5)
    g = rng.standard_normal((64, 64, 3, 3)).astype(np.float32)
    e = rng.laplace(0, 1, (64, 64, 3, 3)).astype(np.float32)
    dg, de = oracle.ks_distances(g)
    assert dg < de
    dg, de = oracle.ks_distances(e)
    assert de < dg
    # the layer then takes that law's threshold rule in every group
    for w, rule in ((g, oracle.GAUSS), (e, oracle.EXP_LEMMA)):
        tk, ak, dk = oracle.ternarize(w, 4, oracle.KS)
        tr, ar, dr = oracle.ternarize(w, 4, rule)
        assert np.array_equal(tk, tr) and np.array_equal(ak, ar) and np.array_equal(dk, dr)


def test_ks_zero_layer():
    assert oracle.ks_distances(np.zeros(100, np.float32)) == (0.0, 0.0)
