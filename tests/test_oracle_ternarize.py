"""Pins for the oracle's ternarization (Sec. 3, Eq. (1)-(5), Lemma 1).

Nothing here re-types the oracle's search: the optimum is checked against
exhaustive enumeration of all ternary codes, hand-worked examples, the
closed forms of Lemma 1 and of the Gaussian case, and structural identities
of the grouped problem (Eq. (2), the 2k+1 capacity bound).
"""
import itertools
import math
import os

import numpy as np
import pytest
from scipy import optimize, stats

import fgq_inputs as fi
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def err_of(w, t, alpha):
    w = np.asarray(w, np.float64)
    return float(np.sum((w - np.float64(alpha) * t.astype(np.float64)) ** 2))


def brute_force(w):
    """Minimum of ||w - alpha*T||^2 over all T in {-1,0,1}^n and alpha >= 0
    (Eq. (1)); for a fixed T the best alpha is max(0, <w,T>/<T,T>)."""
    w = np.asarray(w, np.float64)
    n = w.size
    T = np.array(list(itertools.product((-1, 0, 1), repeat=n)), np.float64)
    dots = T @ w
    nnz = np.abs(T).sum(1)
    alpha = np.where(nnz > 0, np.maximum(dots, 0) / np.maximum(nnz, 1), 0.0)
    err = np.sum(w * w) - 2 * alpha * dots + alpha * alpha * nnz
    i = int(np.argmin(err))
    order = np.sort(err)
    gap = order[1] - order[0] if order.size > 1 else np.inf
    return err[i], T[i], alpha[i], gap


def test_hand_worked_examples():
    path = os.path.join(GOLDEN, "eq5_hand_examples.txt")
    rows = [l for l in open(path) if l.strip() and not l.startswith("#")]
    assert len(rows) >= 10
    for line in rows:
        w, t, a, d, e = [p.strip() for p in line.split("|")]
        w = np.array(w.split(), np.float32)
        t_exp = np.array(t.split(), np.int8)
        t_got, a_got, d_got = oracle.ternarize_group(w)
        np.testing.assert_array_equal(t_got, t_exp, err_msg=line)
        assert a_got == np.float32(float(a)), line
        assert d_got == np.float32(float(d)), line
        assert math.isclose(err_of(w, t_got, a_got), float(e), rel_tol=1e-6, abs_tol=1e-9), line


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6, 7, 8])
def test_matches_exhaustive_enumeration(n):
    rs = np.random.default_rng(1000 + n)
    for trial in range(60):
        kind = trial % 4
        if kind == 0:
            w = rs.standard_normal(n)
        elif kind == 1:
            w = rs.laplace(0, 1, n)
        elif kind == 2:  # ties and zeros
            w = rs.integers(-3, 4, n).astype(np.float64)
        else:            # wide dynamic range
            w = rs.standard_normal(n) * np.exp(rs.uniform(-6, 6, n))
        w = w.astype(np.float32)
        t, a, d = oracle.ternarize_group(w)
        e_bf, t_bf, a_bf, gap = brute_force(w)
        e_or = err_of(w, t, a)
        assert e_or <= e_bf + 1e-6 * max(1.0, float(np.sum(w.astype(np.float64) ** 2))), (w, t, a)
        if gap > 1e-6 * max(1.0, float(np.sum(w.astype(np.float64) ** 2))):
            np.testing.assert_array_equal(t, t_bf.astype(np.int8), err_msg=str(w))
            assert math.isclose(a, a_bf, rel_tol=1e-6), (w, a, a_bf)
        # threshold rule: kept iff |w| > Delta (Sec. 3)
        kept = t != 0
        if kept.any() and not kept.all():
            assert np.all(np.abs(w[kept]) > d)
            assert np.all(np.abs(w[~kept]) <= d)
        assert np.all(t[kept] == np.sign(w[kept]))
        assert a >= 0


def test_g64_local_certificate_and_subvectors():
    """G=64 groups: the chosen prefix beats its neighbours; sub-vectors of
    up to 10 elements agree with enumeration."""
    W = fi.he_weights(8, 64, 3, 3, "cert")
    t, a, d = oracle.ternarize(W, 64)
    Wt = W.transpose(0, 2, 3, 1).reshape(8, -1)  # [O][R][S][C]
    for o in range(8):
        for g in range(t.shape[1] // 64):
            w = Wt[o, g * 64:(g + 1) * 64].astype(np.float64)
            m = np.sort(np.abs(w))[::-1]
            S = np.cumsum(m)
            f = S * S / np.arange(1, 65)
            J = int(np.count_nonzero(t[o, g * 64:(g + 1) * 64]))
            assert f[J - 1] >= f[J - 2] and (J == 64 or f[J - 1] >= f[J])
            assert math.isclose(a[o, g], S[J - 1] / J, rel_tol=1e-7)
    rs = np.random.default_rng(7)
    for _ in range(20):
        w = rs.standard_normal(10).astype(np.float32)
        tt, aa, _ = oracle.ternarize_group(w)
        e_bf, *_ = brute_force(w)
        assert math.isclose(err_of(w, tt, aa), e_bf, rel_tol=1e-6, abs_tol=1e-9)


def test_special_cases():
    # G = 1: every weight is kept exactly (zero ternary error)
    w = np.array([0.3, -1.7, 2.5e-3, -4.0], np.float32)
    for x in w:
        t, a, d = oracle.ternarize_group([x])
        assert a == abs(x) and t[0] == np.sign(x) and d == 0
    # one non-zero
    t, a, d = oracle.ternarize_group([0, 0, -0.125, 0])
    assert a == np.float32(0.125) and list(t) == [0, 0, -1, 0]
    # equal magnitudes: all kept
    t, a, d = oracle.ternarize_group([-0.5, 0.5, 0.5, -0.5])
    assert a == np.float32(0.5) and list(t) == [-1, 1, 1, -1] and d == 0
    # all zero (and negative zero)
    t, a, d = oracle.ternarize_group([0.0, -0.0, 0.0, 0.0])
    assert a == 0 and d == 0 and not t.any()
    # subnormal magnitudes are ordinary positive numbers
    tiny = np.float32(1e-42)
    t, a, d = oracle.ternarize_group([tiny, -tiny, 0, 0])
    assert a == tiny and list(t) == [1, -1, 0, 0]


def test_nonfinite_rejected():
    for bad in (np.nan, np.inf, -np.inf):
        with pytest.raises(oracle.OracleError) as e:
            oracle.ternarize_group([1.0, bad, 0.5, 2.0])
        assert e.value.code == 5
    W = np.ones((2, 4, 1, 1), np.float32)
    W[1, 2, 0, 0] = np.nan
    with pytest.raises(oracle.OracleError):
        oracle.ternarize(W, 4)


def test_layer_grouping_layout_and_decomposition_identity():
    """Eq. (2): the layer is k independent sub-problems over groups of G
    consecutive input channels at a fixed (o, r, s) (Sec. 3.2, Fig. 2), and
    ||W - sum_i alpha_i What_i||^2 = sum_i ||W_i - alpha_i What_i||^2."""
    O, C, R, S, G = 6, 16, 3, 3, 4
    W = fi.he_weights(O, C, R, S, "decomp")
    t, a, d = oracle.ternarize(W, G)
    K = C * R * S
    Wg = W.transpose(0, 2, 3, 1).reshape(O, K // G, G)  # groups along C at each tap
    total = 0.0
    for o in range(O):
        for g in range(K // G):
            tg, ag, dg = oracle.ternarize_group(Wg[o, g])
            np.testing.assert_array_equal(tg, t[o, g * G:(g + 1) * G])
            assert ag == a[o, g] and dg == d[o, g]
            total += err_of(Wg[o, g], tg, ag)
    # reconstruct in the original [O][C][R][S] layout
    rec = (t.reshape(O, K // G, G).astype(np.float64) * a[:, :, None].astype(np.float64))
    rec = rec.reshape(O, R, S, C).transpose(0, 3, 1, 2)
    whole = float(np.sum((W.astype(np.float64) - rec) ** 2))
    assert math.isclose(whole, total, rel_tol=1e-12)
    # 2k+1 distinct values for k groups (Sec. 3.1, model capacity)
    k = O * K // G
    assert np.unique(rec).size <= 2 * k + 1
    # finer groups never approximate worse (each G=4 group solves a
    # sub-problem of a G=16 group)
    t16, a16, _ = oracle.ternarize(W, 16)
    rec16 = (t16.reshape(O, K // 16, 16) * a16[:, :, None].astype(np.float64)).reshape(O, R, S, C)
    err16 = float(np.sum((W.transpose(0, 2, 3, 1).astype(np.float64) - rec16) ** 2))
    assert total <= err16 + 1e-9


def test_paper_weight_layout_groups():
    """Sec. 3.2 stores the weights as [K][C/N][R*S][N] so that each group of
    N is contiguous.  That tensor is a rearrangement of the weights, and
    solving every contiguous N-vector of it by brute force over all 3^N
    ternary assignments (Eq. (1)) reproduces the oracle's codes and scales
    for the group (o, tap, block), i.e. the oracle's groups are the paper's."""
    O, C, R, S, N = 3, 12, 2, 3, 4
    W = fi.he_weights(O, C, R, S, "paper-layout")
    Pw = oracle.paper_weight_layout(W, N)
    assert Pw.shape == (O, C // N, R * S, N)
    np.testing.assert_array_equal(np.sort(Pw.ravel()), np.sort(W.ravel()))
    t, a, _ = oracle.ternarize(W, N)
    K = C * R * S
    t4 = t.reshape(O, R * S, C // N, N)   # k = tap*C + c: [O][tap][block][N]
    a3 = a.reshape(O, R * S, C // N)
    for o in range(O):
        for cb in range(C // N):
            for tap in range(R * S):
                err, T, alpha, gap = brute_force(Pw[o, cb, tap])
                assert gap > 1e-9  # a unique optimum
                np.testing.assert_array_equal(t4[o, tap, cb], T.astype(np.int8))
                assert abs(float(a3[o, tap, cb]) - alpha) <= 1e-6 * max(alpha, 1e-30)
    assert t.shape == (O, K)


def test_lemma1_exponential_magnitudes():
    """Lemma 1 and its proof (Appendix): with |W| ~ Exp(lambda) the kept
    fraction is exp(-lambda*Delta) and sum_kept|W| = n(lambda*Delta+1)
    exp(-lambda*Delta)/lambda, so G(Delta) peaks at Delta* = 1/lambda, where
    alpha* = 2/lambda and the kept fraction is 1/e."""
    lam = 4.0
    rs = fi.rng("lemma1")
    n = 2_000_000
    w = (rs.exponential(1.0 / lam, n) * rs.choice([-1.0, 1.0], n)).astype(np.float32)
    t, a, d = oracle.ternarize_group(w, oracle.EXACT)
    assert abs(d * lam - 1.0) < 0.03
    assert abs(a * lam - 2.0) < 0.01
    assert abs(np.count_nonzero(t) / n - math.exp(-1.0)) < 0.01
    # the Lemma's closed-form threshold (method 1) lands on the same optimum
    tl, al, dl = oracle.ternarize_group(w, oracle.EXP_LEMMA)
    assert abs(dl * lam - 1.0) < 0.005 and abs(al * lam - 2.0) < 0.01
    e_exact, e_lemma = err_of(w, t, a), err_of(w, tl, al)
    assert e_exact <= e_lemma * (1 + 1e-9)
    assert e_lemma <= e_exact * 1.001


def test_gaussian_stationary_point():
    """For N(0,1) weights Eq. (5) maximises phi(D)^2 / Q(D) (the Gaussian
    counterpart of the Lemma's integrals); solved numerically here, the
    optimum is D* ~ 0.612 with alpha* = phi(D*)/Q(D*) ~ 1.224 = 2 D*."""
    res = optimize.minimize_scalar(lambda x: -stats.norm.pdf(x) ** 2 / stats.norm.sf(x),
                                   bounds=(0.01, 3.0), method="bounded",
                                   options={"xatol": 1e-10})
    d_star = res.x
    a_star = stats.norm.pdf(d_star) / stats.norm.sf(d_star)
    assert abs(a_star - 2 * d_star) < 1e-6  # stationarity: Delta* = alpha*/2
    w = fi.rng("gauss-stationary").standard_normal(2_000_000).astype(np.float32)
    t, a, d = oracle.ternarize_group(w)
    assert abs(d - d_star) < 0.03
    assert abs(a - a_star) < 0.01


def test_lemma_method_special_cases():
    t, a, d = oracle.ternarize_group([1, 1, 1, 1], oracle.EXP_LEMMA)
    assert d == 1 and a == 0 and not t.any()  # nothing strictly above the mean
    t, a, d = oracle.ternarize_group([3, -1, 0, 0], oracle.EXP_LEMMA)
    assert d == 1 and a == 3 and list(t) == [1, 0, 0, 0]
