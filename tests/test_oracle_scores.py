"""Pins of the oracle's further detection scores (App. "Gumbel Watermark": the U-score
and its Chernoff bound; App. on Li et al.'s score h*_{gum,Delta}; App. on Lattimore's
truncated power-law score h_{PL,eps}) and of their p-values.

The paper fixes: the null law (pivots iid Unif(0,1)), the U-score's Chernoff bound
with E[e^{lam U}] = (e^lam - 1)/lam, Li et al.'s score as the log-likelihood ratio of
the least-favourable distribution P*_Delta (so e^h is a density under the null and
the watermarked pivot's density under P*), and the centring of Lattimore's score to
null mean 0.  The Li and PL p-values use the same Chernoff construction with their
own null MGFs (a reading: the paper reports ANLPPT for them without stating the
p-value); their validity P(p <= alpha) <= alpha is pinned by simulation.
"""
import math

import numpy as np
import pytest
from scipy import integrate, optimize, special, stats

import oracle

P_MIN = 1e-4
DELTAS = [0.1, 0.3, 0.5, 0.7, 0.9]
EPSES = [0.01, 0.05, 0.2, 1.0]


def _irwin_hall_log_sf(s, M):
    """ln P(U_1 + ... + U_M >= s) exactly (Irwin-Hall distribution, 50 digits)."""
    mpmath = pytest.importorskip("mpmath")
    mpmath.mp.dps = 50
    s = mpmath.mpf(s)
    cdf = sum((-1) ** k * mpmath.binomial(M, k) * (s - k) ** M for k in range(int(mpmath.floor(s)) + 1))
    return float(mpmath.log(1 - cdf / mpmath.factorial(M)))


@pytest.mark.parametrize("M", [1, 2, 5, 10, 20])
def test_u_score_chernoff_bounds_the_exact_tail(M):
    """The Chernoff value is an upper bound on the exact null tail of S_U, and within
    the usual O(log M) of it."""
    for f in (0.55, 0.6, 0.7, 0.8, 0.9):
        S = f * M
        exact = _irwin_hall_log_sf(S, M)
        ch = oracle.chernoff_log_p("U", S, M)
        assert ch >= exact - 1e-9, (M, S, ch, exact)
        assert ch - exact <= math.log(10.0 * math.sqrt(M)) + 2.0, (M, S, ch, exact)
    assert oracle.chernoff_log_p("U", 0.5 * M, M) == 0.0 and oracle.chernoff_log_p("U", 0.2 * M, M) == 0.0
    v = [oracle.chernoff_log_p("U", S, M) for S in np.linspace(0.5 * M, 0.95 * M, 12)]
    assert all(b < a for a, b in zip(v, v[1:]))


@pytest.mark.parametrize("delta", DELTAS)
def test_li_score_is_a_likelihood_ratio(delta):
    """e^{h*} integrates to 1 over the null pivot, h*(r) -> log(k + [q > 0]) as r -> 1,
    and the tilted null MGF at lambda = 1 is 1 (ln E[e^{h}] = 0)."""
    k, q = oracle.li_params(delta)
    assert k >= 1 and 0.0 <= q < 1.0 - delta + 1e-15
    dens = lambda u: math.exp(float(oracle.score_terms([-math.log(u)], delta, 0.1)["Li"][0]))
    total = integrate.quad(dens, 0.0, 1.0, epsabs=0.0, epsrel=1e-12, limit=400)[0]
    assert total == pytest.approx(1.0, abs=1e-9)
    near1 = float(oracle.score_terms([1e-12], delta, 0.1)["Li"][0])
    assert near1 == pytest.approx(math.log(k + (1 if q > 0 else 0)), abs=1e-9)
    assert abs(oracle._null_log_mgf("Li", 1.0, delta, 0.1)[0]) < 1e-9


def test_li_score_under_its_least_favourable_distribution():
    """Text watermarked from a row with probabilities P*_Delta: the pivot's density is
    e^{h*} (so E[e^{-h*(r)}] = 1) and its CDF is sum_v P*(v) r^{1/P*(v)} (H1 pivot law)."""
    delta = 0.3
    k, q = oracle.li_params(delta)
    probs = [1.0 - delta] * k + ([q] if q > 0 else [])
    x = np.log(np.array(probs + [1e-300], np.float64)).astype(np.float32)
    x[-1] = -np.inf
    key, n, m = 0x11A, 4000, 2
    toks = []
    for t in range(n):
        kappa = oracle.context_key(key, t, oracle.window_of(toks, [], m))
        toks.append(oracle.race(x, 1.0, kappa, 0, 1, oracle.LAYOUT_TREE)["token"])
    c = oracle.detect_clocks(key, m, 1, len(x), np.array(toks, np.int32), 0)
    r = np.exp(-c)
    h = oracle.score_terms(c, delta, 0.1)["Li"]
    w = np.exp(-h)
    assert abs(w.mean() - 1.0) < 5.0 * w.std() / math.sqrt(n)
    p = np.array(probs)
    cdf = lambda z: np.sum(p[None, :] * np.power(np.asarray(z)[:, None], 1.0 / p[None, :]), axis=1)
    assert stats.kstest(r, cdf).pvalue > P_MIN


@pytest.mark.parametrize("eps", EPSES)
def test_pl_score_centred_and_bounded(eps):
    c0 = 2.0 - math.sqrt(eps)
    h = lambda u: min(eps ** -0.5, (1.0 - u) ** -0.5) - c0
    pts = [1.0 - eps] if eps < 1.0 else None
    mean = integrate.quad(h, 0.0, 1.0, points=pts, epsabs=1e-14, epsrel=1e-12, limit=400)[0]
    assert abs(mean) < 1e-9
    us = np.linspace(0.0, 1.0 - 1e-15, 1001)
    vals = oracle.score_terms(-np.log1p(-us) if False else -np.log(np.maximum(us, 1e-300)), 0.3, eps)["PL"]
    assert np.all(vals <= eps ** -0.5 - c0 + 1e-12)
    # the oracle's per-token value equals the definition at the pivot r = e^{-c}
    for cc in (1e-6, 0.05, 0.7, 3.0, 30.0):
        r = math.exp(-cc)
        want = min(eps ** -0.5, (1.0 - r) ** -0.5) - c0
        assert float(oracle.score_terms([cc], 0.3, eps)["PL"][0]) == pytest.approx(want, rel=1e-9)


@pytest.mark.parametrize("kind,param", [("U", None), ("Li", 0.3), ("Li", 0.7), ("PL", 0.05), ("PL", 0.5)])
def test_chernoff_p_values_are_valid_under_the_null(kind, param):
    """P(p <= alpha) <= alpha under the null: the bound is decreasing in S, so this is
    the null tail at the score s_alpha where the bound reaches alpha, estimated from
    200000 simulated null sequences of M = 30 uniform pivots."""
    M = 30
    delta = param if kind == "Li" else 0.5
    eps = param if kind == "PL" else 0.01
    rng = np.random.default_rng(3)
    c = rng.exponential(size=(200000, M))        # null pivots r = e^{-c} are uniform
    Ssim = oracle.score_terms(c, delta, eps)[kind].sum(axis=1)
    for alpha in (0.05, 0.01):
        f = lambda S: oracle.chernoff_log_p(kind, S, M, delta, eps) - math.log(alpha)
        lo = M * oracle._null_log_mgf(kind, 0.0, delta, eps)[1] + 1e-9
        hi = lo + 1.0
        while f(hi) > 0:
            hi = lo + 2 * (hi - lo)
        s_alpha = optimize.brentq(f, lo, hi, xtol=1e-10)
        rate = float((Ssim >= s_alpha).mean())
        assert rate <= alpha + 3.0 * math.sqrt(alpha * (1 - alpha) / Ssim.size), (kind, param, alpha, rate)
        assert rate > 0.0  # the bound is not vacuous at this size


def test_score_terms_special_values():
    c = np.array([math.log(2.0)])                 # r = 1/2
    t = oracle.score_terms(c, 0.5, 0.25)
    assert float(t["A"][0]) == pytest.approx(math.log(2.0), rel=1e-14)
    assert float(t["U"][0]) == pytest.approx(0.5, rel=1e-14)
    # Delta = 0.5: k = 2, q = 0, h = log(2 r)
    assert float(t["Li"][0]) == pytest.approx(math.log(1.0), abs=1e-14)
    # eps = 1/4: min(2, (1/2)^{-1/2}) - 1.5 = sqrt(2) - 1.5
    assert float(t["PL"][0]) == pytest.approx(math.sqrt(2.0) - 1.5, rel=1e-14)
