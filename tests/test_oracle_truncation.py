"""Pins of the oracle's logit processing before the race (top-k, then top-p).

The paper's experiments race the processed distribution P_k (temperature, top-k =
50, top-p), Alg. "Batched-target direct-top-k MPFR speculative sampling" and its
exactness theorem: the output follows the autoregressive model with kernel P_k.
Checked: the kept set against a counting definition of the rank (token v is kept
by top-k iff fewer than k tokens beat it, a tie going to the lower index) and the
top-p cut against its mass condition; the race on a truncated row samples P_k; MPFR
samples are iid P_k; speculative output on P_k equals plain keyed decoding on P_k;
detection pivots of P_k-watermarked text follow the H1 pivot law of P_k.
"""
import math

import numpy as np
import pytest
from scipy import special, stats

import oracle

P_MIN = 1e-4


def _rank_kept(x, k):
    """Top-k by counting: v is kept iff #{u : x_u > x_v or (x_u == x_v and u < v)} < k."""
    V = x.size
    keep = np.zeros(V, bool)
    for v in range(V):
        if x[v] == -np.inf:
            continue
        beats = np.sum((x > x[v]) | ((x == x[v]) & (np.arange(V) < v)))
        keep[v] = beats < k
    return keep


def test_top_k_matches_counting_definition():
    rng = np.random.default_rng(1)
    for trial in range(300):
        V = int(rng.integers(1, 60))
        x = rng.choice([-2.0, -1.0, 0.0, 0.5, 1.0, 3.0, -np.inf], V).astype(np.float32)
        if trial % 3 == 0:
            x = rng.standard_normal(V).astype(np.float32)
        k = int(rng.integers(1, V + 3))
        assert np.array_equal(oracle.truncation_mask(x, 1.0, k), _rank_kept(x, k)), (x, k)
        assert oracle.truncation_mask(x, 1.0, k).sum() == min(k, int(np.sum(x != -np.inf)))
    x = rng.standard_normal(100).astype(np.float32)
    assert np.array_equal(oracle.truncation_mask(x, 0.7, 0), x != -np.inf)       # k = 0: nothing cut
    assert np.array_equal(oracle.truncate(x, 0.7, 100), x)                        # k >= V: nothing cut


def test_top_p_mass_condition():
    rng = np.random.default_rng(2)
    for trial in range(300):
        V = int(rng.integers(1, 80))
        x = (2.0 * rng.standard_normal(V)).astype(np.float32)
        if trial % 4 == 0:
            x[rng.integers(0, V, 3)] = x[0]          # ties
        T = float(rng.choice([0.5, 1.0, 1.7]))
        k = int(rng.integers(0, V + 1))
        top_p = float(rng.uniform(0.05, 0.999))
        keep = oracle.truncation_mask(x, T, k, top_p)
        base = oracle.truncation_mask(x, T, k)
        assert np.all(keep <= base)
        pk = special.softmax(np.where(base, x.astype(np.float64) / np.float64(np.float32(T)), -np.inf))
        mass = pk[keep].sum()
        assert mass >= top_p - 1e-12
        # the kept set is a prefix of the top-k order, and dropping its last token falls short
        kept_vals = np.sort(x[keep])
        if keep.sum() > 1:
            smallest = np.flatnonzero(keep)[np.lexsort((np.flatnonzero(keep), x[keep]))][0]
            assert mass - pk[smallest] < top_p + 1e-12
        assert np.all(x[base & ~keep] <= kept_vals[0])


@pytest.mark.parametrize("layout", [oracle.LAYOUT_TREE, oracle.LAYOUT_FLAT])
def test_race_on_truncated_row_samples_p_k(layout):
    rng = np.random.default_rng(3)
    x = (1.5 * rng.standard_normal(40)).astype(np.float32)
    xt = oracle.truncate(x, 0.8, 6, 0.9)
    pk = special.softmax(np.where(xt == -np.inf, -np.inf, xt.astype(np.float64) / np.float64(np.float32(0.8))))
    n = 12000
    ys = np.array([oracle.race(xt, 0.8, oracle.context_key(7, 100 + t, []), 0, 3, layout)["token"] for t in range(n)])
    kept = np.flatnonzero(pk > 0)
    assert set(np.unique(ys)) <= set(kept.tolist())
    assert stats.chisquare(np.bincount(ys, minlength=40)[kept], n * pk[kept]).pvalue > P_MIN
    # MPFR on the truncated row: pairs of samples iid P_k
    cells = np.zeros((kept.size, kept.size))
    pos = {v: i for i, v in enumerate(kept)}
    for t in range(6000):
        u = oracle.mpfr(xt, 0.8, oracle.context_key(9, t, []), 2, layout)["samples"]
        cells[pos[u[0]], pos[u[1]]] += 1
    assert stats.chisquare(cells.ravel(), 6000 * np.outer(pk[kept], pk[kept]).ravel()).pvalue > P_MIN


@pytest.mark.parametrize("mpfr", [False, True])
def test_speculative_output_on_p_k_equals_plain_chain(mpfr):
    V, K, gamma, m, N, top_k = 30, 3, 3, 2, 36, 5
    rng = np.random.default_rng(4)
    P_rows = oracle.truncate_block((1.5 * rng.standard_normal((N + gamma + 2, V))).astype(np.float32), 1.0, top_k,
                                   1.0)
    key, prompt = 0x2E2E, [3, 8]
    plain = list(prompt)
    while len(plain) < N:
        t = len(plain)
        kappa = oracle.context_key(key, t, oracle.window_of(plain, [], m))
        plain.append(oracle.race(P_rows[t], 1.0, kappa, 0, 1 if mpfr else K, oracle.LAYOUT_TREE)["token"])
    text = list(prompt)
    while len(text) < N:
        t0 = len(text)
        tl = np.stack([P_rows[t0 + s] for s in range(gamma + 1)])[None]
        dl = oracle.truncate_block((tl[:, None, :gamma] + rng.standard_normal((1, K, gamma, V))).astype(np.float32),
                                   1.0, top_k, 1.0)
        fn = oracle.verify_block_mpfr if mpfr else oracle.verify_block
        res = fn(key=key, K=K, gamma=gamma, m=m, T_target=1.0, T_draft=1.0, prefix=[text[-m:]], start_pos=[t0],
                 target_logits=tl, draft_logits=dl)
        text += res["out_tokens"][0]
    assert text[:N] == plain[:N]


def test_detection_pivot_law_under_p_k():
    x = np.linspace(2.0, -2.0, 20).astype(np.float32)
    xt = oracle.truncate(x, 1.0, 7)
    pk = special.softmax(np.where(xt == -np.inf, -np.inf, xt.astype(np.float64)))
    key, m, n = 0x3F3F, 2, 3000
    toks = []
    for t in range(n):
        kappa = oracle.context_key(key, t, oracle.window_of(toks, [], m))
        toks.append(oracle.race(xt, 1.0, kappa, 0, 1, oracle.LAYOUT_TREE)["token"])
    c = oracle.detect_clocks(key, m, 1, 20, np.array(toks, np.int32), 0)
    r = np.exp(-c)
    p = pk[pk > 0]
    cdf = lambda z: np.sum(p[None, :] * np.power(np.asarray(z)[:, None], 1.0 / p[None, :]), axis=1)
    assert stats.kstest(r, cdf).pvalue > P_MIN
