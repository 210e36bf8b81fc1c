"""Pins of the oracle's multi-sample PFR (MPFR, identical drafters) on the CPU.

What the paper fixes about MPFR and its speculative use:
* eq. MPFR / Thm. "Exactness of direct finite-support MPFR": the B samples are iid
  from P; B arrivals per token suffice (no token holds more than B of the B smallest
  scores);
* MPFR(P, Pi, 1) is the single exponential race of eq. EFR (slot 0);
* Thm. 4.1 (eq. PML_accept) and Thm. "PML_accept_exact": with Y = MPFR(P, Pi, 1) and
  the B drafts MPFR(Q, Pi, B) from the same process,
  P(Y in drafts) >= 1 - sum_i p_i (p_i/(p_i+q_i))^B and >= 1 - sum_i p_i (a_i/(1+a_i))^B;
  for B = 1 the second is the exact single-race value sum_i p_i / (1 + a_i);
* Alg. "Multi-Draft ... (Formal)": the context tree with multiplicities nu(c), the
  distinct drafts D(c), y(c) at every internal context and the walk -- the oracle's
  path representation must emit what a literal transcription emits;
* Thm. "Exactness of batched-target direct-top-k MPFR decoding": speculative output
  equals plain keyed autoregressive decoding.
"""
import itertools
import math

import numpy as np
import pytest
from scipy import special, stats

import oracle
import workloads

LAYOUTS = [oracle.LAYOUT_TREE, oracle.LAYOUT_FLAT]
P_MIN = 1e-4


def _kappa(t, salt=0x3A3A):
    return oracle.context_key(0xC0FFEE0000 + salt, t, [])


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_single_sample_is_the_race(layout):
    rng = np.random.default_rng(1)
    for t in range(200):
        V = int(rng.integers(1, 300))
        x = (1.5 * rng.standard_normal(V)).astype(np.float32)
        x[rng.random(V) < 0.1] = -np.inf
        r = oracle.race(x, 0.8, _kappa(t), 0, 1, layout)
        m = oracle.mpfr(x, 0.8, _kappa(t), 1, layout)
        assert m["samples"][0] == r["token"]
        if r["token"] >= 0:
            assert m["scores"][0] == pytest.approx(r["best"], abs=1e-12)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_brute_force_and_truncation(layout):
    """Sorted scores equal a brute-force sort of ln(cumulative clocks) - l/T over all
    (token, arrival) pairs, and computing 2B arrivals per token leaves the first B
    samples unchanged (the truncation of the finite-support algorithm is exact)."""
    rng = np.random.default_rng(2)
    for t in range(150):
        V = int(rng.integers(1, 9))
        nu = int(rng.integers(1, 6))
        x = rng.choice([-1.0, 0.0, 0.5, 2.0, -np.inf], V).astype(np.float32)
        T = float(rng.choice([0.5, 1.0, 2.0]))
        kappa = _kappa(1000 + t)
        res = oracle.mpfr(x, T, kappa, nu, layout, n_out=nu)
        G = np.cumsum(np.stack([oracle.clocks(kappa, j, V, layout) for j in range(2 * nu)]), axis=0)
        cand = sorted((math.log(G[j, v]) - float(x[v]) / float(np.float32(T)), v, j)
                      for v in range(V) for j in range(2 * nu) if x[v] != -np.inf)
        want = [c[1] for c in cand[:nu]] + [-1] * max(0, nu - len(cand))
        assert res["samples"] == want, (res, cand[:nu])
        longer = oracle.mpfr(x, T, kappa, 2 * nu, layout, n_out=2 * nu)
        assert longer["tokens"][:nu] == res["tokens"][:nu]


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_samples_are_iid_p(layout):
    """(U_1, U_2, U_3) ~ P x P x P on a 4-token vocabulary (chi-square over the 64
    cells), and each of the first two samples ~ P on a config-1 row."""
    x = np.array([0.9, 0.1, -0.4, 0.5], np.float32)
    p = special.softmax(x.astype(np.float64))
    n = 24000
    cells = np.zeros(64)
    for t in range(n):
        u = oracle.mpfr(x, 1.0, _kappa(t, 7), 3, layout)["samples"]
        cells[u[0] * 16 + u[1] * 4 + u[2]] += 1
    expected = n * np.einsum("i,j,k->ijk", p, p, p).ravel()
    assert expected.min() > 20
    assert stats.chisquare(cells, expected).pvalue > P_MIN
    xr, pr = workloads.zipf_probs(1024, 2.0, 1.1, 1.0, seed=4)
    order = np.argsort(-pr)
    bins, acc, cur = np.zeros(1024, int), 0.0, 0
    for v in order:
        bins[v] = cur
        acc += pr[v]
        if acc * 3000 >= 25:
            cur, acc = cur + 1, 0.0
    nb = bins.max() + 1
    first, second = [], []
    for t in range(3000):
        u = oracle.mpfr(xr, 1.0, _kappa(t, 9), 2, layout)["samples"]
        first.append(bins[u[0]])
        second.append(bins[u[1]])
    e = np.bincount(bins, weights=pr, minlength=nb) * 3000
    assert stats.chisquare(np.bincount(first, minlength=nb), e).pvalue > P_MIN
    assert stats.chisquare(np.bincount(second, minlength=nb), e).pvalue > P_MIN


def _alpha(p, q):
    return np.array([p[i] * np.sum(np.maximum(q / q[i] - p / p[i], 0.0)) for i in range(len(p))])


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("B", [1, 2, 4])
def test_mpfr_acceptance_bounds(layout, B):
    """Thm. 4.1 and the exact-alpha bound on P(Y in {X_1..X_B}), Y = MPFR(P, Pi, 1),
    X = MPFR(Q, Pi, B) from the same keyed process; equality for B = 1."""
    xp = np.array([1.0, 0.2, -0.4, 1.5, 0.0, -1.2, 0.7, 0.3], np.float32)
    xq = np.array([0.6, 0.9, -0.2, 1.0, 0.4, -0.5, 0.1, 0.8], np.float32)
    p = special.softmax(xp.astype(np.float64))
    q = special.softmax(xq.astype(np.float64))
    a = _alpha(p, q)
    thm41 = 1.0 - float(np.sum(p * (p / (p + q)) ** B))
    exact_alpha = 1.0 - float(np.sum(p * (a / (1 + a)) ** B))
    n = 20000
    hits = 0
    for t in range(n):
        kappa = _kappa(50000 + t, B)
        y = oracle.race(xp, 1.0, kappa, 0, 1, layout)["token"]
        xs = oracle.mpfr(xq, 1.0, kappa, B, layout)["samples"]
        hits += int(y in xs)
    rate = hits / n
    se = math.sqrt(max(rate * (1 - rate), 1e-4) / n)
    assert rate >= thm41 - 4.5 * se, (rate, thm41)
    assert rate >= exact_alpha - 4.5 * se, (rate, exact_alpha)
    if B == 1:  # the single race's acceptance is exactly sum p_i / (1 + alpha_i)
        assert abs(rate - float(np.sum(p / (1 + a)))) < 4.5 * se
    assert thm41 < 1.0 and exact_alpha < 1.0


def _formal_tree_block(key, K, gamma, m, prefix, t0, Q, P, layout):
    """Literal form of Alg. "Multi-Draft ... (Formal)" for one block, with a proposal
    row Q[s] and a target row P[s] per depth (the same at every context of a depth):
    contexts with multiplicities, D(c), y(c) at every context up to depth gamma, the
    walk and the bonus."""
    def Pi(c):
        return oracle.context_key(key, t0 + len(c), oracle.window_of(prefix, list(c), m))
    levels = [{(): K}]
    D = {}
    for s in range(gamma):
        nxt = {}
        for c, nu in levels[-1].items():
            xs = oracle.mpfr(Q[s], 1.0, Pi(c), nu, layout)["samples"]
            D[c] = set(xs)
            for u in D[c]:
                nxt[c + (u,)] = nxt.get(c + (u,), 0) + xs.count(u)
        levels.append(nxt)
    y = {c: oracle.race(P[len(c)], 1.0, Pi(c), 0, 1, layout)["token"] for lv in levels for c in lv}
    cstar, out = (), []
    for s in range(gamma):
        out.append(y[cstar])
        if y[cstar] not in D[cstar]:
            return out
        cstar = cstar + (y[cstar],)
    out.append(y[cstar])
    return out


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_block_equals_formal_algorithm(layout):
    rng = np.random.default_rng(3)
    for trial in range(60):
        V = int(rng.integers(2, 6))
        K = int(rng.integers(1, 5))
        gamma = int(rng.integers(1, 4))
        m = int(rng.integers(0, 3))
        prefix = [int(v) for v in rng.integers(0, V, m)]
        t0 = m
        key = 0xABC000 + trial
        Q = (1.0 * rng.standard_normal((gamma, V))).astype(np.float32)
        P = (Q[list(range(gamma)) + [gamma - 1]] + 0.5 * rng.standard_normal((gamma + 1, V))).astype(np.float32)
        want = _formal_tree_block(key, K, gamma, m, prefix, t0, Q, P, layout)
        dl = np.broadcast_to(Q[None, None], (1, K, gamma, V)).copy()
        res = oracle.verify_block_mpfr(key=key, K=K, gamma=gamma, m=m, T_target=1.0, T_draft=1.0, prefix=[prefix],
                                       start_pos=[t0], target_logits=P[None], draft_logits=dl, layout=layout)
        assert res["out_tokens"][0] == want, (trial, res["out_tokens"][0], want)


def test_mpfr_speculative_output_equals_plain_keyed_chain():
    """Several MPFR speculative blocks over a position-indexed toy LM emit exactly the
    tokens of plain keyed decoding with the slot-0 race (batched-target exactness)."""
    V, K, gamma, m, N = 25, 4, 3, 2, 40
    rng = np.random.default_rng(5)
    P_rows = (1.5 * rng.standard_normal((N + gamma + 2, V))).astype(np.float32)
    key = 0x1D1D1D
    prompt = [3, 8]
    plain = list(prompt)
    while len(plain) < N:
        t = len(plain)
        kappa = oracle.context_key(key, t, oracle.window_of(plain, [], m))
        plain.append(oracle.race(P_rows[t], 1.0, kappa, 0, 1, oracle.LAYOUT_TREE)["token"])
    text, blocks = list(prompt), 0
    while len(text) < N:
        t0 = len(text)
        tl = np.stack([P_rows[t0 + s] for s in range(gamma + 1)])[None]
        dl = np.broadcast_to((tl[:, :gamma] + 0.7 * rng.standard_normal((1, gamma, V)))[:, None],
                             (1, K, gamma, V)).astype(np.float32).copy()
        res = oracle.verify_block_mpfr(key=key, K=K, gamma=gamma, m=m, T_target=1.0, T_draft=1.0,
                                       prefix=[text[-m:]], start_pos=[t0], target_logits=tl, draft_logits=dl)
        text += res["out_tokens"][0]
        blocks += 1
    assert text[:N] == plain[:N]
    assert blocks < N - len(prompt)


def test_mpfr_draft_multiplicities():
    """Per depth, the K paths split into contexts whose sizes sum to K; every context's
    drafts at the next depth are nu(c) MPFR samples, so a context with nu(c) = 1
    drafts exactly the slot-0 race of its row."""
    w = workloads.custom(30, 4, 3, 3, m=2, tau=0.8, sigma=1.5, alpha=0.8)
    blk = workloads.make_block(w, 4)
    dl = workloads.as_f32_numpy(blk["draft_logits"])
    tl = workloads.as_f32_numpy(blk["target_logits"])
    pre, sp = blk["prefix_tokens"].numpy(), blk["start_pos"].numpy()
    res = oracle.verify_block_mpfr(key=w.key, K=w.K, gamma=w.gamma, m=w.m, T_target=1.0, T_draft=1.0,
                                   prefix=pre, start_pos=sp, target_logits=tl, draft_logits=dl)
    for b in range(w.B):
        d = res["draft_tokens"][b]
        for s in range(w.gamma):
            groups = oracle.context_groups([d[k, :s] for k in range(w.K)])
            assert sum(len(g) for g in groups) == w.K
            for g in groups:
                kappa = oracle.context_key(w.key, int(sp[b]) + s, oracle.window_of(list(pre[b]), d[g[0], :s], w.m))
                samples = oracle.mpfr(dl[b][g[0]][s], 1.0, kappa, len(g))["samples"]
                assert [int(d[k, s]) for k in g] == samples
                if len(g) == 1:
                    assert samples[0] == oracle.race(dl[b][g[0]][s], 1.0, kappa, 0, 1)["token"]
        tau = res["out_len"][b]
        assert list(res["out_tokens"][b]) == list(res["target_tokens"][b][:tau])
