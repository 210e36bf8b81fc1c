"""Law of the TREE clock layout at production vocabulary sizes (oracle pins, CPU).

The tree layout builds each slot's clocks top-down over a fixed token hierarchy
(8-token chunks, then 16-ary nodes of 128, 2048 and 32768 tokens, root = all V).
Whatever the hierarchy, the construction must give iid Exp(1) clocks per
(slot, token): that is what the race needs to be the exponential race of eq. EFR
(Thm. "PFR reduces to EFR": argmin_v E_v / p_v ~ p) and what the detector's null
law assumes (App. "Gumbel Watermark").  The checks below use only consequences of
"iid Exp(1)" that a wrong node size, a wrong level shift, a wrong position draw
or a reused draw would break:

* pooled and per-position Kolmogorov-Smirnov tests against Exp(1), with positions
  inside the truncated last node of every level;
* n * (minimum of a node of n tokens) ~ Exp(1) for every level-3 and level-4 node,
  separately for the truncated last nodes (a node given the wrong size fails);
* V * (row minimum) ~ Exp(1); the argmin position uniform over the vocabulary,
  and its node proportional to the node's size;
* Renyi spacings at the top of the sorted row: (V - i) * (E_(i+1) - E_(i)) are iid
  Exp(1) (memorylessness across nodes: the smallest clocks of a row sit in
  different nodes);
* no correlation between neighbouring node minima or between slots;
* the target race on a row whose mass spans every level-4 node, including the
  truncated one, draws its token from p (chi-square per level-3 node), with the
  winning slot uniform and independent of the token (augmented race,
  Prop. "heterogeneous PML bound").

At V = 40000, 70001 and 128256 levels 3 and 4 have several children and truncated
last nodes (70001 truncates every level, down to a 1-token chunk); 2^19 is the
largest vocabulary, every node full.
"""
import math

import numpy as np
import pytest
from scipy import special, stats

import oracle

P_MIN = 1e-4  # deterministic seeds: a correct oracle passes with margin, a wrong one fails by orders
SHIFT = {1: 3, 2: 7, 3: 11, 4: 15}


def node_sizes(V, level):
    n = -(-V // (1 << SHIFT[level]))
    sizes = np.full(n, 1 << SHIFT[level], dtype=np.int64)
    sizes[-1] = V - (n - 1) * (1 << SHIFT[level])
    return sizes


def node_minima(E, level):
    sh = SHIFT[level]
    n = -(-E.size // (1 << sh))
    pad = np.full(n << sh, np.inf)
    pad[: E.size] = E
    return pad.reshape(n, 1 << sh).min(axis=1)


def _collect(V, n_keys, slots, layout, seed, n_sub=150, n_spacings=40):
    """Statistics of the full clock rows of n_keys random keys and the given slots."""
    rng = np.random.default_rng(seed)
    n3, n4 = node_sizes(V, 3), node_sizes(V, 4)
    last3 = V - int(n3[-1])
    last4 = V - int(n4[-1])
    fixed = sorted({0, 1, 7, 8, 127, 128, 2047, 2048, min(V - 1, 32767), min(V - 1, 32768), last4,
                    last4 + int(n4[-1]) // 2, last3, last3 + int(n3[-1]) // 2, V - 9, V - 8, V - 2, V - 1})
    fixed = [p for p in fixed if 0 <= p < V]
    out = {"fixed_pos": fixed, "fixed": [], "sub": [], "min": [], "argmin": [], "m3": [], "m4": [],
           "spacings": [], "slot_pairs": [], "lag": {1: [], 4: [], 8: [], 128: [], 2048: []}, "dups": []}
    for _ in range(n_keys):
        kappa = tuple(int(x) for x in rng.integers(0, 2**32, 2, dtype=np.uint64))
        rows = []
        for j in slots:
            E = oracle.clocks(kappa, j, V, layout)
            rows.append(E)
            out["fixed"].append(E[fixed])
            out["sub"].append(E[rng.integers(0, V, n_sub)])
            out["min"].append(E.min())
            out["argmin"].append(int(E.argmin()))
            out["m3"].append(node_minima(E, 3))
            out["m4"].append(node_minima(E, 4))
            for lag in out["lag"]:
                out["lag"][lag].append(np.corrcoef(E[:-lag], E[lag:])[0, 1])
            out["dups"].append(E.size - np.unique(E).size)
            top = np.sort(np.partition(E, n_spacings)[: n_spacings + 1])
            out["spacings"].append((V - np.arange(1, n_spacings + 1)) * np.diff(top))
        if len(rows) > 1:
            out["slot_pairs"].append((node_minima(rows[0], 3), node_minima(rows[1], 3)))
    for k in ("fixed", "sub", "m3", "m4", "spacings"):
        out[k] = np.array(out[k])
    out["min"] = np.array(out["min"])
    out["argmin"] = np.array(out["argmin"])
    return out


CASES = [(40000, 300), (70001, 300), (128256, 200)]


@pytest.fixture(scope="module", params=CASES, ids=[f"V{v}" for v, _ in CASES])
def tree_stats(request):
    V, n_keys = request.param
    return V, _collect(V, n_keys, (0, 3), oracle.LAYOUT_TREE, seed=V)


def test_tree_clocks_exponential_pooled_and_per_position(tree_stats):
    V, st = tree_stats
    assert np.all(st["sub"] > 0) and np.all(np.isfinite(st["sub"]))
    assert stats.kstest(st["sub"].ravel(), "expon").pvalue > P_MIN
    for i, pos in enumerate(st["fixed_pos"]):
        assert stats.kstest(st["fixed"][:, i], "expon").pvalue > P_MIN, (V, pos)


def test_tree_node_minima(tree_stats):
    """n * min over a node of n tokens ~ Exp(1): every level-3 and level-4 node,
    the truncated last ones on their own."""
    V, st = tree_stats
    for level, key in ((3, "m3"), (4, "m4")):
        sizes = node_sizes(V, level)
        scaled = st[key] * sizes[None, :]
        assert stats.kstest(scaled.ravel(), "expon").pvalue > P_MIN, (V, level)
        assert stats.kstest(scaled[:, -1], "expon").pvalue > P_MIN, (V, level, "last", int(sizes[-1]))
        if level == 4:
            for i in range(scaled.shape[1]):
                assert stats.kstest(scaled[:, i], "expon").pvalue > P_MIN, (V, level, i)
        # pooled mean of n * min is 1 per node: a node whose size were wrong by a
        # factor f would be off by f over all keys
        mean_last = scaled[:, -1].mean()
        assert abs(mean_last - 1.0) < 5.0 / math.sqrt(scaled.shape[0]), (V, level, mean_last)


def test_tree_row_minimum_and_argmin(tree_stats):
    V, st = tree_stats
    n = st["min"].size
    assert stats.kstest(V * st["min"], "expon").pvalue > P_MIN
    assert stats.kstest((st["argmin"] + 0.5) / V, "uniform").pvalue > P_MIN
    # the argmin falls into a level-4 node with probability size / V; the
    # truncated last node's share is checked on its own (binomial)
    sizes4 = node_sizes(V, 4)
    counts = np.bincount(st["argmin"] >> SHIFT[4], minlength=sizes4.size)
    assert stats.chisquare(counts, n * sizes4 / V).pvalue > P_MIN
    assert stats.binomtest(int(counts[-1]), n, float(sizes4[-1]) / V).pvalue > P_MIN


def test_tree_clocks_uncorrelated_and_distinct(tree_stats):
    """Clocks at lags 1, 4, 8, 128 and 2048 (inside a chunk, across chunk halves,
    groups and level-3 nodes) are uncorrelated, and a row holds no more equal
    clocks than 2^23-level uniforms give by chance (about V^2 / 2^24 pairs): a
    Philox word shared by two tokens would make half the row pairwise equal."""
    V, st = tree_stats
    for lag, r in st["lag"].items():
        r = np.array(r)
        # each row's correlation has standard error ~ 1/sqrt(V); their mean ~ 1/sqrt(V * rows)
        assert abs(r.mean()) < 5.0 / math.sqrt(V * r.size), (V, lag, r.mean())
        assert np.all(np.abs(r) < 6.0 / math.sqrt(V)), (V, lag, np.abs(r).max())
    expected = V * (V - 1) / 2 / 2.0**23 * 1.05  # exponential clocks: slightly denser near 0
    dups = np.array(st["dups"])
    assert dups.mean() < expected + 6 * math.sqrt(expected / dups.size) + 1, (V, dups.mean(), expected)


def test_tree_minimum_value_independent_of_position(tree_stats):
    """The row minimum's value and its position are independent (one Philox word
    gives the value, two others the position)."""
    V, st = tree_stats
    n = st["min"].size
    r = np.corrcoef(V * st["min"], (st["argmin"] + 0.5) / V)[0, 1]
    assert abs(r) < 4.5 / math.sqrt(n), (V, r)
    lo = st["argmin"] < V // 2
    assert stats.ks_2samp(V * st["min"][lo], V * st["min"][~lo]).pvalue > P_MIN


def test_tree_top_spacings_are_exponential(tree_stats):
    """Renyi representation of iid Exp(1): the normalised spacings of the sorted row
    are iid Exp(1).  At the top of the row they compare clocks from different
    nodes and levels, which a construction that got a node's offset wrong fails."""
    V, st = tree_stats
    sp = st["spacings"]
    assert stats.kstest(sp.ravel(), "expon").pvalue > P_MIN
    for i in (0, 1, 2, 5, 20, sp.shape[1] - 1):
        assert stats.kstest(sp[:, i], "expon").pvalue > P_MIN, (V, i)


def test_tree_node_minima_uncorrelated(tree_stats):
    V, st = tree_stats
    m3 = st["m3"] * node_sizes(V, 3)[None, :]
    a, b = m3[:, :-1].ravel(), m3[:, 1:].ravel()
    assert abs(np.corrcoef(a, b)[0, 1]) < 5.0 / math.sqrt(a.size)
    n3 = node_sizes(V, 3)[None, :]
    s0 = (np.array([p[0] for p in st["slot_pairs"]]) * n3).ravel()
    s1 = (np.array([p[1] for p in st["slot_pairs"]]) * n3).ravel()
    assert abs(np.corrcoef(s0, s1)[0, 1]) < 5.0 / math.sqrt(s0.size)


def test_tree_maximum_vocabulary_law():
    """V = 2^19: sixteen full level-4 nodes under the root."""
    V = 1 << 19
    st = _collect(V, 60, (1,), oracle.LAYOUT_TREE, seed=19, n_sub=400)
    assert stats.kstest(st["sub"].ravel(), "expon").pvalue > P_MIN
    assert stats.kstest(V * st["min"], "expon").pvalue > P_MIN
    scaled4 = st["m4"] * node_sizes(V, 4)[None, :]
    assert stats.kstest(scaled4.ravel(), "expon").pvalue > P_MIN
    scaled3 = st["m3"] * node_sizes(V, 3)[None, :]
    assert stats.kstest(scaled3.ravel(), "expon").pvalue > P_MIN
    assert stats.kstest(st["spacings"].ravel(), "expon").pvalue > P_MIN


def test_flat_clocks_large_vocabulary_law():
    """The flat layout at a large, ragged vocabulary (same statistics)."""
    V = 70001
    st = _collect(V, 120, (0, 3), oracle.LAYOUT_FLAT, seed=5)
    assert stats.kstest(st["sub"].ravel(), "expon").pvalue > P_MIN
    for i, pos in enumerate(st["fixed_pos"]):
        assert stats.kstest(st["fixed"][:, i], "expon").pvalue > P_MIN, pos
    assert stats.kstest(V * st["min"], "expon").pvalue > P_MIN
    assert stats.kstest(st["spacings"].ravel(), "expon").pvalue > P_MIN


@pytest.mark.parametrize("layout", [oracle.LAYOUT_TREE, oracle.LAYOUT_FLAT])
def test_target_marginal_spanning_level4_nodes(layout):
    """The target race over K = 2 slots at V = 70001 on a row whose probability mass
    is spread over all three level-4 nodes (the last one truncated to 4465 tokens)
    and all 35 level-3 nodes: the token follows p (chi-square over the level-3
    nodes, the truncated last one included) and the winning slot is uniform and
    independent of the token's node."""
    V, K, T, n = 70001, 2, 1.0, 1200
    rng = np.random.default_rng(70001)
    x = (1.2 * rng.standard_normal(V)).astype(np.float32)
    x[V - 4465:] += np.float32(1.5)       # extra mass in the truncated level-4 node
    x[V - 369:] += np.float32(1.0)        # and in the truncated last level-3 node
    p = special.softmax(x.astype(np.float64) / T)
    p3 = np.bincount(np.arange(V) >> SHIFT[3], weights=p)
    ys, js = [], []
    for t in range(n):
        kappa = oracle.context_key(0x7E57, 10**6 + t, [])
        r = oracle.race(x, T, kappa, 0, K, layout)
        ys.append(r["token"])
        js.append(r["slot"])
    ys, js = np.array(ys), np.array(js)
    obs = np.bincount(ys >> SHIFT[3], minlength=p3.size)
    assert stats.chisquare(obs, n * p3).pvalue > P_MIN
    assert p3[-1] * n > 5
    assert stats.chisquare(np.bincount(js, minlength=K)).pvalue > P_MIN
    node4 = ys >> SHIFT[4]
    table = np.zeros((3, K))
    np.add.at(table, (node4, js), 1)
    assert stats.chi2_contingency(table).pvalue > P_MIN
