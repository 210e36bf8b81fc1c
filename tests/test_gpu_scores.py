"""GPU parity of the further detection scores and their p-values.

psd_detect_scores (S_A, S_U, S_Li(Delta), S_PL(eps) from one pass over the text)
against sums of the oracle's per-token scores of its exact target clocks, within
1e-9 relative (+1e-12); psd_detect_scores_pvalue against the oracle's p-values:
ln p_A within the Gamma-tail tolerance of the p-value tests, the Chernoff bounds
(U, Li, PL) within 1e-7 relative + 1e-9 (the two sides share no code: adaptive
quadrature and Brent's method on the CPU, composite Gauss-Legendre and bisection on
the GPU); psd_detection_rate exactly.
"""
import math
import os
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads  # noqa: E402

DEV = "cuda"
LAYOUTS = [0, 1]
KINDS = ["A", "U", "Li", "PL"]
SCORE_PARAMS = [(0.3, 0.05), (0.5, 0.01), (0.9, 1.0)]


@pytest.fixture(scope="module")
def psd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21858_amd import psd as m
    return m


def _np(t):
    return t.detach().cpu().numpy()


def _texts(w, key, wrong, layout, n_pos=60):
    """Watermarked text (keyed target race at every position, made by the oracle), text
    made with another key, and uniform text."""
    rng = np.random.default_rng(layout)
    P = w.m + n_pos
    rows = workloads.target_rows_fp32(w, 6 * P, workloads._gen(7 + layout, "cpu"), "cpu").view(6, P, w.V)
    rows = rows.to(w.torch_dtype).float().numpy()
    toks = np.zeros((8, P), np.int32)
    toks[:, :w.m] = rng.integers(0, w.V, (8, w.m))
    for i in range(6):
        k = key if i < 3 else wrong
        for t in range(w.m, P):
            kappa = oracle.context_key(k, t, [int(x) for x in toks[i, t - w.m:t]])
            toks[i, t] = oracle.race(rows[i, t], w.T_target, kappa, 0, w.K, layout)["token"]
    toks[6:, w.m:] = rng.integers(0, w.V, (2, n_pos))
    toks[0, 9] = w.V + 5  # out of range: not scored
    return toks


def _check_logp(kind, got, S, M, delta, eps):
    if kind == "A":
        ref = oracle.gamma_tail_log_p(S, M)
        if not (M > 0 and S > 0 and math.isfinite(S)):
            assert got == ref or (math.isnan(got) and math.isnan(ref)), (kind, S, M, got, ref)
            return
        tol = 4e-15 * (S + M * abs(math.log(S)) + math.lgamma(M + 1.0)) + 1e-14 + 1e-11 * abs(ref)
    else:
        ref = oracle.chernoff_log_p(kind, S, M, delta, eps)
        if math.isnan(ref):
            assert math.isnan(got), (kind, S, M, got)
            return
        tol = 1e-7 * abs(ref) + 1e-9
    assert abs(got - ref) <= tol, (kind, S, M, delta, eps, got, ref)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("mode", [0, 1])
def test_detect_scores_parity(psd, layout, mode):
    w = workloads.custom(5000, 4, 4, 1, dtype="bf16", m=3, sigma=3.0, alpha=1.2)
    key, wrong = 0x1111222233334444, 0x5555666677778888
    K_eff = 1 if mode == 1 else w.K
    w_gen = workloads.custom(5000, K_eff, 4, 1, dtype="bf16", m=3, sigma=3.0, alpha=1.2)
    tk = _texts(w_gen, key, wrong, layout)
    n0 = np.full(tk.shape[0], w.m, np.int32)
    n0[4] = 100  # nothing scored
    p = psd.make_params(key, w.V, w.K, w.m, dtype=torch.bfloat16, clocks=layout, mode=mode)
    tkd, n0d = torch.from_numpy(tk).to(DEV), torch.from_numpy(n0).to(DEV)
    for delta, eps in SCORE_PARAMS:
        for budget in (tk.shape[1], w.m + 20):  # the whole text and a 20-token prefix of every row
            scores, count = psd.detect_scores(p, tkd, n0d, delta, eps, seq_len=budget)
            logp = psd.detect_scores_pvalue(scores, count, delta, eps)
            torch.cuda.synchronize()
            sc, ct, lp = _np(scores), _np(count), _np(logp)
            for i in range(tk.shape[0]):
                c = oracle.detect_clocks(key, w.m, K_eff, w.V, tk[i][:budget], int(n0[i]), layout)
                c = c[~np.isnan(c)]
                terms = oracle.score_terms(c, delta, eps)
                assert ct[i] == c.size
                for q, kind in enumerate(KINDS):
                    ref = float(terms[kind].sum())
                    assert abs(sc[i, q] - ref) <= 1e-9 * abs(ref) + 1e-12, (i, kind, sc[i, q], ref)
                    _check_logp(kind, float(lp[i, q]), float(sc[i, q]), int(ct[i]), delta, eps)
            if budget == tk.shape[1]:
                # the keyed texts stand out under every score; the others do not (alpha = 1e-3)
                assert np.all(lp[:3, 0] < math.log(1e-3)) and np.all(lp[3:, :] > math.log(1e-3))
                n_det = psd.detection_rate(logp[:, 0], 1e-3)
                torch.cuda.synchronize()
                assert int(n_det[0]) == int((lp[:, 0] <= math.log(1e-3)).sum()) == 3


def test_score_pvalue_grid(psd):
    """p-values of synthetic (S, M) across and beyond each score's range, and the
    degenerate inputs (M = 0, S at or below the null mean, NaN S, negative M)."""
    rng = np.random.default_rng(5)
    for delta, eps in SCORE_PARAMS:
        rows, ms = [], []
        for M in (1, 2, 7, 30, 512, 5000):
            for f in (-0.5, 0.0, 0.05, 0.2, 0.5):
                # S for each score: its null mean plus f times its range above the mean
                mean = [1.0, 0.5, oracle._null_log_mgf("Li", 0.0, delta, eps)[1], 0.0]
                top = [8.0, 1.0, math.log(oracle.li_params(delta)[0] + (1 if oracle.li_params(delta)[1] > 0 else 0)),
                       eps ** -0.5 - (2 - math.sqrt(eps))]
                rows.append([M * (mu + f * (t - mu)) for mu, t in zip(mean, top)])
                ms.append(M)
        rows += [[5.0, 3.0, 1.0, 1.0], [float("nan")] * 4, [2.0, 1.0, 0.5, 0.3]]
        ms += [0, 5, -1]
        S = torch.tensor(rows, dtype=torch.float64, device=DEV)
        M = torch.tensor(ms, dtype=torch.int32, device=DEV)
        lp = _np(psd.detect_scores_pvalue(S, M, delta, eps))
        torch.cuda.synchronize()
        for i in range(len(rows)):
            for q, kind in enumerate(KINDS):
                if kind == "A" and rows[i][q] == rows[i][q] and ms[i] > 0 and rows[i][q] > 20 * ms[i]:
                    continue
                _check_logp(kind, float(lp[i, q]), float(rows[i][q]), int(ms[i]), delta, eps)
        for q in range(4):
            for alpha in (0.01, 0.5):
                cnt = psd.detection_rate(torch.from_numpy(lp[:, q].copy()).to(DEV), alpha)
                torch.cuda.synchronize()
                assert int(cnt[0]) == int((lp[:, q] <= math.log(alpha)).sum())
