"""GPU checks of the multi-block generation loop (psd_toy_logits, psd_advance,
psd_generate) against host definitions and the CPU oracle.

* toy model rows: every element of psd_toy_logits equals workloads.ToyModel (the
  same definition written in numpy), bit for bit;
* psd_advance equals a host transcription of its contract (commit, -1 ends a
  sequence, finished sequences repeat their last block);
* psd_generate's text is plain keyed decoding with the toy target rows: at every
  position t, the token equals the oracle's race of row (b, t) in the context of
  the text before it (distinct drafters: all K slots; identical drafters: slot 0;
  near-ties either way), on both clock layouts, with and without top-k; it equals a
  host loop of the same calls, its graph replay equals its eager run, and changing
  the drafters changes the block count but not one token (App. C);
* the stress workload (V=256000, K=16, gamma=4, 256 x 512 positions, half with a
  wrong key) generated on the device, then detected.
"""
import concurrent.futures
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
WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))
SCORE_TOL = 1e-9


@pytest.fixture(scope="module")
def psd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21858_amd import psd as m
    return m


def _np(t):
    return t.detach().cpu().numpy()


def _lm(psd, tm):
    return psd.make_toy_lm(tm.seed, tm.draft_seed, tm.sigma, tm.alpha, tm.tau, tm.tau_split)


def _prompts(B, m, V, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randint(0, V, (B, m), generator=g, dtype=torch.int64).to(torch.int32)


def plain_chain_check(tm, key, K, m, V, T, layout, text, picks, mpfr, bf16=True, top_k=0, top_p=1.0):
    """Every picked (b, t): the text's token is the oracle's race of the toy target row
    in the text's own context (near-ties either way).  Returns (exact, near) counts."""
    nsl = 1 if mpfr else K

    def one(bt):
        b, t = bt
        row = tm.target_row(b, t, V, bf16)
        if top_k:
            row = oracle.truncate(row, T, top_k, top_p)
        kappa = oracle.context_key(key, t, [int(x) for x in text[b, t - m:t]])
        r = oracle.race(row, T, kappa, 0, nsl, layout)
        got = int(text[b, t])
        if got == r["token"]:
            return "exact"
        if got >= 0 and r["token"] >= 0 and oracle.token_score(row, T, kappa, 0, nsl, got, layout) - r["best"] \
                < oracle.NEAR_TIE:
            return "near"
        return ("mismatch", b, t, got, r["token"], r["best"], r["second"])

    with concurrent.futures.ThreadPoolExecutor(WORKERS) as ex:
        res = list(ex.map(one, picks))
    bad = [r for r in res if isinstance(r, tuple)]
    assert not bad, bad[:3]
    return res.count("exact"), res.count("near")


def host_loop(psd, params, lm, prompts, n_pos, G):
    """The same blocks driven from Python with a synchronisation per block."""
    B, m = prompts.shape
    text = torch.full((B, m + n_pos), -1, dtype=torch.int32, device=DEV)
    text[:, :m] = prompts.to(DEV)
    length = torch.empty(B, dtype=torch.int64, device=DEV)
    start = torch.empty(B, dtype=torch.int64, device=DEV)
    prefix = torch.empty((B, m), dtype=torch.int32, device=DEV)
    act = torch.empty(1, dtype=torch.int32, device=DEV)
    psd.advance(params, G, m + n_pos, text, length, prefix, start, act)
    ws = psd.new_workspace(params, B, G, DEV)
    blocks = 0
    while True:
        tl, dl = psd.toy_logits(params, lm, G, start)
        out = psd.verify(params, ws, prefix, start, tl, dl)
        psd.advance(params, G, m + n_pos, text, length, prefix, start, act, out["out_tokens"], out["out_len"])
        blocks += 1
        torch.cuda.synchronize()
        if int(act[0]) == 0:
            break
        assert blocks <= n_pos
    assert psd.workspace_errors(ws) == 0
    return text, blocks


# ---------------------------------------------------------------- toy rows, advance

@pytest.mark.parametrize("V,K,G,B,dtype", [(1, 2, 2, 2, "bf16"), (7, 3, 2, 3, "fp32"), (1000, 4, 3, 4, "bf16"),
                                           (4099, 5, 1, 2, "fp32"), (128256, 4, 4, 3, "bf16"),
                                           (151936, 8, 2, 2, "fp32")])
def test_toy_logits_bit_exact(psd, V, K, G, B, dtype):
    print(f"[toy] V={V} K={K} G={G} B={B} {dtype}", flush=True)
    tm = workloads.ToyModel(seed=0xABCDEF + V, draft_seed=0x123457 * K, sigma=3.0, alpha=1.2, tau=(0.3, 1.5),
                            tau_split=B // 2)
    bf16 = dtype == "bf16"
    params = psd.make_params(1, V, K, 4, dtype=torch.bfloat16 if bf16 else torch.float32)
    start = torch.tensor([5 + 1000 * b + (b * b) % 7 for b in range(B)], dtype=torch.int64)
    start[-1] = (1 << 33) + 3  # positions are taken mod 2^32 in the row words
    tl, dl = psd.toy_logits(params, _lm(psd, tm), G, start.to(DEV))
    torch.cuda.synchronize()
    tl, dl = _np(tl.float()), _np(dl.float())
    for b in range(B):
        for s in range(G + 1):
            t = int(start[b]) + s
            ref = tm.target_row(b, t, V, bf16)
            assert np.array_equal(tl[b, s].view(np.uint32), ref.view(np.uint32)), (b, s)
            if s < G:
                for k in range(K):
                    ref = tm.draft_row(b, k, t, V, bf16)
                    assert np.array_equal(dl[b, k, s].view(np.uint32), ref.view(np.uint32)), (b, k, s)


def _advance_ref(text, length, out_tokens, out_len, m, max_len, G):
    text, length = text.copy(), length.copy()
    B = text.shape[0]
    for b in range(B):
        L = int(length[b])
        if out_len is not None and L < max_len:
            for i in range(int(out_len[b])):
                if L >= max_len:
                    break
                y = int(out_tokens[b][i])
                if y < 0:
                    text[b, L:max_len] = -1
                    L = max_len
                    break
                text[b, L] = y
                L += 1
        elif out_len is None:
            L = m
        length[b] = L
    start = np.minimum(length, max_len - 1)
    prefix = np.stack([text[b, start[b] - m:start[b]] for b in range(B)]) if m else np.zeros((B, 0), np.int32)
    return text, length, start, prefix, int((length < max_len).sum())


def test_advance_matches_contract(psd):
    rng = np.random.default_rng(3)
    B, G, m, max_len, stride = 37, 4, 3, 20, 26
    params = psd.make_params(1, 1000, 2, m)
    text = np.full((B, stride), -7, np.int32)
    text[:, :m] = rng.integers(0, 1000, (B, m))
    t_d = torch.from_numpy(text).to(DEV)
    length = torch.empty(B, dtype=torch.int64, device=DEV)
    start = torch.empty(B, dtype=torch.int64, device=DEV)
    prefix = torch.empty((B, m), dtype=torch.int32, device=DEV)
    act = torch.empty(1, dtype=torch.int32, device=DEV)
    psd.advance(params, G, max_len, t_d, length, prefix, start, act)
    ref = _advance_ref(text, np.zeros(B, np.int64), None, None, m, max_len, G)
    for step in range(12):
        torch.cuda.synchronize()
        for got, want in zip((t_d, length, start, prefix), ref[:4]):
            assert np.array_equal(_np(got), want), step
        assert int(act[0]) == ref[4]
        ot = rng.integers(0, 1000, (B, G + 1)).astype(np.int32)
        ol = rng.integers(1, G + 2, B).astype(np.int32)
        ot[rng.random((B, G + 1)) < 0.03] = -1   # an empty row ends its sequence
        psd.advance(params, G, max_len, t_d, length, prefix, start, act, torch.from_numpy(ot).to(DEV),
                    torch.from_numpy(ol).to(DEV))
        ref = _advance_ref(ref[0], ref[1], ot, ol, m, max_len, G)
    assert ref[4] < B


# ---------------------------------------------------------------- generation

@pytest.mark.parametrize("mpfr", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_generate_is_plain_keyed_decoding(psd, layout, mpfr):
    B, V, K, G, m, n_pos = 6, 3000, 4, 4, 3, 40
    tm = workloads.ToyModel(seed=77 + layout, draft_seed=5, sigma=3.0, alpha=1.2, tau=(0.4, 1.0), tau_split=3)
    key = 0x0123456789ABCDEF
    params = psd.make_params(key, V, K, m, 0.8, 0.8, dtype=torch.bfloat16, clocks=layout,
                             mode=psd.PSD_MODE_MPFR if mpfr else psd.PSD_MODE_HET)
    prompts = _prompts(B, m, V, 1).to(DEV)
    text, blocks, bits = psd.generate(params, _lm(psd, tm), prompts, n_pos, G, check_every=4)
    torch.cuda.synchronize()
    assert bits == 0 and blocks <= n_pos + 3
    tx = _np(text)
    assert np.array_equal(tx[:, :m], _np(prompts)) and (tx[:, m:] >= 0).all() and (tx < V).all()
    picks = [(b, t) for b in range(B) for t in range(m, m + n_pos)]
    exact, near = plain_chain_check(tm, key, K, m, V, 0.8, layout, tx, picks, mpfr)
    print(f"[gen] layout={layout} mpfr={mpfr} blocks={blocks} exact={exact} near={near}", flush=True)
    host, hb = host_loop(psd, params, _lm(psd, tm), prompts, n_pos, G)
    assert torch.equal(host, text)
    assert blocks - 4 < hb <= blocks


@pytest.mark.parametrize("mpfr", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_generate_graph_replay_and_drafter_substitution(psd, layout, mpfr):
    """The captured loop replays to the eager run's text; other drafters (another noise
    stream, other scales) change how many blocks it takes, not the text."""
    B, V, K, G, m, n_pos = 8, 5000, 4, 4, 4, 64
    key = 0x5A5A5A5A12345678
    params = psd.make_params(key, V, K, m, 1.0, 1.0, dtype=torch.bfloat16, clocks=layout,
                             mode=psd.PSD_MODE_MPFR if mpfr else psd.PSD_MODE_HET)
    prompts = _prompts(B, m, V, 2).to(DEV)
    runs = {}
    for name, tau, dseed, graph, every in (("eager", (0.5, 0.5), 9, False, 8), ("graph", (0.5, 0.5), 9, True, 8),
                                           ("graph5", (0.5, 0.5), 9, True, 5), ("close", (0.1, 0.1), 10, True, 8),
                                           ("far", (3.0, 3.0), 11, False, 16)):
        tm = workloads.ToyModel(seed=99, draft_seed=dseed, sigma=3.0, alpha=1.2, tau=tau)
        for rep in range(2 if graph else 1):  # replays after eager work in between
            text, blocks, bits = psd.generate(params, _lm(psd, tm), prompts, n_pos, G, check_every=every,
                                              use_graph=graph)
            torch.cuda.synchronize()
            assert bits == 0
            _ = torch.ones(1024, device=DEV).sum().item()
            if rep:
                assert torch.equal(text, runs[name][0])
            runs[name] = (text, blocks)
        print(f"[gen] {name}: {runs[name][1]} blocks", flush=True)
    for name in runs:
        assert torch.equal(runs[name][0], runs["eager"][0]), name
    assert runs["close"][1] < runs["far"][1]
    tm = workloads.ToyModel(seed=99, draft_seed=9, sigma=3.0, alpha=1.2, tau=(0.5, 0.5))
    rng = np.random.default_rng(layout)
    picks = [(int(b), int(t)) for b, t in zip(rng.integers(0, B, 40), rng.integers(m, m + n_pos, 40))]
    plain_chain_check(tm, key, K, m, V, 1.0, layout, _np(runs["eager"][0]), picks, mpfr)


@pytest.mark.parametrize("mpfr", [False, True])
def test_generate_top_k(psd, mpfr):
    B, V, K, G, m, n_pos = 4, 4000, 4, 4, 2, 32
    tm = workloads.ToyModel(seed=5, draft_seed=6, sigma=2.0, alpha=1.0, tau=(0.6, 0.6))
    key = 0x1234
    params = psd.make_params(key, V, K, m, 0.9, 0.9, dtype=torch.bfloat16, clocks=0,
                             mode=psd.PSD_MODE_MPFR if mpfr else psd.PSD_MODE_HET, top_k=50, top_p=0.9)
    prompts = _prompts(B, m, V, 3).to(DEV)
    text, blocks, bits = psd.generate(params, _lm(psd, tm), prompts, n_pos, G, check_every=4, use_graph=True)
    torch.cuda.synchronize()
    assert bits == 0
    picks = [(b, t) for b in range(B) for t in range(m, m + n_pos)]
    plain_chain_check(tm, key, K, m, V, 0.9, 0, _np(text), picks, mpfr, top_k=50, top_p=0.9)


def test_generate_stress_workload_then_detect(psd):
    """V=256000, K=16, gamma=4, bf16: 128 sequences x 512 positions with the key and 128
    with a wrong key, generated on the device (captured blocks), then detected with the
    key; the text is the plain keyed chain at sampled positions, S_A and M equal the
    oracle's on a sample of sequences, and the halves separate."""
    w = workloads.WORKLOADS[5]
    n_pos, half, layout = 512, w.B // 2, 0
    key, wrong = w.key, w.key ^ 0x5DEECE66D
    tm = workloads.ToyModel(seed=2026, draft_seed=12, sigma=w.sigma, alpha=w.alpha, tau=w.tau, tau_split=half // 2)
    texts, info = [], []
    for i, k in enumerate((key, wrong)):
        params = psd.make_params(k, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout)
        prompts = _prompts(half, w.m, w.V, 40 + i).to(DEV)
        print(f"[gen] stress half {i}: {half} x {n_pos} positions", flush=True)
        text, blocks, bits = psd.generate(params, _lm(psd, tm), prompts, n_pos, w.gamma, check_every=16,
                                          use_graph=True)
        torch.cuda.synchronize()
        assert bits == 0
        info.append(blocks)
        print(f"[gen]   {blocks} blocks", flush=True)
        texts.append(text)
    tk = [_np(t) for t in texts]
    rng = np.random.default_rng(7)
    for i, k in enumerate((key, wrong)):
        picks = [(int(b), int(t)) for b, t in zip(rng.integers(0, half, 12), rng.integers(w.m, w.m + n_pos, 12))]
        plain_chain_check(tm, k, w.K, w.m, w.V, w.T_target, layout, tk[i], picks, False)
    toks = torch.cat(texts, 0).contiguous()
    n0 = torch.full((w.B,), w.m, dtype=torch.int32, device=DEV)
    p = psd.make_params(key, w.V, w.K, w.m, dtype=w.torch_dtype, clocks=layout)
    score, count = psd.detect(p, toks, n0)[:2]
    torch.cuda.synchronize()
    score, count, all_tk = _np(score), _np(count), _np(toks)
    sample = list(range(0, w.B, 16))
    with concurrent.futures.ThreadPoolExecutor(WORKERS) as ex:
        refs = list(ex.map(lambda i: oracle.detect_sequence(key, w.m, w.K, w.V, all_tk[i], w.m, layout), sample))
    for i, (S, M, _) in zip(sample, refs):
        assert count[i] == M == n_pos and abs(score[i] - S) <= SCORE_TOL * abs(S), (i, score[i], S)
    z = (score - count) / np.sqrt(count)
    assert np.all(z[:half] > 5.0), z[:half].min()
    assert np.all(np.abs(z[half:]) < 4.5), np.abs(z[half:]).max()
