"""GPU parity of top-k / top-p truncated races against the CPU oracle.

With params.top_k > 0 every row (draft and target) is truncated before its race:
the top_k largest logits (ties to the lowest index), then the shortest prefix of
those whose softmax mass at the row's temperature reaches top_p; the other tokens
have probability 0.  The oracle races the same rows with the truncated tokens set
to -inf (oracle.truncate_block), so the truncation itself is checked through every
race it feeds: drafts, target tokens, accepted lengths and emitted tokens exactly
(near-ties as in the other parity tests), and the LSE of each kept set within 1e-5
relative (floor 1e-5 below |LSE| = 1).
"""
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
LSE_TOL = 1e-5
RADIX_WORD = 6  # workspace control word counting rows selected by the radix fallback
LAYOUTS = [0, 1]
WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module")
def psd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21858_amd import psd as m
    return m


def _np(t):
    return t.detach().cpu().numpy()


def _params(psd, w, layout, mpfr, top_k, top_p):
    return psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout,
                           mode=psd.PSD_MODE_MPFR if mpfr else psd.PSD_MODE_HET, top_k=top_k, top_p=top_p)


def run_gpu(psd, w, blk, layout, mpfr, top_k, top_p, target_rows=1, mode="fused"):
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = _params(psd, w, layout, mpfr, top_k, top_p)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    if mode == "static":
        B, K, G = w.B, w.K, w.gamma
        shp = (B, G + 1) if target_rows == 1 else (B, K, G + 1)
        out = {"draft_tokens": torch.full((B, K, G), -7, dtype=torch.int32, device=DEV),
               "out_tokens": torch.empty((B, G + 1), dtype=torch.int32, device=DEV),
               "out_len": torch.empty((B,), dtype=torch.int32, device=DEV),
               "target_lse": torch.empty(shp, dtype=torch.float32, device=DEV),
               "draft_lse": torch.empty((B, K, G), dtype=torch.float32, device=DEV),
               "target_tokens": torch.empty(shp, dtype=torch.int32, device=DEV)}
        psd.verify_static(params, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                          target_rows=target_rows, out=out, status=status)
        torch.cuda.synchronize()
        assert int(status[0]) == 0
        return out
    ws = psd.new_workspace(params, w.B, w.gamma, DEV)
    if mode == "fused":
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                         target_rows=target_rows, want_lse=True, want_targets=True, status=status)
    else:  # psd_draft per depth, then verify with the drafts given
        dt = torch.full((w.B, w.K, w.gamma), -7, dtype=torch.int32, device=DEV)
        dl = torch.empty((w.B, w.K, w.gamma), dtype=torch.float32, device=DEV)
        st_d = torch.full((1,), -1, dtype=torch.int32, device=DEV)
        for s in range(w.gamma):
            psd.draft(params, ws, g["prefix_tokens"], g["start_pos"], w.gamma, s,
                      g["draft_logits"][:, :, s:s + 1].contiguous(), dt, dl, status=st_d)
            torch.cuda.synchronize()
            assert int(st_d[0]) == 0
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], None, dt,
                         target_rows=target_rows, want_lse=True, want_targets=True, status=status)
        out["draft_lse"] = dl
    torch.cuda.synchronize()
    assert int(status[0]) == 0 and psd.workspace_errors(ws) == 0
    out["_radix_rows"] = int(ws[4 * RADIX_WORD:4 * RADIX_WORD + 4].view(torch.int32)[0])
    return out


def run_topk(psd, w, seed, layout, mpfr, top_k, top_p=1.0, target_rows=1, mode="fused", gen_device="cpu",
             seqs=None, blk=None):
    print(f"[topk] {w.name} V={w.V} K={w.K} g={w.gamma} B={w.B} {w.dtype} layout={layout} mpfr={mpfr} "
          f"top_k={top_k} top_p={top_p} rows={target_rows} mode={mode} seed={seed}", flush=True)
    if blk is None:
        blk = workloads.make_block(w, seed, device=gen_device, target_rows=target_rows)
    out = run_gpu(psd, w, blk, layout, mpfr, top_k, top_p, target_rows, mode)
    seqs = list(range(w.B)) if seqs is None else list(seqs)
    gpu = {k: _np(v)[seqs] for k, v in out.items() if not k.startswith("_")}
    tl = oracle.truncate_block(workloads.as_f32_numpy(blk["target_logits"][seqs]), w.T_target, top_k, top_p)
    dl = oracle.truncate_block(workloads.as_f32_numpy(blk["draft_logits"][seqs]), w.T_draft, top_k, top_p)
    ref = oracle.verify_block_parallel(WORKERS, mpfr_mode=mpfr, key=w.key, K=w.K, gamma=w.gamma, m=w.m,
                                       T_target=w.T_target, T_draft=w.T_draft,
                                       prefix=_np(blk["prefix_tokens"])[seqs], start_pos=_np(blk["start_pos"])[seqs],
                                       target_logits=tl, draft_logits=dl, target_rows=target_rows, layout=layout,
                                       gpu=gpu)
    st = ref["stats"]
    assert st["mismatch"] == 0, st["mismatches"][:3]
    for i in range(len(seqs)):
        n = int(gpu["out_len"][i])
        assert n == ref["out_len"][i], (i, n, ref["out_len"][i])
        assert list(gpu["out_tokens"][i][:n]) == ref["out_tokens"][i]
        assert all(x == -1 for x in gpu["out_tokens"][i][n:])
    for key, v in ref["target_lse"].items():
        got = gpu["target_lse"][key] if target_rows == 1 else gpu["target_lse"][key[0]][key[1]][key[2]]
        assert (got == v == -np.inf) or abs(got - v) <= LSE_TOL * max(1.0, abs(v)), (key, got, v)
    for (b, k, s), v in ref["draft_lse"].items():
        got = gpu["draft_lse"][b][k][s]
        assert (got == v == -np.inf) or abs(got - v) <= LSE_TOL * max(1.0, abs(v)), ((b, k, s), got, v)
    # every emitted token lies in its row's kept set (the race never leaves the support)
    kept_t = tl != -np.inf
    for i in range(len(seqs)):
        for s in range(int(gpu["out_len"][i])):
            y = int(gpu["out_tokens"][i][s])
            if target_rows == 1:
                assert y < 0 or kept_t[i, s, y], (i, s, y)
    print(f"[topk]   exact={st['exact']} near_tie={st['near_tie']} "
          f"mean_tau={np.mean([ref['out_len'][i] for i in range(len(seqs))]):.3f}", flush=True)
    return out, ref, blk


@pytest.mark.parametrize("mpfr", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_topk50_config3(psd, layout, mpfr):
    """top-k = 50, the paper's setting, on the Llama-3 vocabulary block (every 2nd sequence)."""
    w = workloads.WORKLOADS[3]
    out, _, _ = run_topk(psd, w, 5, layout, mpfr, 50, gen_device=DEV, seqs=range(0, w.B, 2))
    assert out["_radix_rows"] == 0  # random rows: the group-maximum candidates suffice


@pytest.mark.parametrize("mpfr", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("top_k,top_p", [(50, 0.9), (256, 0.95), (7, 0.5), (256, 1.0)])
def test_top_p_config2(psd, layout, mpfr, top_k, top_p):
    w = workloads.WORKLOADS[2]
    run_topk(psd, w, 6, layout, mpfr, top_k, top_p, seqs=range(0, w.B, 2))


@pytest.mark.parametrize("mpfr", [False, True])
def test_top1_is_greedy(psd, mpfr):
    """top-k = 1 with drafts equal to the target rows: every draft is the row's argmax
    (lowest index on ties), the target agrees and the whole block is accepted."""
    w = workloads.custom(3000, 4, 5, 6, dtype="bf16", m=3, tau=0.5, sigma=2.0, alpha=1.0)
    blk = workloads.make_block(w, 7)
    blk["draft_logits"] = blk["target_logits"][:, None, :w.gamma].expand(w.B, w.K, w.gamma, w.V).contiguous()
    out, _, _ = run_topk(psd, w, 7, 0, mpfr, 1, blk=blk)
    am = _np(blk["target_logits"].float().argmax(dim=-1))  # torch argmax: first maximal index
    assert (_np(out["out_len"]) == w.gamma + 1).all()
    assert np.array_equal(_np(out["out_tokens"]), am)
    assert (_np(out["draft_tokens"]) == am[:, None, :w.gamma]).all()


@pytest.mark.parametrize("mpfr", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_topk_beyond_support_equals_untruncated(psd, layout, mpfr):
    """top_k at least the number of finite logits keeps every token: the list path must
    reproduce the full-vocabulary race kernels exactly, including rows with a few finite
    logits and rows with none."""
    w = workloads.custom(200, 4, 4, 4, dtype="fp32", m=2, tau=0.7, sigma=2.0, alpha=1.0)
    blk = workloads.make_block(w, 8)
    tl, dl = blk["target_logits"], blk["draft_logits"]
    tl[1, 2, :] = -np.inf            # a target row with no finite logit
    tl[2, :, 3:] = -np.inf           # target rows with three finite logits
    dl[0, 1, 0, :] = -np.inf         # a draft row with none
    dl[3, :, :, 5:] = -np.inf        # draft rows with five
    a, _, _ = run_topk(psd, w, 8, layout, mpfr, 256, blk=blk)
    b = run_gpu(psd, w, blk, layout, mpfr, 0, 1.0)
    for k in ("draft_tokens", "out_tokens", "out_len", "target_tokens"):
        assert torch.equal(a[k], b[k]), k
    for k in ("target_lse", "draft_lse"):
        x, y = _np(a[k]), _np(b[k])
        fin = np.isfinite(y)
        assert np.array_equal(np.isfinite(x), fin)
        assert np.allclose(x[fin], y[fin], rtol=1e-5, atol=1e-5), k


@pytest.mark.parametrize("mpfr", [False, True])
def test_topk_ties_and_signed_zeros(psd, mpfr):
    """Logits on a coarse grid (many exact ties at the cut, +0 and -0 both present): the
    kept set takes tied tokens in index order, as the oracle does."""
    w = workloads.custom(1500, 4, 4, 4, dtype="bf16", m=2, tau=0.7, sigma=2.0, alpha=1.0)
    blk = workloads.make_block(w, 9)
    for k in ("target_logits", "draft_logits"):
        x = torch.round(blk[k].float() * 2.0) / 2.0
        x = torch.where((x == 0) & (torch.arange(w.V) % 2 == 1), torch.tensor(-0.0), x)
        blk[k] = x.to(w.torch_dtype)
    for top_k, top_p in ((20, 1.0), (64, 0.8), (3, 1.0)):
        run_topk(psd, w, 9, 1, mpfr, top_k, top_p, blk=blk)
    # rows whose ties at the cut overflow the candidate buffers (every logit equal, or
    # two values, at V = 5000): selected again by radix passes, with the same result as
    # the oracle
    w = workloads.custom(5000, 4, 4, 4, dtype="bf16", m=2, tau=0.7, sigma=2.0, alpha=1.0)
    blk = workloads.make_block(w, 9)
    tl, dl = blk["target_logits"], blk["draft_logits"]
    tl[0] = 1.5
    tl[1, :, ::2] = 0.5
    tl[1, :, 1::2] = -0.0
    dl[2, :2] = -2.0
    out, _, _ = run_topk(psd, w, 9, 0, mpfr, 50, 0.9, blk=blk)
    assert out["_radix_rows"] > 0

@pytest.mark.parametrize("mpfr", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_topk_two_call_per_path_and_static(psd, layout, mpfr):
    w = workloads.custom(5000, 4, 4, 4, dtype="bf16", m=3, tau=0.5, sigma=2.0, alpha=1.0, T_draft=0.8)
    blk = workloads.make_block(w, 10)
    a, _, _ = run_topk(psd, w, 10, layout, mpfr, 40, 0.9, blk=blk)
    b, _, _ = run_topk(psd, w, 10, layout, mpfr, 40, 0.9, blk=blk, mode="two_call")
    c = run_gpu(psd, w, blk, layout, mpfr, 40, 0.9, mode="static")
    for k in ("draft_tokens", "out_tokens", "out_len", "target_tokens"):
        assert torch.equal(a[k], b[k]), k
        assert torch.equal(a[k], c[k]), k
    run_topk(psd, w, 11, layout, mpfr, 40, 0.9, target_rows=w.K)


def test_topk_fp32_large_vocab_many_drafts(psd):
    """fp32 rows of the Qwen vocabulary, 8 drafts of 8 tokens (a few sequences)."""
    w = workloads.WORKLOADS[4]
    w = workloads.custom(w.V, w.K, w.gamma, 6, dtype="fp32", m=w.m, tau=0.6, sigma=2.5, alpha=1.0)
    run_topk(psd, w, 12, 0, False, 50, 0.95)
    run_topk(psd, w, 12, 1, True, 50, 0.95)
