"""GPU parity of identical-drafter (MPFR) mode against the CPU oracle.

psd_verify / psd_draft with mode MPFR draw each context's nu(c) drafts as the
labels of its nu(c) smallest mapped-Poisson scores (cumulative clocks) and race
the target rows on slot 0; detection scores the slot-0 clock.  Per context the
GPU's samples must equal the oracle's in order, except inside runs of oracle
scores closer than 1e-6 (either order of near-tied arrivals is valid); target
tokens, accepted lengths and emitted tokens exactly as in the distinct-drafter
tests; LSE within 1e-5 relative (floor 1e-5 below |LSE| = 1).
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


def run_mpfr(psd, w, seed, layout, target_rows=1, mode="fused", gen_device="cpu", seqs=None, blk=None):
    print(f"[mpfr] {w.name} V={w.V} K={w.K} g={w.gamma} B={w.B} {w.dtype} T_Q={w.T_draft} layout={layout} "
          f"rows={target_rows} mode={mode} seed={seed}", flush=True)
    if blk is None:
        blk = workloads.make_block(w, seed, device=gen_device, target_rows=target_rows)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout,
                             mode=psd.PSD_MODE_MPFR)
    ws = psd.new_workspace(params, w.B, w.gamma, DEV)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    dl = torch.full((w.B, w.K, w.gamma), 7.0, dtype=torch.float32, device=DEV)
    if mode == "fused":
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                         target_rows=target_rows, want_lse=True, want_targets=True, status=status,
                         out={"draft_lse": dl})
    else:
        dt = torch.full((w.B, w.K, w.gamma), -7, dtype=torch.int32, device=DEV)
        st_d = torch.full((1,), -1, dtype=torch.int32, device=DEV)
        step = 2 if mode == "draft2" else 1  # two depths per call: one launch runs both
        for s in range(0, w.gamma, step):
            psd.draft(params, ws, g["prefix_tokens"], g["start_pos"], w.gamma, s,
                      g["draft_logits"][:, :, s:s + step].contiguous(), dt, dl, status=st_d)
            torch.cuda.synchronize()
            assert int(st_d[0]) == 0
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], None, dt,
                         target_rows=target_rows, want_lse=True, want_targets=True, status=status)
        out["draft_lse"] = dl
    torch.cuda.synchronize()
    assert int(status[0]) == 0 and psd.workspace_errors(ws) == 0
    seqs = list(range(w.B)) if seqs is None else list(seqs)
    gpu = {k: _np(v)[seqs] for k, v in out.items()}
    ref = oracle.verify_block_parallel(WORKERS, mpfr_mode=True, key=w.key, K=w.K, gamma=w.gamma, m=w.m,
                                       T_target=w.T_target, T_draft=w.T_draft,
                                       prefix=_np(blk["prefix_tokens"])[seqs], start_pos=_np(blk["start_pos"])[seqs],
                                       target_logits=workloads.as_f32_numpy(blk["target_logits"][seqs]),
                                       draft_logits=workloads.as_f32_numpy(blk["draft_logits"][seqs]),
                                       target_rows=target_rows, layout=layout, gpu=gpu)
    st = ref["stats"]
    assert st["mismatch"] == 0, st["mismatches"][:3]
    merged = 0
    for i in range(len(seqs)):
        n = int(gpu["out_len"][i])
        assert n == ref["out_len"][i], (i, n, ref["out_len"][i])
        assert list(gpu["out_tokens"][i][:n]) == ref["out_tokens"][i]
        assert all(x == -1 for x in gpu["out_tokens"][i][n:])
        d = gpu["draft_tokens"][i]
        merged += sum(len(oracle.context_groups([d[k, :s] for k in range(w.K)])) < w.K for s in range(1, w.gamma))
    for key, v in ref["target_lse"].items():
        got = gpu["target_lse"][key] if target_rows == 1 else gpu["target_lse"][key[0]][key[1]][key[2]]
        assert (got == v == -np.inf) or abs(got - v) <= LSE_TOL * max(1.0, abs(v)), (key, got, v)
    for (b, k, s), v in ref["draft_lse"].items():
        got = gpu["draft_lse"][b][k][s]
        assert (got == v == -np.inf) or abs(got - v) <= LSE_TOL * max(1.0, abs(v)), ((b, k, s), got, v)
    print(f"[mpfr]   exact={st['exact']} near_tie={st['near_tie']} depths with shared contexts={merged} "
          f"mean_tau={np.mean([ref['out_len'][i] for i in range(len(seqs))]):.3f}", flush=True)
    out["merged_depths"] = merged
    return out, ref


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_config1(psd, layout):
    for seed in range(4):
        run_mpfr(psd, workloads.WORKLOADS[1], seed, layout)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("case", [
    dict(V=1000, K=4, gamma=4, B=4, dtype="fp32", m=4, T_draft=0.3),   # peaked drafts: contexts merge deeper
    dict(V=777, K=3, gamma=3, B=3, dtype="bf16", m=0, T_draft=1.0),    # ragged, no window
    dict(V=3, K=5, gamma=3, B=3, dtype="fp32", m=2, T_draft=1.0),      # more drafts than tokens
    dict(V=1, K=2, gamma=2, B=1, dtype="fp32", m=1, T_draft=1.0),      # one token
    dict(V=40000, K=8, gamma=3, B=2, dtype="bf16", m=3, T_draft=0.5),  # several level-4 nodes, nu up to 8
    dict(V=20000, K=16, gamma=2, B=2, dtype="fp32", m=16, T_draft=2.0),  # nu = 16, long window
    dict(V=500, K=32, gamma=3, B=2, dtype="bf16", m=2, T_draft=1.0),    # the most drafters
    dict(V=300, K=2, gamma=32, B=2, dtype="fp32", m=4, T_draft=1.0),    # the most depths in one launch
])
def test_mpfr_ragged_and_edge_shapes(psd, layout, case):
    w = workloads.custom(case["V"], case["K"], case["gamma"], case["B"], dtype=case["dtype"], m=case["m"],
                         tau=0.7, sigma=2.0, alpha=1.0, T_draft=case["T_draft"])
    out, _ = run_mpfr(psd, w, 12, layout)
    if case["T_draft"] < 0.5:  # peaked drafts: paths share contexts past depth 0 (multiplicities > 1)
        assert out["merged_depths"] > 0


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_two_call_and_per_path(psd, layout):
    w = workloads.custom(5000, 4, 4, 4, dtype="bf16", m=3, tau=0.5, sigma=2.0, alpha=1.0, T_draft=0.6)
    blk = workloads.make_block(w, 3)
    a, _ = run_mpfr(psd, w, 3, layout, blk=blk)
    b, _ = run_mpfr(psd, w, 3, layout, mode="two_call", blk=blk)
    for k in ("draft_tokens", "out_tokens", "out_len", "target_tokens"):
        assert torch.equal(a[k], b[k]), k
    run_mpfr(psd, w, 4, layout, target_rows=w.K)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_wide_batch_streams_in_each_depth(psd, layout):
    """B K >= 1024 drafts with every depth's launch streaming its own rows (smaller
    batches stream all draft rows in one launch first): same parity bar, every 16th
    sequence checked."""
    w = workloads.custom(3000, 4, 3, 256, dtype="bf16", m=3, tau=0.5, sigma=2.0, alpha=1.0, T_draft=0.6)
    run_mpfr(psd, w, 21, layout, gen_device=DEV, seqs=range(0, w.B, 16))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_many_listed_tokens(psd, layout):
    """Flat and two-valued draft rows with 16 identical drafters: the seeds bound theta
    loosely, hundreds of tokens are listed (theta tightened, then nu = 16 arrivals of
    each), more than one workgroup's threads -- the samples then come from nu rounds
    that each rebuild only the winner's next arrival; random rows of the same block
    take the all-arrivals-at-once form.  Same parity bar."""
    w = workloads.custom(5000, 16, 2, 3, dtype="bf16", m=2, tau=0.5, sigma=2.0, alpha=1.0, T_draft=1.0)
    blk = workloads.make_block(w, 31)
    dl = blk["draft_logits"]
    dl[0] = 0.25                       # every logit equal
    dl[1, :, :, ::2] = 1.0             # two values
    dl[1, :, :, 1::2] = -1.0
    run_mpfr(psd, w, 31, layout, blk=blk)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_config2_full(psd, layout):
    run_mpfr(psd, workloads.WORKLOADS[2], 2, layout)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_config3_all_sequences(psd, layout):
    run_mpfr(psd, workloads.WORKLOADS[3], 3, layout, gen_device=DEV)


def test_mpfr_rows_without_finite_logits(psd):
    """Rows with no finite logit.  All paths of sequence 0 at depth 1: the context draws
    -1 for each of them, and the deeper contexts build on those drafts.  Path 2 of
    sequence 1 at depth 0: its context's proposal row is path 0's, so only its own LSE
    reads -inf.  A target row of sequence 2: its target is -1 and ends the block there.
    Everything as the oracle has it."""
    w = workloads.custom(700, 4, 4, 3, dtype="fp32", m=2, tau=0.7, sigma=2.0, alpha=1.0, T_draft=1.0)
    blk = workloads.make_block(w, 14)
    blk["draft_logits"][0, :, 1, :] = -np.inf
    blk["draft_logits"][1, 2, 0, :] = -np.inf
    blk["target_logits"][2, 3, :] = -np.inf
    for layout in LAYOUTS:
        out, _ = run_mpfr(psd, w, 14, layout, blk=blk)
        assert (out["draft_tokens"][0, :, 1] == -1).all()
        assert out["draft_lse"][1, 2, 0] == -np.inf


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_config4_sampled(psd, layout):
    """V=151936, K=8, gamma=8, B=128, fp32 logits: B K = 1024, so one sampling launch per
    depth, each streaming its rows (three workgroups per CU).  Every 16th sequence
    against the oracle."""
    run_mpfr(psd, workloads.WORKLOADS[4], 4, layout, gen_device=DEV, seqs=range(0, 128, 16))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_mpfr_config5_sampled(psd, layout):
    """V=256000, K=16, gamma=4, B=256, bf16: one sampling launch per depth with 4096
    workgroups, contexts of up to 16 identical drafters.  Every 32nd sequence against
    the oracle."""
    run_mpfr(psd, workloads.WORKLOADS[5], 5, layout, gen_device=DEV, seqs=range(3, 256, 32))


def test_mpfr_detection_pivot_is_slot0(psd):
    """Detection in MPFR mode scores the slot-0 clock: it equals the oracle's K = 1 score."""
    w = workloads.WORKLOADS[3]
    toks = workloads.uniform_tokens(8, 200, w.V, seed=4)
    n0 = torch.full((8,), w.m, dtype=torch.int32)
    for layout in LAYOUTS:
        p = psd.make_params(w.key, w.V, w.K, w.m, dtype=w.torch_dtype, clocks=layout, mode=psd.PSD_MODE_MPFR)
        score, count, per = psd.detect(p, toks.to(DEV), n0.to(DEV), per_token=True)
        torch.cuda.synchronize()
        for i in range(8):
            S, M, _ = oracle.detect_sequence(w.key, w.m, 1, w.V, _np(toks)[i], w.m, layout)
            assert int(count[i]) == M and abs(float(score[i]) - S) <= 1e-9 * abs(S)


def test_mpfr_side_stream_status_and_forced_wait_timeouts(psd):
    """With one shared target chain, the target races run on the library's side
    stream beside the drafting launches, and the walk kernel adds their error bits
    to the call's status word.  With a spin limit of one poll (set from the host) the
    race's waits for other workgroups give up at once: every kernel still exits, and
    bit 0 reaches the status word and the workspace's sticky bits.  With the limit
    restored and the workspace cleared, the same call is healthy and matches the oracle."""
    w = workloads.WORKLOADS[2]
    blk = workloads.make_block(w, 7)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype,
                             mode=psd.PSD_MODE_MPFR)
    ws = psd.new_workspace(params, w.B, w.gamma, DEV)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    print(f"[mpfr] forced wait timeouts {w.name}", flush=True)
    try:
        psd.set_spin_limit(1)
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                         status=status)
        torch.cuda.synchronize()
    finally:
        psd.set_spin_limit(0)
    assert int(status[0]) & psd.ERR_SPIN, int(status[0])
    assert psd.workspace_errors(ws) & psd.ERR_SPIN
    lens = _np(out["out_len"])
    assert np.all((lens >= 1) & (lens <= w.gamma + 1))  # outputs unreliable but well formed
    psd.workspace_clear(ws)
    status.fill_(-1)
    psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"], status=status)
    torch.cuda.synchronize()
    assert int(status[0]) == 0 and psd.workspace_errors(ws) == 0
    run_mpfr(psd, w, 7, 0, blk=blk)


def test_mpfr_side_stream_follows_caller_stream(psd):
    """The side stream's target races wait for the caller's earlier work on its
    stream.  On a non-default stream, a copy writes the target rows into a buffer
    that held other rows (every target race would pick token 5 there), and the call
    follows at once.  The outputs equal those of the oracle-checked call on rows
    already in place, and the target winners are returned on the caller's stream."""
    w = workloads.WORKLOADS[3]
    blk = workloads.make_block(w, 13, device=DEV)
    ref, _ = run_mpfr(psd, w, 13, 0, blk=blk, seqs=range(0, w.B, 16))
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype,
                             mode=psd.PSD_MODE_MPFR)
    ws = psd.new_workspace(params, w.B, w.gamma, DEV)
    buf = torch.zeros_like(g["target_logits"])
    buf[..., 5] = 30.0
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    print(f"[mpfr] caller stream ordering {w.name}", flush=True)
    with torch.cuda.stream(s):
        buf.copy_(g["target_logits"])
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], buf, g["draft_logits"],
                         want_targets=True, status=status)
        got = {k: v.clone() for k, v in out.items()}
    s.synchronize()
    assert int(status[0]) == 0 and psd.workspace_errors(ws) == 0
    for k in ("out_tokens", "out_len", "draft_tokens", "target_tokens"):
        assert torch.equal(got[k], ref[k]), k


@pytest.mark.parametrize("cfg", [1, 3])
def test_mpfr_draft_calls_of_two_depths(psd, cfg):
    """psd_draft over two depths per call: the second call's launch takes the first
    call's drafts from draft_tokens and its own first depth's drafts from the tagged
    slots of the same launch.  Samples, tokens and lengths as the oracle's."""
    w = workloads.WORKLOADS[cfg]
    assert w.gamma % 2 == 0
    run_mpfr(psd, w, 20 + cfg, 0, mode="draft2", gen_device=DEV, seqs=range(0, w.B, max(1, w.B // 8)))


def test_mpfr_epoch_across_sampling_forms(psd):
    """Two block shapes share one workspace: B K = 1000, more workgroups than fit the
    device together at this kernel's occupancy (768 on MI355X) but still under the
    streaming launch's limit, so one sampling launch per depth follows a streaming
    launch that records the call's epoch; and B K = 128,
    where one sampling launch runs every depth beside the streaming launch and waits
    for its tagged words.  The shapes' tagged words sit at different offsets, so a stale
    tag would show up as a wrong draft.  Alternating the two, every call equals the same
    call on a fresh workspace, which matches the oracle."""
    wa = workloads.custom(2048, 8, 4, 125, dtype="bf16", T_target=0.8, T_draft=0.8)
    wb = workloads.custom(2048, 8, 4, 16, dtype="bf16", T_target=0.8, T_draft=0.8)
    blk_a = workloads.make_block(wa, 31, device=DEV)
    blk_b = workloads.make_block(wb, 32, device=DEV)
    ref_a, _ = run_mpfr(psd, wa, 31, 0, blk=blk_a, seqs=range(0, wa.B, 25))
    ref_b, _ = run_mpfr(psd, wb, 32, 0, blk=blk_b, seqs=range(0, wb.B, 4))
    pa = psd.make_params(wa.key, wa.V, wa.K, wa.m, wa.T_target, wa.T_draft, dtype=wa.torch_dtype,
                         mode=psd.PSD_MODE_MPFR)
    pb = psd.make_params(wb.key, wb.V, wb.K, wb.m, wb.T_target, wb.T_draft, dtype=wb.torch_dtype,
                         mode=psd.PSD_MODE_MPFR)
    n = max(psd.workspace_bytes(pa, wa.B, wa.gamma), psd.workspace_bytes(pb, wb.B, wb.gamma))
    ws = torch.zeros(n, dtype=torch.uint8, device=DEV)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    for rep in range(3):
        for name, p, blk, ref in (("B=125", pa, blk_a, ref_a), ("B=16", pb, blk_b, ref_b)):
            print(f"[mpfr] shared workspace, pass {rep}, {name}", flush=True)
            out = psd.verify(p, ws, blk["prefix_tokens"], blk["start_pos"], blk["target_logits"],
                             blk["draft_logits"], want_targets=True, status=status)
            torch.cuda.synchronize()
            assert int(status[0]) == 0 and psd.workspace_errors(ws) == 0
            for k in ("out_tokens", "out_len", "draft_tokens", "target_tokens"):
                assert torch.equal(out[k], ref[k]), (rep, name, k)


def test_modes_alternate_on_one_workspace(psd):
    """Distinct-drafter and identical-drafter calls of one block alternate on one
    workspace (sized for the larger): the race kernel's epoch and the identical-drafter
    launches' epoch advance independently, and every call equals the same call on a
    fresh workspace."""
    w = workloads.WORKLOADS[2]
    blk = workloads.make_block(w, 17, device=DEV)
    ph = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype)
    pm = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, mode=psd.PSD_MODE_MPFR)

    def call(p, ws):
        out = psd.verify(p, ws, blk["prefix_tokens"], blk["start_pos"], blk["target_logits"], blk["draft_logits"],
                         want_targets=True)
        torch.cuda.synchronize()
        assert psd.workspace_errors(ws) == 0
        return {k: v.clone() for k, v in out.items()}

    ref = {"het": call(ph, psd.new_workspace(ph, w.B, w.gamma, DEV)),
           "mpfr": call(pm, psd.new_workspace(pm, w.B, w.gamma, DEV))}
    n = max(psd.workspace_bytes(ph, w.B, w.gamma), psd.workspace_bytes(pm, w.B, w.gamma))
    ws = torch.zeros(n, dtype=torch.uint8, device=DEV)
    for rep in range(3):
        for name, p in (("het", ph), ("mpfr", pm), ("mpfr", pm), ("het", ph)):
            print(f"[mpfr] shared workspace, pass {rep}, {name}", flush=True)
            got = call(p, ws)
            for k in ("out_tokens", "out_len", "draft_tokens", "target_tokens"):
                assert torch.equal(got[k], ref[name][k]), (rep, name, k)
