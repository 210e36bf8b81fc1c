"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Token indices, accepted lengths and Philox words must match exactly, except
near-ties (oracle score gap below 1e-6 in natural-log units, i.e. a relative gap
of E/p below 1e-6), where either token is accepted and the comparison continues
in the GPU's context.  Log-sum-exp values must agree within 1e-5 relative, with
an absolute floor of 1e-5 below |LSE| = 1 (fp32 accumulation has an absolute
error floor); detection scores within 1e-9 relative (they are summed in fp64
from exact clocks).  The oracle checks the sequences of a call on several host
threads (its C code runs without the interpreter lock).
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
LSE_TOL = 1e-5
SCORE_TOL = 1e-9
LAYOUTS = [0, 1]  # tree, flat
WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module")
def psd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21858_amd import psd as m
    return m


def _np(t):
    return t.detach().cpu().numpy()


def _sync():
    torch.cuda.synchronize()


def run_block(psd, w, seed, layout, target_rows=1, mode="fused", gen_device="cpu", seqs=None, blk=None):
    """Run one verify call on the GPU and check it against the oracle on `seqs`."""
    print(f"[parity] {w.name} V={w.V} K={w.K} g={w.gamma} B={w.B} {w.dtype} layout={layout} rows={target_rows} "
          f"mode={mode} seed={seed}", flush=True)
    if blk is None:
        blk = workloads.make_block(w, seed, device=gen_device, target_rows=target_rows)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout)
    ws = psd.new_workspace(params, w.B, w.gamma, DEV)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    if mode == "fused":
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                         target_rows=target_rows, want_lse=True, want_targets=True, status=status)
    else:  # psd_draft per depth, then verify with the drafts given
        dt = torch.full((w.B, w.K, w.gamma), -7, dtype=torch.int32, device=DEV)
        dl = torch.empty((w.B, w.K, w.gamma), dtype=torch.float32, device=DEV)
        for s in range(w.gamma):
            psd.draft(params, ws, g["prefix_tokens"], g["start_pos"], w.gamma, s,
                      g["draft_logits"][:, :, s:s + 1].contiguous(), dt, dl)
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], None, dt,
                         target_rows=target_rows, want_lse=True, want_targets=True, status=status)
        out["draft_lse"] = dl
    _sync()
    assert int(status[0]) == 0  # the call's own error bits, written by its last workgroup
    assert psd.workspace_errors(ws) == 0
    seqs = list(range(w.B)) if seqs is None else list(seqs)
    gpu = {k: _np(v)[seqs] for k, v in out.items()}
    tl = workloads.as_f32_numpy(blk["target_logits"][seqs])
    dl = workloads.as_f32_numpy(blk["draft_logits"][seqs])
    ref = oracle.verify_block_parallel(WORKERS, key=w.key, K=w.K, gamma=w.gamma, m=w.m, T_target=w.T_target,
                                       T_draft=w.T_draft, prefix=_np(blk["prefix_tokens"])[seqs],
                                       start_pos=_np(blk["start_pos"])[seqs], target_logits=tl, draft_logits=dl,
                                       target_rows=target_rows, layout=layout, gpu=gpu)
    st = ref["stats"]
    assert st["mismatch"] == 0, st["mismatches"][:5]
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
    print(f"[parity]   exact={st['exact']} near_tie={st['near_tie']} mean_tau="
          f"{np.mean([ref['out_len'][i] for i in range(len(seqs))]):.3f}", flush=True)
    return out, ref


# ---------------------------------------------------------------- keyed randomness

def test_philox_words_bit_exact(psd):
    rng = np.random.default_rng(1)
    n = 4096
    ctr = rng.integers(0, 2**32, (n, 4), dtype=np.uint64).astype(np.uint32)
    key = rng.integers(0, 2**32, (n, 2), dtype=np.uint64).astype(np.uint32)
    ctr[0] = 0
    key[0] = 0
    ctr[1] = 0xFFFFFFFF
    key[1] = 0xFFFFFFFF
    out = _np(psd.philox(torch.from_numpy(ctr.view(np.int32)).to(DEV), torch.from_numpy(key.view(np.int32)).to(DEV)))
    out = out.view(np.uint32)
    for i in range(0, n, 7):
        assert list(out[i]) == oracle.philox(ctr[i], key[i]), i


def test_philox_known_answers(psd):
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", "philox4x32_10_kat.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                rows.append([int(x, 16) for x in line.split()])
    w = np.array(rows, dtype=np.uint64).astype(np.uint32)
    ctr = torch.from_numpy(np.ascontiguousarray(w[:, :4]).view(np.int32)).to(DEV)
    key = torch.from_numpy(np.ascontiguousarray(w[:, 4:6]).view(np.int32)).to(DEV)
    out = _np(psd.philox(ctr, key)).view(np.uint32)
    assert np.array_equal(out, w[:, 6:10])


def test_context_keys_bit_exact(psd):
    rng = np.random.default_rng(2)
    for m in (0, 1, 4, 16):
        n = 300
        t = rng.integers(0, 2**40, n).astype(np.int64)
        win = rng.integers(-1, 300000, (n, m)).astype(np.int32)
        p = psd.make_params(0x0123456789ABCDEF, 1000, 2, m)
        got = _np(psd.context_keys(p, torch.from_numpy(t).to(DEV), torch.from_numpy(win).to(DEV))).view(np.uint32)
        for i in range(n):
            assert tuple(int(x) for x in got[i]) == oracle.context_key(0x0123456789ABCDEF, int(t[i]), list(win[i]))


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("V", [1, 9, 1000, 128256, 1 << 19])
def test_clock_values(psd, layout, V):
    rng = np.random.default_rng(V + layout)
    n = 2000
    kappa = rng.integers(0, 2**32, (n, 2), dtype=np.uint64).astype(np.uint32)
    slot = rng.integers(0, 32, n).astype(np.int32)
    tok = rng.integers(0, V, n).astype(np.int32)
    p = psd.make_params(1, V, 32, 0, clocks=layout)
    got = _np(psd.clock_values(p, torch.from_numpy(kappa.view(np.int32)).to(DEV), torch.from_numpy(slot).to(DEV),
                               torch.from_numpy(tok).to(DEV)))
    for i in range(0, n, 3):
        want = oracle.clock(kappa[i], int(slot[i]), V, int(tok[i]), layout)
        assert abs(got[i] - want) <= 1e-13 * want, (i, got[i], want)


# ---------------------------------------------------------------- full path, small configs

@pytest.mark.parametrize("layout", LAYOUTS)
def test_config1_fused(psd, layout):
    for seed in range(6):
        run_block(psd, workloads.WORKLOADS[1], seed, layout)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("case", [
    dict(V=1000, K=3, gamma=4, B=3, dtype="fp32", m=4),   # ragged V (not a multiple of 8)
    dict(V=777, K=2, gamma=2, B=2, dtype="bf16", m=0),    # ragged, no context window
    dict(V=3, K=2, gamma=3, B=4, dtype="fp32", m=2),      # tiny vocabulary
    dict(V=1, K=1, gamma=1, B=1, dtype="fp32", m=1),      # degenerate: one token
    dict(V=4100, K=5, gamma=6, B=2, dtype="bf16", m=7),   # several groups + ragged tail
    dict(V=33000, K=1, gamma=3, B=2, dtype="fp32", m=3),  # single draft, two level-4 nodes
    dict(V=20000, K=7, gamma=2, B=3, dtype="bf16", m=16), # long window
])
def test_ragged_and_edge_shapes(psd, layout, case):
    w = workloads.custom(case["V"], case["K"], case["gamma"], case["B"], dtype=case["dtype"], m=case["m"],
                         tau=0.7, sigma=2.0, alpha=1.0)
    run_block(psd, w, 11, layout)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_per_path_target_rows(psd, layout):
    w = workloads.custom(3000, 3, 3, 4, dtype="bf16", m=3, tau=0.5, sigma=2.0, alpha=1.0)
    run_block(psd, w, 5, layout, target_rows=3)
    run_block(psd, w, 6, layout, target_rows=3, mode="two_call")


@pytest.mark.parametrize("layout", LAYOUTS)
def test_two_call_path_equals_fused(psd, layout):
    w = workloads.custom(5000, 4, 4, 5, dtype="fp32", m=4, tau=0.6)
    blk = workloads.make_block(w, 21)
    a, _ = run_block(psd, w, 21, layout, blk=blk)
    b, _ = run_block(psd, w, 21, layout, mode="two_call", blk=blk)
    for k in ("draft_tokens", "out_tokens", "out_len", "target_tokens"):
        assert torch.equal(a[k], b[k]), k


def test_temperatures_and_neg_inf(psd):
    w = workloads.custom(2048, 3, 3, 3, dtype="fp32", m=2, T_target=0.3, T_draft=2.5)
    blk = workloads.make_block(w, 4)
    blk["target_logits"][0, 1, :2000] = -float("inf")   # a nearly empty row
    blk["target_logits"][1, 2, :] = -float("inf")       # an empty target row -> -1, rejection
    blk["draft_logits"][2, 0, 0, :] = -float("inf")     # an empty draft row -> -1
    blk["draft_logits"][2, 1, 1, 100:] = -float("inf")
    for layout in LAYOUTS:
        out, ref = run_block(psd, w, 4, layout, blk=blk)
        assert int(out["target_tokens"][1, 2]) == -1
        assert int(out["draft_tokens"][2, 0, 0]) == -1
        assert math.isinf(float(out["target_lse"][1, 2]))


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_flat_and_two_level_rows(psd, layout, dtype):
    """Rows whose logits are all equal, or take two values, leave almost every group
    and chunk able to win: the evaluation lists overflow their LDS capacity and the
    overflow is scored by each chunk's own lane."""
    w = workloads.custom(20000, 4, 2, 2, dtype=dtype, m=3)
    blk = workloads.make_block(w, 31)
    tl, dl = blk["target_logits"], blk["draft_logits"]
    tl[0, 0, :] = 0.0
    tl[0, 1, :] = 0.5
    tl[1, 0, :] = torch.where(torch.arange(w.V) % 3 == 0, 1.0, 0.0).to(tl.dtype)
    dl[0, 0, 0, :] = 0.0
    dl[1, 2, 1, :] = torch.where(torch.arange(w.V) % 5 == 0, 2.0, 1.0).to(dl.dtype)
    run_block(psd, w, 31, layout, blk=blk)


def test_determinism_and_workspace_reuse(psd):
    w = workloads.custom(6000, 3, 3, 4, dtype="bf16", m=4)
    blk = workloads.make_block(w, 8)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = psd.make_params(w.key, w.V, w.K, w.m, dtype=torch.bfloat16)
    ws = psd.new_workspace(params, 8, 5, DEV)  # larger than needed, reused
    outs = []
    for _ in range(3):
        outs.append(psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                               want_lse=True, want_targets=True))
    small = workloads.custom(6000, 3, 2, 2, dtype="bf16", m=4)
    sb = workloads.make_block(small, 9)
    sg = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in sb.items()}
    psd.verify(params, ws, sg["prefix_tokens"], sg["start_pos"], sg["target_logits"], sg["draft_logits"])
    outs.append(psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                           want_lse=True, want_targets=True))
    _sync()
    assert psd.workspace_errors(ws) == 0
    for o in outs[1:]:
        for k in o:
            assert torch.equal(o[k], outs[0][k]), k


# ---------------------------------------------------------------- full-size configs

@pytest.mark.parametrize("layout", LAYOUTS)
def test_config2_full(psd, layout):
    run_block(psd, workloads.WORKLOADS[2], 2, layout)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config3_all_sequences(psd, layout):
    """The headline shape, every one of the 64 sequences (both draft-noise halves)."""
    run_block(psd, workloads.WORKLOADS[3], 3, layout, gen_device=DEV)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config3_per_path_target_rows(psd, layout):
    """Per-path target rows (target_rows = K) at the headline shape, all sequences."""
    w = workloads.WORKLOADS[3]
    run_block(psd, w, 33, layout, target_rows=w.K, gen_device=DEV)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config4_every_8th_sequence(psd, layout):
    """V=151936, K=8, gamma=8, B=128 fp32: sequences 0, 8, ..., 120 checked in full."""
    run_block(psd, workloads.WORKLOADS[4], 4, layout, gen_device=DEV, seqs=range(0, 128, 8))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config5_every_8th_sequence(psd, layout):
    """V=256000, K=16, gamma=4, B=256 bf16: sequences 3, 11, ..., 251 checked in full."""
    run_block(psd, workloads.WORKLOADS[5], 5, layout, gen_device=DEV, seqs=range(3, 256, 8))


@pytest.mark.parametrize("layout", LAYOUTS)
def test_large_logit_offsets_and_small_temperatures(psd, layout):
    """fp32 logits shifted by +1e4, -1e4 and +3e3 (softmax-invariant) at T_P = 0.05 and
    T_Q = 0.02, scaled so that the distributions are the generator's at T = 1: |l|/T
    reaches 5e5, where l/T alone rounds by ~0.03 in fp32.  The race scores and bounds
    use (l - row maximum)/T, so the pruning margins still hold."""
    w = workloads.custom(20000, 3, 3, 4, dtype="fp32", m=3, T_target=0.05, T_draft=0.02, tau=0.7, sigma=2.0,
                         alpha=1.0)
    blk = workloads.make_block(w, 41)
    for b, off in enumerate((1e4, -1e4, 3000.0, 0.0)):
        blk["target_logits"][b] = blk["target_logits"][b] * 0.05 + off
        blk["draft_logits"][b] = blk["draft_logits"][b] * 0.02 + off
    run_block(psd, w, 41, layout, blk=blk)


def test_status_word_and_forced_wait_timeouts(psd):
    """The call's status word carries its own error bits.  With a spin limit of one
    poll (set from the host), the waits for other workgroups' values give up at
    once: the call still completes (every kernel exits) and reports bit 0, in the
    status word and in the workspace's sticky bits.  After the limit is restored
    and the workspace cleared, the same call is healthy again and matches the oracle."""
    w = workloads.WORKLOADS[2]
    blk = workloads.make_block(w, 7)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in blk.items()}
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype)
    ws = psd.new_workspace(params, w.B, w.gamma, DEV)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    try:
        psd.set_spin_limit(1)
        out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                         status=status)
        _sync()
    finally:
        psd.set_spin_limit(0)
    assert int(status[0]) & psd.ERR_SPIN, int(status[0])
    assert psd.workspace_errors(ws) & psd.ERR_SPIN
    lens = _np(out["out_len"])
    assert np.all((lens >= 1) & (lens <= w.gamma + 1))  # outputs unreliable but well formed
    psd.workspace_clear(ws)
    status.fill_(-1)
    out = psd.verify(params, ws, g["prefix_tokens"], g["start_pos"], g["target_logits"], g["draft_logits"],
                     status=status, want_targets=True)
    _sync()
    assert int(status[0]) == 0 and psd.workspace_errors(ws) == 0
    run_block(psd, w, 7, 0, blk=blk)


# ---------------------------------------------------------------- detection

def _generate(psd, w, key, n_pos, seed, layout=0):
    """Multi-block generation over a position-indexed toy LM with the GPU sampler."""
    from gen_loop import generate, table_positions
    B, K, G, V = w.B, w.K, w.gamma, w.V
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    prompt = torch.randint(0, V, (B, w.m), generator=gen, device=DEV, dtype=torch.int64).to(torch.int32)
    P = table_positions(w.m, n_pos, G)
    rows = workloads.target_rows_fp32(w, B * P, gen, DEV).view(B, P, V)
    params = psd.make_params(key, V, K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout)
    ws = psd.new_workspace(params, B, G, DEV)

    def verify(prefix, start, tl, dl):
        out = psd.verify(params, ws, prefix, start, tl, dl)
        _sync()
        assert psd.workspace_errors(ws) == 0
        return _np(out["out_tokens"]), _np(out["out_len"])

    text, _ = generate(verify, rows, prompt, n_pos, G, K, 0.8, gen, w.torch_dtype)
    return text


@pytest.mark.parametrize("layout", LAYOUTS)
def test_detect_parity_and_power(psd, layout):
    w = workloads.custom(5000, 4, 4, 6, dtype="bf16", m=3, sigma=3.0, alpha=1.2)
    key, wrong = 0x1111222233334444, 0x5555666677778888
    wm = _generate(psd, w, key, 60, 1, layout)
    nw = _generate(psd, w, wrong, 60, 2, layout)
    toks = torch.cat([wm, nw], 0)
    toks[0, 10] = 99999   # out of range: not scored
    n0 = torch.full((toks.shape[0],), w.m, dtype=torch.int32, device=DEV)
    n0[1] = 200           # nothing scored
    p = psd.make_params(key, w.V, w.K, w.m, dtype=torch.bfloat16, clocks=layout)
    score, count, per = psd.detect(p, toks, n0, per_token=True)
    log_p, anl = psd.detect_pvalue(score, count)
    _sync()
    score, count, per, tk = _np(score), _np(count), _np(per), _np(toks)
    _check_pvalues(score, count, _np(log_p), _np(anl))
    for i in range(tk.shape[0]):
        S, M, ref_per = oracle.detect_sequence(key, w.m, w.K, w.V, tk[i], int(_np(n0)[i]), layout)
        assert count[i] == M
        assert abs(score[i] - S) <= SCORE_TOL * abs(S) + 1e-12, (i, score[i], S)
        ok = ~np.isnan(ref_per)
        assert np.array_equal(np.isnan(per[i]), ~ok)
        assert np.allclose(per[i][ok], ref_per[ok], rtol=1e-5, atol=1e-6)
    # watermarked text scores far above its null mean M; the wrong key's does not
    z = (score - count) / np.sqrt(np.maximum(count, 1))
    assert np.all(z[[0, 2, 3, 4, 5]] > 3.0), z
    assert np.all(np.abs(z[6:]) < 4.5), z


@pytest.mark.parametrize("layout", LAYOUTS)
def test_config5_generate_then_detect(psd, layout):
    """The stress workload's detection statement: 512 positions generated per sequence
    by the GPU sampler (V=256000, K=16, gamma=4, bf16), 128 sequences with the key and
    128 with a wrong key, then psd_detect and psd_detect_pvalue over all 256 x 512
    tokens against the oracle.  Target rows come from a position-indexed toy LM
    whose row at (sequence b, position t) is entry (131 b + 977 t) mod 512 of a fixed
    table, so memory stays bounded and a position revisited by a later block reads
    the same row.  Checked: the emitted text equals the plain keyed chain at sampled
    positions; every S_A, M and per-token A_t equals the oracle's; ln p_A matches
    the oracle's Poisson sum; the keyed half separates from the wrong-key half."""
    from gen_loop import generate
    w = workloads.WORKLOADS[5]
    n_pos, half = 512, w.B // 2
    key, wrong = w.key, w.key ^ 0x5DEECE66D
    gen = torch.Generator(device=DEV)
    gen.manual_seed(55 + layout)
    n_table = 512
    table = workloads.target_rows_fp32(w, n_table, gen, DEV)

    def rows_for(b0):
        def rows_at(idx):
            b = torch.arange(b0, b0 + idx.shape[0], device=DEV).view(-1, 1)
            return table[(131 * b + 977 * idx) % n_table]
        return rows_at

    texts = []
    for i, k in enumerate((key, wrong)):
        print(f"[gen] layout={layout} key {'right' if i == 0 else 'wrong'}: {half} x {n_pos} positions", flush=True)
        prompt = torch.randint(0, w.V, (half, w.m), generator=gen, device=DEV, dtype=torch.int64).to(torch.int32)
        params = psd.make_params(k, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout)
        ws = psd.new_workspace(params, half, w.gamma, DEV)
        status = torch.zeros((1,), dtype=torch.int32, device=DEV)

        def verify(prefix, start, tl, dl):
            out = psd.verify(params, ws, prefix, start, tl, dl, status=status)
            _sync()
            assert int(status[0]) == 0
            return _np(out["out_tokens"]), _np(out["out_len"])

        text, blocks = generate(verify, rows_for(i * half), prompt, n_pos, w.gamma, w.K, w.tau[0], gen,
                                w.torch_dtype)
        print(f"[gen]   {blocks} blocks", flush=True)
        texts.append(text)
    toks = torch.cat(texts, 0).contiguous()
    tk = _np(toks)
    # the emitted text is the plain keyed target chain (sampled positions, both halves)
    rng = np.random.default_rng(layout)
    picks = [(int(b), int(t)) for b, t in zip(rng.integers(0, w.B, 24), rng.integers(w.m, w.m + n_pos, 24))]
    tab = table.cpu().to(torch.bfloat16).float().numpy()

    def chain_token(bt):
        b, t = bt
        kk = key if b < half else wrong
        kappa = oracle.context_key(kk, t, [int(x) for x in tk[b, t - w.m:t]])
        return oracle.race(tab[(131 * b + 977 * t) % n_table], w.T_target, kappa, 0, w.K, layout)

    import concurrent.futures
    with concurrent.futures.ThreadPoolExecutor(WORKERS) as ex:
        races = list(ex.map(chain_token, picks))
    for (b, t), r in zip(picks, races):
        if int(tk[b, t]) != r["token"]:  # a near-tie may go either way
            s_gpu = oracle.token_score(tab[(131 * b + 977 * t) % n_table], w.T_target,
                                       oracle.context_key(key if b < half else wrong, t,
                                                          [int(x) for x in tk[b, t - w.m:t]]),
                                       0, w.K, int(tk[b, t]), layout)
            assert s_gpu - r["best"] < oracle.NEAR_TIE, (b, t, int(tk[b, t]), r)
    # detection of all 256 x 512 tokens with the key
    n0 = torch.full((w.B,), w.m, dtype=torch.int32, device=DEV)
    p = psd.make_params(key, w.V, w.K, w.m, dtype=w.torch_dtype, clocks=layout)
    score, count, per = psd.detect(p, toks, n0, per_token=True)
    log_p, anl = psd.detect_pvalue(score, count)
    _sync()
    score, count, per = _np(score), _np(count), _np(per)

    def ref_seq(i):
        return oracle.detect_sequence(key, w.m, w.K, w.V, tk[i], w.m, layout)

    with concurrent.futures.ThreadPoolExecutor(WORKERS) as ex:
        refs = list(ex.map(ref_seq, range(w.B)))
    for i, (S, M, ref_per) in enumerate(refs):
        assert count[i] == M == n_pos, (i, count[i], M)
        assert abs(score[i] - S) <= SCORE_TOL * abs(S), (i, score[i], S)
        ok = ~np.isnan(ref_per)
        assert np.allclose(per[i][ok], ref_per[ok], rtol=1e-5, atol=1e-6), i
    _check_pvalues(score, count, _np(log_p), _np(anl))
    z = (score - count) / np.sqrt(count)
    print(f"[detect] z keyed: min {z[:half].min():.1f} median {np.median(z[:half]):.1f}; "
          f"wrong key: max |z| {np.abs(z[half:]).max():.2f}", flush=True)
    assert np.all(z[:half] > 5.0), z[:half].min()
    assert np.all(np.abs(z[half:]) < 4.5), np.abs(z[half:]).max()
    assert np.all(_np(log_p)[:half] < math.log(1e-6)) and np.median(_np(log_p)[half:]) > math.log(0.05)
    # every score (Aaronson, U, Li Delta = 0.3, PL eps = 0.05), TPR@1%FPR on the keyed half
    # and the empirical FPR on the wrong-key half (App. "Drafter-substitution ablation")
    delta, eps = 0.3, 0.05
    sc4, ct4 = psd.detect_scores(p, toks, n0, delta, eps)
    lp4 = psd.detect_scores_pvalue(sc4, ct4, delta, eps)
    tpr = [int(psd.detection_rate(lp4[:half, q], 0.01)[0]) / half for q in range(4)]
    fpr = [int(psd.detection_rate(lp4[half:, q], 0.01)[0]) / half for q in range(4)]
    _sync()
    sc4, lp4 = _np(sc4), _np(lp4)
    assert np.allclose(sc4[:, 0], score, rtol=1e-12, atol=0.0)
    for i in list(range(0, w.B, 37)):
        c = oracle.detect_clocks(key, w.m, w.K, w.V, tk[i], w.m, layout)
        terms = oracle.score_terms(c[~np.isnan(c)], delta, eps)
        for q, kind in enumerate(("A", "U", "Li", "PL")):
            assert abs(sc4[i, q] - terms[kind].sum()) <= SCORE_TOL * abs(terms[kind].sum()) + 1e-12, (i, kind)
        for q, kind in enumerate(("U", "Li", "PL"), start=1):
            ref = oracle.chernoff_log_p(kind, float(sc4[i, q]), n_pos, delta, eps)
            assert abs(lp4[i, q] - ref) <= 1e-7 * abs(ref) + 1e-9, (i, kind, lp4[i, q], ref)
    print(f"[detect] TPR@1%FPR A/U/Li/PL {tpr}  empirical FPR {fpr}", flush=True)
    assert tpr[0] == 1.0 and all(t >= 0.9 for t in tpr)
    assert all(f <= 0.06 for f in fpr)


def _check_pvalues(score, count, log_p, anl):
    """ln p_A and ANLPPT_A against the oracle's Poisson-sum evaluation of the same (S_A, M).
    Tolerance: both sides form ln p from terms of size S + M |ln S| + ln M! to a few
    ulps (their difference cancels down to ln p), so 4e-15 of that size, plus 1e-11
    relative for the truncation of the term sums."""
    for S, M, lp, a in zip(score, count, log_p, anl):
        ref = oracle.gamma_tail_log_p(float(S), int(M))
        if math.isnan(ref):
            assert math.isnan(lp), (S, M, lp)
            continue
        if M > 0 and S > 0 and math.isfinite(S):
            tol = 4e-15 * (S + M * abs(math.log(S)) + math.lgamma(M + 1.0)) + 1e-14 + 1e-11 * abs(ref)
            assert abs(lp - ref) <= tol, (S, M, lp, ref)
        else:
            assert lp == ref, (S, M, lp, ref)
        if M > 0:
            assert a == pytest.approx(-lp / M, rel=1e-15, abs=0.0) or (math.isinf(lp) and math.isinf(a))
        else:
            assert math.isnan(a)


def test_detect_pvalue_grid(psd):
    """psd_detect_pvalue over counts from 1 to 10^6 and scores from far below to far
    above the null mean (the series and the Poisson form, both sides of S = M + 1),
    and the degenerate inputs: M = 0, S = 0, S = inf, NaN S, negative M.  301 sequences:
    two blocks of 256 threads, the second ragged."""
    cases = [(0, 5.0), (7, 0.0), (3, math.inf), (3, math.nan), (-1, 2.0), (1, 1e5), (2, 700.0)]
    for M in (1, 2, 3, 10, 100, 512, 5000, 100000, 10**6):
        for f, d in ((0.001, 0.0), (0.5, 0.0), (1.0, -1.0), (1.0, 0.0), (1.0, 1.0), (1.0, 1.5), (1.5, 0.0),
                     (3.0, 0.0), (20.0, 0.0), (1000.0, 0.0)):
            if f * M + d > 0:
                cases.append((M, f * M + d))
    rng = np.random.default_rng(11)
    while len(cases) < 301:
        M = int(rng.integers(1, 2000))
        cases.append((M, float(rng.gamma(M) * rng.uniform(0.5, 2.0))))
    count = torch.tensor([c[0] for c in cases], dtype=torch.int32, device=DEV)
    score = torch.tensor([c[1] for c in cases], dtype=torch.float64, device=DEV)
    log_p, anl = psd.detect_pvalue(score, count)
    # out_anlppt is nullable: the same ln p_A without it
    log_p2 = torch.empty_like(log_p)
    assert psd.lib().psd_detect_pvalue(len(cases), score.data_ptr(), count.data_ptr(), log_p2.data_ptr(), None,
                                       None) == psd.PSD_OK
    _sync()
    _check_pvalues(_np(score), _np(count), _np(log_p), _np(anl))
    assert np.array_equal(_np(log_p), _np(log_p2), equal_nan=True)
    # watermark-strength reading: S_A well above M gives a tiny p-value
    assert _np(log_p)[5] == pytest.approx(-1e5, rel=1e-14)


def _cpu_watermarked_text(key, w, n_seq, n_pos, seed, layout):
    """Text of the keyed target race at every position (what speculative decoding
    emits: the CPU pins show it equals the plain keyed chain), made by the oracle."""
    rng = np.random.default_rng(seed)
    P = w.m + n_pos
    rows = workloads.target_rows_fp32(w, n_seq * P, workloads._gen(seed, "cpu"), "cpu").view(n_seq, P, w.V)
    rows = rows.to(w.torch_dtype).float().numpy()
    toks = np.zeros((n_seq, P), np.int32)
    toks[:, :w.m] = rng.integers(0, w.V, (n_seq, w.m))
    for i in range(n_seq):
        for t in range(w.m, P):
            kappa = oracle.context_key(key, t, [int(x) for x in toks[i, t - w.m:t]])
            toks[i, t] = oracle.race(rows[i, t], w.T_target, kappa, 0, w.K, layout)["token"]
    return toks


@pytest.mark.parametrize("layout", LAYOUTS)
def test_detect_parity_cpu_text(psd, layout):
    """psd_detect on watermarked text (made on the CPU with the key), text made with
    another key and uniform text, against the oracle; out-of-range tokens and an
    empty scored range included."""
    w = workloads.custom(5000, 4, 4, 1, dtype="bf16", m=3, sigma=3.0, alpha=1.2)
    key, wrong = 0x1111222233334444, 0x5555666677778888
    wm = _cpu_watermarked_text(key, w, 4, 60, 1, layout)
    nw = _cpu_watermarked_text(wrong, w, 3, 60, 2, layout)
    un = workloads.uniform_tokens(2, 63, w.V, seed=3).numpy()
    tk = np.concatenate([wm, nw, un], 0).astype(np.int32)
    tk[0, 10] = 99999   # out of range: not scored
    tk[5, 20] = -4      # negative: not scored
    n0 = np.full(tk.shape[0], w.m, np.int32)
    n0[1] = 200         # nothing scored
    p = psd.make_params(key, w.V, w.K, w.m, dtype=torch.bfloat16, clocks=layout)
    score, count, per = psd.detect(p, torch.from_numpy(tk).to(DEV), torch.from_numpy(n0).to(DEV), per_token=True)
    _sync()
    score, count, per = _np(score), _np(count), _np(per)
    for i in range(tk.shape[0]):
        S, M, ref_per = oracle.detect_sequence(key, w.m, w.K, w.V, tk[i], int(n0[i]), layout)
        assert count[i] == M
        assert abs(score[i] - S) <= SCORE_TOL * abs(S) + 1e-12, (i, score[i], S)
        ok = ~np.isnan(ref_per)
        assert np.array_equal(np.isnan(per[i]), ~ok)
        assert np.allclose(per[i][ok], ref_per[ok], rtol=1e-5, atol=1e-6)
    z = (score - count) / np.sqrt(np.maximum(count, 1))
    assert np.all(z[[0, 2, 3]] > 3.0), z
    assert np.all(np.abs(z[4:]) < 4.5), z


@pytest.mark.parametrize("layout", LAYOUTS)
def test_detect_exact_minimum_many_tokens(psd, layout):
    """The detector finds each token's smallest clock over K = 16 slots from float
    clocks and rebuilds only the near-minimum slots exactly: over 64 x 512 scored
    tokens (a few dozen near-ties expected) every per-token A_t must equal the
    oracle's, rounded to float32, within 2 ulp -- far tighter than the error a
    wrong slot would cause -- and every score within 1e-12 relative."""
    w5 = workloads.WORKLOADS[5]
    n_seq, n_pos = 64, 512
    toks = workloads.uniform_tokens(n_seq, w5.m + n_pos, w5.V, seed=77)
    n0 = torch.full((n_seq,), w5.m, dtype=torch.int32)
    p = psd.make_params(w5.key, w5.V, w5.K, w5.m, dtype=w5.torch_dtype, clocks=layout)
    score, count, per = psd.detect(p, toks.to(DEV), n0.to(DEV), per_token=True)
    _sync()
    score, count, per, tk = _np(score), _np(count), _np(per), _np(toks)
    for i in range(n_seq):
        S, M, ref_per = oracle.detect_sequence(w5.key, w5.m, w5.K, w5.V, tk[i], w5.m, layout)
        assert count[i] == M == n_pos
        assert abs(score[i] - S) <= 1e-12 * abs(S), (i, score[i], S)
        ref32 = ref_per[w5.m:].astype(np.float32)
        got = per[i][w5.m:]
        assert np.all(np.abs(got - ref32) <= 2 * np.spacing(np.abs(ref32))), (i, np.max(np.abs(got - ref32)))
