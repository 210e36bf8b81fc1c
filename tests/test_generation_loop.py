"""CPU checks of the multi-block generation loop used by the GPU detection test.

The loop's first GPU runs faulted in torch.gather: blocks kept being built for
sequences that had already finished, at positions length .. length + gamma with
length up to m + n_pos + gamma, beyond a table of m + n_pos + gamma + 2 rows.
These tests show that index range and run the fixed loop with the oracle as the
sampler (host-side index checks on every block)."""
import numpy as np
import torch

import oracle
import workloads
from gen_loop import block_starts, generate, table_positions


def test_old_table_was_too_small():
    m, n_pos, gamma = 3, 60, 4
    old_rows = n_pos + m + gamma + 2
    worst_length = (m + n_pos - 1) + (gamma + 1)   # an unfinished sequence accepting a full block
    assert worst_length + gamma >= old_rows        # the old loop read past the table
    start = block_starts(torch.tensor([worst_length]), m, n_pos)
    assert int(start) + gamma < table_positions(m, n_pos, gamma)


def test_generation_loop_indices():
    w = workloads.custom(64, 3, 3, 3, m=2, sigma=2.0, alpha=1.0)
    n_pos = 25
    gen = torch.Generator().manual_seed(5)
    P = table_positions(w.m, n_pos, w.gamma)
    rows = workloads.target_rows_fp32(w, w.B * P, gen, "cpu").view(w.B, P, w.V)
    prompt = torch.randint(0, w.V, (w.B, w.m), generator=gen, dtype=torch.int64).to(torch.int32)
    key = 0xFEED

    def verify(prefix, start, tl, dl):
        res = oracle.verify_block(key=key, K=w.K, gamma=w.gamma, m=w.m, T_target=1.0, T_draft=1.0,
                                  prefix=prefix.numpy(), start_pos=start.numpy(), target_logits=tl.numpy(),
                                  draft_logits=dl.numpy())
        out = np.full((w.B, w.gamma + 1), -1, np.int32)
        for b in range(w.B):
            out[b, :res["out_len"][b]] = res["out_tokens"][b]
        return out, np.array([res["out_len"][b] for b in range(w.B)])

    text, blocks = generate(verify, rows, prompt, n_pos, w.gamma, w.K, 0.7, gen, torch.float32)
    assert text.shape == (w.B, w.m + n_pos)
    # the generated text equals the plain keyed chain of the toy LM
    for b in range(w.B):
        seq = [int(x) for x in prompt[b]]
        for t in range(w.m, w.m + n_pos):
            kappa = oracle.context_key(key, t, seq[-w.m:])
            seq.append(oracle.race(rows[b, t].numpy(), 1.0, kappa, 0, w.K)["token"])
        assert seq == [int(x) for x in text[b]]
    assert blocks < n_pos
