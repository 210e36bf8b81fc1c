"""Multi-block speculative generation over a position-indexed toy LM.

The target row of sequence b at absolute position t is rows[b, t]; each block
verifies gamma drafts and appends the emitted tokens.  `verify` is pluggable (the
HIP library, or the CPU oracle), so the loop's index arithmetic is exercised on
the CPU too.  Every index is checked on the host before it is used.
"""
import numpy as np
import torch


def table_positions(m: int, n_pos: int, gamma: int) -> int:
    """Rows per sequence: a block starting at position t (t <= m + n_pos - 1 for a
    sequence still generating) reads positions t .. t + gamma."""
    return m + n_pos + gamma


def block_starts(length: torch.Tensor, m: int, n_pos: int) -> torch.Tensor:
    """Start position of the next block; finished sequences are clamped to the last
    valid start (their result is discarded)."""
    return torch.clamp(length, max=m + n_pos - 1)


def generate(verify, rows, prompt, n_pos, gamma, K, noise, gen, dtype):
    """rows: float32 [B][table_positions][V]; prompt: int32 [B][m].
    verify(prefix, start_pos, target_logits, draft_logits) -> (out_tokens, out_len) host arrays."""
    B, P, V = rows.shape
    m = prompt.shape[1]
    assert P == table_positions(m, n_pos, gamma), (P, m, n_pos, gamma)
    dev = rows.device
    length = torch.full((B,), m, dtype=torch.int64, device=dev)
    buf = torch.full((B, m + n_pos + gamma + 1), -1, dtype=torch.int32, device=dev)
    buf[:, :m] = prompt
    blocks = 0
    while int(length.min()) < m + n_pos:
        start = block_starts(length, m, n_pos)
        idx = start.view(B, 1) + torch.arange(gamma + 1, device=dev).view(1, gamma + 1)
        assert int(idx.min()) >= 0 and int(idx.max()) < P, (int(idx.max()), P)
        pidx = start.view(B, 1) - m + torch.arange(m, device=dev).view(1, m)
        assert m == 0 or (int(pidx.min()) >= 0 and int(pidx.max()) < buf.shape[1])
        tl = torch.gather(rows, 1, idx.view(B, gamma + 1, 1).expand(B, gamma + 1, V)).to(dtype).contiguous()
        dl = (tl[:, None, :gamma].float() + noise * torch.randn((B, K, gamma, V), generator=gen, device=dev)).to(dtype)
        prefix = torch.gather(buf, 1, pidx).contiguous() if m else buf[:, :0].contiguous()
        out_tokens, out_len = verify(prefix, start, tl, dl)
        out_len = np.asarray(out_len)
        assert np.all((out_len >= 1) & (out_len <= gamma + 1)), out_len
        for b in range(B):
            L0 = int(length[b])
            if L0 >= m + n_pos:
                continue
            n = int(out_len[b])
            assert L0 + n <= buf.shape[1]
            buf[b, L0:L0 + n] = torch.as_tensor(np.asarray(out_tokens[b][:n]), dtype=torch.int32, device=dev)
            length[b] = L0 + n
        blocks += 1
    return buf[:, :m + n_pos].contiguous(), blocks
