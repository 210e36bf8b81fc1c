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
    """rows: float32 [B][table_positions][V], or a function of the absolute positions
    idx int64 [B][gamma+1] (each in [0, table_positions)) returning the target rows
    float32 [B][gamma+1][V] of those positions; prompt: int32 [B][m].
    verify(prefix, start_pos, target_logits, draft_logits) -> (out_tokens, out_len) host arrays."""
    B, m = prompt.shape
    P = table_positions(m, n_pos, gamma)
    if callable(rows):
        rows_at = rows
    else:
        assert rows.shape[0] == B and rows.shape[1] == P, (rows.shape, P)
        V = rows.shape[2]
        rows_at = lambda idx: torch.gather(rows, 1, idx.view(B, gamma + 1, 1).expand(B, gamma + 1, V))
    dev = prompt.device
    # the text and the lengths live on the host: every index is checked there
    length = np.full(B, m, dtype=np.int64)
    buf = np.full((B, m + n_pos + gamma + 1), -1, dtype=np.int32)
    buf[:, :m] = prompt.cpu().numpy()
    blocks = 0
    while int(length.min()) < m + n_pos:
        start = np.minimum(length, m + n_pos - 1)  # block_starts: finished sequences clamped
        idx = start[:, None] + np.arange(gamma + 1)[None, :]
        assert int(idx.min()) >= 0 and int(idx.max()) < P, (int(idx.max()), P)
        pidx = start[:, None] - m + np.arange(m)[None, :]
        assert m == 0 or (int(pidx.min()) >= 0 and int(pidx.max()) < buf.shape[1])
        tl = rows_at(torch.from_numpy(idx).to(dev)).to(dtype).contiguous()
        V = tl.shape[-1]
        dl = (tl[:, None, :gamma].float() + noise * torch.randn((B, K, gamma, V), generator=gen, device=dev)).to(dtype)
        prefix = torch.from_numpy(np.ascontiguousarray(np.take_along_axis(buf, pidx, 1) if m else buf[:, :0])).to(dev)
        out_tokens, out_len = verify(prefix, torch.from_numpy(start).to(dev), tl, dl)
        out_tokens, out_len = np.asarray(out_tokens), np.asarray(out_len)
        assert np.all((out_len >= 1) & (out_len <= gamma + 1)), out_len
        for b in range(B):
            L0 = int(length[b])
            if L0 >= m + n_pos:
                continue
            n = int(out_len[b])
            assert L0 + n <= buf.shape[1]
            buf[b, L0:L0 + n] = out_tokens[b][:n]
            length[b] = L0 + n
        blocks += 1
    return torch.from_numpy(np.ascontiguousarray(buf[:, :m + n_pos])).to(dev), blocks
