"""Seeded synthetic inputs shaped like the paper's decoding workloads.

This module holds no part of the sampler's arithmetic: it only draws logits,
prompts and keys.  Both the HIP path and the CPU oracle receive exactly the bits
it produces (the oracle gets a host copy), so it is the one module they share.

Logit recipe (a stand-in for next-token logits of Llama-2/3- and Qwen-sized
vocabularies; the paper's models and datasets are not available):

* per target row (sequence b, depth s): a seeded random permutation pi of the
  ranks 1..V and ``z_v = sigma * N(0,1) - alpha * ln pi(v)`` (Zipf-like head with
  Gaussian jitter);
* draft row (b, k, s) = ``z + tau_b * N(0,1)``, drawn independently per draft k
  and depth s (a drafter that disagrees with the target by ``tau``);
* generated in float32, then rounded to bfloat16 (round-to-nearest-even) when
  the workload is bf16; temperatures are NOT baked in (the kernels apply them);
* prompt = ``m`` uniform tokens per sequence, ``start_pos = m``;
* key = SplitMix64(20261202 * 100 + config id).

The target row depends only on (b, absolute position), as in a position-indexed
toy language model, so all K draft paths of a block share the target row of a
depth.
"""
from __future__ import annotations

import dataclasses

import torch

MASK64 = (1 << 64) - 1


def splitmix64(x: int) -> int:
    """SplitMix64 output for state x (Steele, Lea, Flood, OOPSLA 2014)."""
    z = (x + 0x9E3779B97F4A7C15) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic decoding configuration."""
    cid: int
    name: str
    V: int            # vocabulary size
    K: int            # number of drafts (list size)
    gamma: int        # draft length (lookahead)
    B: int            # sequences per block
    dtype: str        # "fp32" | "bf16"
    sigma: float
    alpha: float
    tau: tuple        # draft noise per half of the batch (tau_first_half, tau_second_half)
    T_target: float
    T_draft: float
    m: int            # context window of the keyed source

    @property
    def key(self) -> int:
        return splitmix64(20261202 * 100 + self.cid)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def rows(self):
        """(draft rows, target rows) of one verify call with shared target rows."""
        return self.B * self.K * self.gamma, self.B * (self.gamma + 1)

    def algorithmic_bytes(self) -> int:
        d, t = self.rows()
        return (d + t) * self.V * self.elem_bytes

    def with_batch(self, B: int) -> "Workload":
        return dataclasses.replace(self, B=B)


WORKLOADS = {
    1: Workload(1, "tiny V=1024 K=2 gamma=4 B=1 fp32", 1024, 2, 4, 1, "fp32", 2.0, 1.1, (0.8, 0.8), 1.0, 1.0, 4),
    2: Workload(2, "Llama-2 vocab V=32000 K=4 gamma=5 B=16 bf16", 32000, 4, 5, 16, "bf16", 3.0, 1.1, (0.5, 0.5),
                1.0, 1.0, 4),
    3: Workload(3, "Llama-3 vocab V=128256 K=4 gamma=4 B=64 bf16", 128256, 4, 4, 64, "bf16", 3.0, 1.2, (0.3, 1.0),
                0.7, 0.7, 4),
    4: Workload(4, "Qwen vocab V=151936 K=8 gamma=8 B=128 fp32", 151936, 8, 8, 128, "fp32", 2.5, 1.0, (0.6, 0.6),
                1.0, 1.0, 8),
    5: Workload(5, "stress V=256000 K=16 gamma=4 B=256 bf16", 256000, 16, 4, 256, "bf16", 3.0, 1.2, (0.8, 0.8),
                1.0, 1.0, 4),
}


def custom(V, K, gamma, B, dtype="fp32", sigma=2.0, alpha=1.1, tau=0.8, T_target=1.0, T_draft=1.0, m=4, cid=0):
    """A workload with explicit sizes (edge cases, parity sweeps)."""
    t = tau if isinstance(tau, tuple) else (tau, tau)
    return Workload(cid, "custom", V, K, gamma, B, dtype, sigma, alpha, t, T_target, T_draft, m)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed & 0x7FFFFFFFFFFFFFFF)
    return g


def target_rows_fp32(w: Workload, n_rows: int, gen: torch.Generator, device) -> torch.Tensor:
    """n_rows Zipf+Gaussian rows, float32 [n_rows, V]."""
    u = torch.rand(n_rows, w.V, generator=gen, device=device)
    ranks = torch.argsort(u, dim=1).to(torch.float32) + 1.0
    z = w.sigma * torch.randn(n_rows, w.V, generator=gen, device=device) - w.alpha * torch.log(ranks)
    return z


def make_block(w: Workload, seed: int, device="cpu", target_rows: int = 1, with_drafts: bool = True,
               row_chunk: int = 64) -> dict:
    """Inputs of one verify call.

    Returns target_logits [B][gamma+1][V] (or [B][K][gamma+1][V] when
    target_rows == K, each path getting its own jittered copy), draft_logits
    [B][K][gamma][V] (None unless with_drafts), prefix_tokens int32 [B][m],
    start_pos int64 [B] and the key.  Rows are drawn in chunks of row_chunk
    target rows to bound temporary memory."""
    gen = _gen(seed, device)
    B, K, G1, V = w.B, w.K, w.gamma + 1, w.V
    tdt = w.torch_dtype
    tshape = (B, G1, V) if target_rows == 1 else (B, K, G1, V)
    target = torch.empty(tshape, dtype=tdt, device=device)
    draft = torch.empty((B, K, w.gamma, V), dtype=tdt, device=device) if with_drafts else None
    for b0 in range(0, B, max(1, row_chunk // G1)):
        b1 = min(B, b0 + max(1, row_chunk // G1))
        z = target_rows_fp32(w, (b1 - b0) * G1, gen, device).view(b1 - b0, G1, V)
        if target_rows == 1:
            target[b0:b1] = z.to(tdt)
        else:
            for k in range(K):
                jit = 0.05 * torch.randn(z.shape, generator=gen, device=device)
                target[b0:b1, k] = (z + jit).to(tdt)
        if with_drafts:
            for bb in range(b0, b1):
                tau = w.tau[0] if bb < B // 2 or B == 1 else w.tau[1]
                noise = torch.randn((K, w.gamma, V), generator=gen, device=device)
                draft[bb] = (z[bb - b0, : w.gamma].unsqueeze(0) + tau * noise).to(tdt)
    prefix = torch.randint(0, V, (B, w.m), generator=gen, device=device, dtype=torch.int64).to(torch.int32)
    start = torch.full((B,), w.m, dtype=torch.int64, device=device)
    return {"target_logits": target, "draft_logits": draft, "prefix_tokens": prefix, "start_pos": start,
            "key": w.key, "workload": w}


def as_f32_numpy(t: torch.Tensor):
    """Exact float32 host copy of a logits tensor (bf16 widens exactly)."""
    return t.detach().to("cpu").to(torch.float32).numpy()


def uniform_tokens(n_seq: int, seq_len: int, V: int, seed: int, device="cpu") -> torch.Tensor:
    """Token matrix int32 [n_seq][seq_len] with iid uniform tokens (unwatermarked text)."""
    gen = _gen(seed, device)
    return torch.randint(0, V, (n_seq, seq_len), generator=gen, device=device, dtype=torch.int64).to(torch.int32)


def zipf_probs(V: int, sigma: float, alpha: float, T: float, seed: int):
    """One Zipf+Gaussian row: (float32 logits, float64 softmax of logits/T) for statistics tests."""
    w = custom(V, 1, 1, 1, sigma=sigma, alpha=alpha)
    logits = target_rows_fp32(w, 1, _gen(seed, "cpu"), "cpu")[0].numpy().astype("float32")
    x = logits.astype("float64") / float(torch.tensor(T, dtype=torch.float32))
    p = torch.softmax(torch.from_numpy(x), 0).numpy()
    return logits, p


def mib(n_bytes: int) -> float:
    return n_bytes / float(1 << 20)


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


__all__ = ["Workload", "WORKLOADS", "custom", "make_block", "as_f32_numpy", "uniform_tokens", "splitmix64",
           "zipf_probs", "mib", "ceil_div"]
