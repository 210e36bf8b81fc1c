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


# ---------------------------------------------------------------- position-indexed toy model

@dataclasses.dataclass(frozen=True)
class ToyModel:
    """A synthetic position-indexed language model for multi-block generation.

    The target row of sequence b at absolute position t is a fixed function of
    (seed, b, t) and drafter k's row adds noise keyed by (draft_seed, b, k, t), both
    built from integer hashes (SplitMix64 per row, Wellons' lowbias32 per element)
    and fp32 operations rounded one at a time, so that any implementation of the
    definition gives the same bits (the library's psd_toy_logits is another one):

    * R_T = sm(seed ^ sm(b << 32 | t)), R_P = sm(R_T ^ 0xD1B54A32D192ED03),
      R_D = sm(draft_seed ^ sm((k + 1) << 56 ^ b << 32 ^ t)), t mod 2^32;
    * rank r(v) = (a v + c) mod V, c = R_P mod V, a = (R_P >> 32) mod V (0 -> 1)
      moved up (V wraps to 1) to the first value coprime to V;
    * x = lo32(R) + v * 0x9E3779B9 mod 2^32; a word h gives the uniforms
      (lo16(h) + 1/2) / 2^16 and (hi16(h) + 1/2) / 2^16;
    * target: n = (4 uniforms of lowbias32(x), lowbias32(x ^ hi32(R_T)) summed - 2) * sqrt(3),
      q(r) = fp32(bits(fp32(1 + r)) - 0x3F800000) (2^23 x a piecewise-linear log2),
      w = fp32(-alpha ln 2 / 2^23), z = sigma * n + w * q(r(v));
    * draft: n' = (2 uniforms of lowbias32(x) summed - 1) * sqrt(6) (x from R_D),
      d = z + tau_b * n', tau_b = tau[0] for b < tau_split, else tau[1];
    * bf16 rows: round-to-nearest-even of the fp32 values.
    """
    seed: int
    draft_seed: int
    sigma: float
    alpha: float
    tau: tuple = (1.0, 1.0)
    tau_split: int = 0

    def _words(self, b: int, t: int):
        t32 = t & 0xFFFFFFFF
        rt = splitmix64(self.seed ^ splitmix64(((b << 32) | t32) & MASK64))
        rp = splitmix64(rt ^ 0xD1B54A32D192ED03)
        return rt, rp

    def target_row(self, b: int, t: int, V: int, bf16: bool = True, fp32_values: bool = False):
        """float32 [V]: the target row (bf16 values widened, unless bf16 is False)."""
        import numpy as np
        rt, rp = self._words(b, t)
        c = rp % V
        a = (rp >> 32) % V
        if a == 0:
            a = 1
        while _gcd(a, V) != 1:
            a = 1 if a + 1 == V else a + 1
        v = np.arange(V, dtype=np.uint32)
        x = np.uint32(rt & 0xFFFFFFFF) + v * np.uint32(0x9E3779B9)
        u4 = _two_uniforms(_lowbias32(x)) + _two_uniforms(_lowbias32(x ^ np.uint32(rt >> 32)))
        n = (u4 - np.float32(2.0)) * np.float32(1.7320508075688772)
        r = (np.arange(V, dtype=np.int64) * a + c) % V
        q = ((r + 1).astype(np.float32).view(np.uint32) - np.uint32(0x3F800000)).astype(np.int32).astype(np.float32)
        w = np.float32(-float(np.float32(self.alpha)) * 0.69314718055994531 * 2.0 ** -23)
        z = np.float32(self.sigma) * n + w * q
        return z if (fp32_values or not bf16) else _bf16_rne(z)

    def draft_row(self, b: int, k: int, t: int, V: int, bf16: bool = True):
        """float32 [V]: drafter k's row at (b, t)."""
        import numpy as np
        z = self.target_row(b, t, V, fp32_values=True)
        rd = splitmix64(self.draft_seed ^ splitmix64((((k + 1) << 56) ^ (b << 32) ^ (t & 0xFFFFFFFF)) & MASK64))
        x = np.uint32(rd & 0xFFFFFFFF) + np.arange(V, dtype=np.uint32) * np.uint32(0x9E3779B9)
        n2 = (_two_uniforms(_lowbias32(x)) - np.float32(1.0)) * np.float32(2.449489742783178)
        tau = np.float32(self.tau[0] if b < self.tau_split else self.tau[1])
        d = z + tau * n2
        return _bf16_rne(d) if bf16 else d


def _gcd(a: int, b: int) -> int:
    while b:
        a, b = b, a % b
    return a


def _lowbias32(x):
    import numpy as np
    x = x ^ (x >> np.uint32(16))
    x = x * np.uint32(0x7FEB352D)
    x = x ^ (x >> np.uint32(15))
    x = x * np.uint32(0x846CA68B)
    return x ^ (x >> np.uint32(16))


def _two_uniforms(h):
    import numpy as np
    return ((h & np.uint32(0xFFFF)).astype(np.float32) + (h >> np.uint32(16)).astype(np.float32)
            + np.float32(1.0)) * np.float32(2.0 ** -16)


def _bf16_rne(z):
    """float32 array -> the bf16 round-to-nearest-even values, as float32."""
    import numpy as np
    u = np.asarray(z, np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return (r << np.uint32(16)).view(np.float32)


def mib(n_bytes: int) -> float:
    return n_bytes / float(1 << 20)


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


__all__ = ["Workload", "WORKLOADS", "custom", "make_block", "as_f32_numpy", "uniform_tokens", "splitmix64",
           "zipf_probs", "mib", "ceil_div", "ToyModel"]
