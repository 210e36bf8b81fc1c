"""Thin ctypes binding of libpsd (the C ABI in include/psd.h).

Argument marshalling only: every step of the sampler runs in the HIP kernels of
libpsd.  PyTorch provides device memory and the current stream.  If the built
library is missing, importing this module raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libpsd.so")

PSD_OK, PSD_E_ARG, PSD_E_UNSUPPORTED, PSD_E_HIP, PSD_E_WORKSPACE = 0, -1, -2, -3, -4
PSD_F32, PSD_BF16 = 0, 1
PSD_MODE_HET, PSD_MODE_MPFR = 0, 1
PSD_CLOCKS_TREE, PSD_CLOCKS_FLAT = 0, 1
ERR_SPIN, ERR_CAND = 1, 2


class PsdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"psd status {status}: {msg}")
        self.status = status


class Params(ctypes.Structure):
    _fields_ = [
        ("key", ctypes.c_uint64),
        ("vocab", ctypes.c_int32),
        ("num_drafts", ctypes.c_int32),
        ("ctx_window", ctypes.c_int32),
        ("temp_target", ctypes.c_float),
        ("temp_draft", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("mode", ctypes.c_int32),
        ("clocks", ctypes.c_int32),
        ("top_k", ctypes.c_int32),
        ("top_p", ctypes.c_float),
    ]


class Block(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("gamma", ctypes.c_int32),
        ("prefix_tokens", ctypes.c_void_p),
        ("start_pos", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("status", ctypes.c_void_p),
    ]


class ToyLM(ctypes.Structure):
    """psd_toy_lm: the synthetic position-indexed model of psd_toy_logits / psd_generate."""
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("draft_seed", ctypes.c_uint64),
        ("sigma", ctypes.c_float),
        ("alpha", ctypes.c_float),
        ("tau", ctypes.c_float * 2),
        ("tau_split", ctypes.c_int32),
    ]


def make_toy_lm(seed: int, draft_seed: int, sigma: float, alpha: float, tau=(1.0, 1.0), tau_split: int = 0) -> ToyLM:
    lm = ToyLM(seed & 0xFFFFFFFFFFFFFFFF, draft_seed & 0xFFFFFFFFFFFFFFFF, sigma, alpha)
    lm.tau[0], lm.tau[1] = float(tau[0]), float(tau[1])
    lm.tau_split = int(tau_split)
    return lm


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(Params)
    Bp = ctypes.POINTER(Block)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sigs = {
        "psd_abi_version": ([], i32),
        "psd_last_error": ([], ctypes.c_char_p),
        "psd_workspace_bytes": ([P, i32, i32], sz),
        "psd_workspace_clear": ([vp, sz, vp], i32),
        "psd_workspace_errors": ([vp, vp, ctypes.POINTER(ctypes.c_uint32)], i32),
        "psd_draft": ([P, Bp, i32, i32, vp, vp, vp, vp], i32),
        "psd_verify": ([P, Bp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp], i32),
        "psd_verify_static": ([P, Bp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp], i32),
        "psd_detect": ([P, i32, i32, vp, vp, vp, vp, vp, vp], i32),
        "psd_detect_pvalue": ([i32, vp, vp, vp, vp, vp], i32),
        "psd_philox": ([i32, vp, vp, vp, vp], i32),
        "psd_context_keys": ([P, i32, vp, vp, vp, vp], i32),
        "psd_clock_values": ([P, i32, vp, vp, vp, vp, vp], i32),
        "psd_set_spin_limit": ([ctypes.c_uint32], None),
        "psd_detect_scores": ([P, vp, i32, i32, i32, vp, vp, vp, vp, vp], i32),
        "psd_detect_scores_pvalue": ([vp, i32, vp, vp, vp, vp], i32),
        "psd_detection_rate": ([i32, vp, i32, ctypes.c_double, vp, vp], i32),
        "psd_advance": ([P, i32, i32, ctypes.c_int64, vp, vp, vp, ctypes.c_int64, vp, vp, vp, vp, vp], i32),
        "psd_toy_logits": ([P, ctypes.POINTER(ToyLM), i32, i32, vp, vp, vp, vp], i32),
        "psd_generate_workspace_bytes": ([P, i32, i32], sz),
        "psd_generate": ([P, ctypes.POINTER(ToyLM), i32, i32, i32, vp, ctypes.c_int64, vp, sz, i32, i32,
                          ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_uint32), vp], i32),
    }
    for name, (args, res) in sigs.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    return lib


_lib = _load()
EXPORTS = ("psd_abi_version", "psd_last_error", "psd_workspace_bytes", "psd_workspace_clear",
           "psd_workspace_errors", "psd_draft", "psd_verify", "psd_verify_static", "psd_detect", "psd_detect_pvalue", "psd_philox",
           "psd_context_keys", "psd_clock_values", "psd_set_spin_limit", "psd_detect_scores",
           "psd_detect_scores_pvalue", "psd_detection_rate", "psd_advance", "psd_toy_logits",
           "psd_generate_workspace_bytes", "psd_generate")


def lib():
    return _lib


def _check(status: int):
    if status != PSD_OK:
        raise PsdError(status, (_lib.psd_last_error() or b"").decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def make_params(key: int, vocab: int, num_drafts: int, ctx_window: int, temp_target: float = 1.0,
                temp_draft: float = 1.0, dtype=torch.bfloat16, mode: int = PSD_MODE_HET,
                clocks: int = PSD_CLOCKS_TREE, top_k: int = 0, top_p: float = 1.0) -> Params:
    dt = dtype if isinstance(dtype, int) else (PSD_BF16 if dtype == torch.bfloat16 else PSD_F32)
    return Params(key & 0xFFFFFFFFFFFFFFFF, vocab, num_drafts, ctx_window, temp_target, temp_draft, dt, mode,
                  clocks, top_k, top_p)


def workspace_bytes(params: Params, batch: int, gamma: int) -> int:
    return int(_lib.psd_workspace_bytes(ctypes.byref(params), batch, gamma))


def new_workspace(params: Params, batch: int, gamma: int, device="cuda") -> torch.Tensor:
    """Zero-filled device workspace (torch allocation, 256-byte aligned)."""
    n = workspace_bytes(params, batch, gamma)
    if n == 0:
        raise PsdError(PSD_E_ARG, "invalid parameters for workspace sizing")
    return torch.zeros(n, dtype=torch.uint8, device=device)


def workspace_clear(ws: torch.Tensor, stream=None):
    _check(_lib.psd_workspace_clear(_ptr(ws), ws.numel(), _stream(stream)))


def workspace_errors(ws: torch.Tensor, stream=None) -> int:
    out = ctypes.c_uint32(0)
    _check(_lib.psd_workspace_errors(_ptr(ws), _stream(stream), ctypes.byref(out)))
    return int(out.value)


def _block(batch, gamma, prefix, start_pos, ws, status=None):
    return Block(batch, gamma, prefix.data_ptr() if prefix is not None and prefix.numel() else None,
                 start_pos.data_ptr(), ws.data_ptr(), ws.numel(), None if status is None else status.data_ptr())


def set_spin_limit(polls: int = 0):
    """Test hook: polls of a bounded wait before it gives up (0 = default)."""
    _lib.psd_set_spin_limit(polls)


def draft(params: Params, ws, prefix_tokens, start_pos, gamma: int, s_begin: int, draft_logits, draft_tokens,
          draft_lse=None, stream=None, status=None):
    """psd_draft: draft depths [s_begin, s_begin + draft_logits.shape[2]).  status: optional
    int32 [1] device tensor receiving the call's error bits."""
    B = int(start_pos.shape[0])
    blk = _block(B, gamma, prefix_tokens, start_pos, ws, status)
    _check(_lib.psd_draft(ctypes.byref(params), ctypes.byref(blk), s_begin, int(draft_logits.shape[2]),
                          _ptr(draft_logits), _ptr(draft_tokens), _ptr(draft_lse), _stream(stream)))


def verify(params: Params, ws, prefix_tokens, start_pos, target_logits, draft_logits=None, draft_tokens=None,
           target_rows: int = 1, want_lse: bool = False, want_targets: bool = False, out=None, stream=None,
           status=None):
    """psd_verify; allocates the outputs it is not given.  Returns a dict of tensors.  status:
    optional int32 [1] device tensor receiving the call's error bits."""
    B = int(start_pos.shape[0])
    K = params.num_drafts
    gamma = int(target_logits.shape[-2]) - 1
    dev = target_logits.device
    o = {} if out is None else dict(out)
    if draft_tokens is None:
        draft_tokens = torch.empty((B, K, gamma), dtype=torch.int32, device=dev)
    o["draft_tokens"] = draft_tokens
    o.setdefault("out_tokens", torch.empty((B, gamma + 1), dtype=torch.int32, device=dev))
    o.setdefault("out_len", torch.empty((B,), dtype=torch.int32, device=dev))
    tshape = (B, gamma + 1) if target_rows == 1 else (B, K, gamma + 1)
    if want_lse:
        o.setdefault("target_lse", torch.empty(tshape, dtype=torch.float32, device=dev))
        if draft_logits is not None:
            o.setdefault("draft_lse", torch.empty((B, K, gamma), dtype=torch.float32, device=dev))
    if want_targets:
        o.setdefault("target_tokens", torch.empty(tshape, dtype=torch.int32, device=dev))
    blk = _block(B, gamma, prefix_tokens, start_pos, ws, status)
    _check(_lib.psd_verify(ctypes.byref(params), ctypes.byref(blk), target_rows, _ptr(target_logits),
                           _ptr(draft_logits), _ptr(draft_tokens), _ptr(o["out_tokens"]), _ptr(o["out_len"]),
                           _ptr(o.get("target_lse")), _ptr(o.get("draft_lse")), _ptr(o.get("target_tokens")),
                           _stream(stream)))
    return o


def verify_static(params: Params, prefix_tokens, start_pos, target_logits, draft_logits=None, draft_tokens=None,
                  target_rows: int = 1, out=None, status=None, stream=None):
    """psd_verify_static (the library's fixed scratch, no workspace).  Outputs come
    from `out` (a dict of tensors: draft_tokens, out_tokens, out_len and optionally
    target_lse, draft_lse, target_tokens) or are allocated here by torch when missing."""
    B = int(start_pos.shape[0])
    K = params.num_drafts
    gamma = int(target_logits.shape[-2]) - 1
    dev = target_logits.device
    o = {} if out is None else dict(out)
    if draft_tokens is None:
        draft_tokens = o.get("draft_tokens")
    if draft_tokens is None:
        draft_tokens = torch.empty((B, K, gamma), dtype=torch.int32, device=dev)
    o["draft_tokens"] = draft_tokens
    o.setdefault("out_tokens", torch.empty((B, gamma + 1), dtype=torch.int32, device=dev))
    o.setdefault("out_len", torch.empty((B,), dtype=torch.int32, device=dev))
    blk = Block(B, gamma, prefix_tokens.data_ptr() if prefix_tokens is not None and prefix_tokens.numel() else None,
                start_pos.data_ptr(), None, 0, None if status is None else status.data_ptr())
    _check(_lib.psd_verify_static(ctypes.byref(params), ctypes.byref(blk), target_rows, _ptr(target_logits),
                                  _ptr(draft_logits), _ptr(draft_tokens), _ptr(o["out_tokens"]), _ptr(o["out_len"]),
                                  _ptr(o.get("target_lse")), _ptr(o.get("draft_lse")), _ptr(o.get("target_tokens")),
                                  _stream(stream)))
    return o


def detect(params: Params, tokens, n0, per_token: bool = False, stream=None):
    """psd_detect -> (score f64 [n_seq], count i32 [n_seq], per-token f32 or None)."""
    n_seq, seq_len = int(tokens.shape[0]), int(tokens.shape[1])
    dev = tokens.device
    score = torch.empty((n_seq,), dtype=torch.float64, device=dev)
    count = torch.empty((n_seq,), dtype=torch.int32, device=dev)
    per = torch.empty((n_seq, seq_len), dtype=torch.float32, device=dev) if per_token else None
    _check(_lib.psd_detect(ctypes.byref(params), n_seq, seq_len, _ptr(tokens), _ptr(n0), _ptr(score), _ptr(count),
                           _ptr(per), _stream(stream)))
    return score, count, per


class ScoreParams(ctypes.Structure):
    _fields_ = [("li_delta", ctypes.c_double), ("pl_eps", ctypes.c_double)]


def detect_scores(params: Params, tokens, n0, li_delta: float, pl_eps: float, seq_len: int = None, stream=None):
    """psd_detect_scores -> (scores f64 [n_seq][4] = S_A, S_U, S_Li, S_PL; count i32 [n_seq]).
    seq_len < tokens.shape[1] scores that prefix of every row."""
    n_seq, stride = int(tokens.shape[0]), int(tokens.shape[1])
    seq_len = stride if seq_len is None else int(seq_len)
    sp = ScoreParams(li_delta, pl_eps)
    scores = torch.empty((n_seq, 4), dtype=torch.float64, device=tokens.device)
    count = torch.empty((n_seq,), dtype=torch.int32, device=tokens.device)
    _check(_lib.psd_detect_scores(ctypes.byref(params), ctypes.byref(sp), n_seq, seq_len, stride, _ptr(tokens),
                                  _ptr(n0), _ptr(scores), _ptr(count), _stream(stream)))
    return scores, count


def detect_scores_pvalue(scores, count, li_delta: float, pl_eps: float, stream=None):
    """psd_detect_scores_pvalue -> ln p f64 [n_seq][4] (A exact; U, Li, PL Chernoff bounds)."""
    n = int(scores.shape[0])
    sp = ScoreParams(li_delta, pl_eps)
    out = torch.empty((n, 4), dtype=torch.float64, device=scores.device)
    _check(_lib.psd_detect_scores_pvalue(ctypes.byref(sp), n, _ptr(scores), _ptr(count), _ptr(out),
                                         _stream(stream)))
    return out


def detection_rate(log_p, alpha: float, stream=None):
    """psd_detection_rate over a column of log p-values ([n] or [n][c] with one column
    selected by the caller's view) -> int32 [1] count with ln p <= ln alpha."""
    n = int(log_p.shape[0])
    stride = int(log_p.stride(0))
    out = torch.empty((1,), dtype=torch.int32, device=log_p.device)
    _check(_lib.psd_detection_rate(n, _ptr(log_p), stride, alpha, _ptr(out), _stream(stream)))
    return out


def detect_pvalue(score, count, stream=None):
    """psd_detect_pvalue -> (ln p_A f64 [n_seq], ANLPPT_A f64 [n_seq]) of S_A ~ Gamma(M, 1) under the null."""
    n = int(score.shape[0])
    log_p = torch.empty((n,), dtype=torch.float64, device=score.device)
    anl = torch.empty((n,), dtype=torch.float64, device=score.device)
    _check(_lib.psd_detect_pvalue(n, _ptr(score), _ptr(count), _ptr(log_p), _ptr(anl), _stream(stream)))
    return log_p, anl


def philox(ctr, key, stream=None):
    n = int(ctr.shape[0])
    out = torch.empty((n, 4), dtype=torch.int32, device=ctr.device)
    _check(_lib.psd_philox(n, _ptr(ctr), _ptr(key), _ptr(out), _stream(stream)))
    return out


def context_keys(params: Params, t, windows, stream=None):
    n = int(t.shape[0])
    out = torch.empty((n, 2), dtype=torch.int32, device=t.device)
    _check(_lib.psd_context_keys(ctypes.byref(params), n, _ptr(t), _ptr(windows) if windows is not None and
                                 windows.numel() else None, _ptr(out), _stream(stream)))
    return out


def clock_values(params: Params, kappa, slot, token, stream=None):
    n = int(slot.shape[0])
    out = torch.empty((n,), dtype=torch.float64, device=slot.device)
    _check(_lib.psd_clock_values(ctypes.byref(params), n, _ptr(kappa), _ptr(slot), _ptr(token), _ptr(out),
                                 _stream(stream)))
    return out


# ---------------------------------------------------------------- multi-block generation

def advance(params: Params, gamma: int, max_len: int, text, length, prefix, start_pos, n_active, out_tokens=None,
            out_len=None, stream=None):
    """psd_advance: commit one block (out_len None: set up the first block from the prompts)."""
    B = int(text.shape[0])
    _check(_lib.psd_advance(ctypes.byref(params), B, gamma, int(max_len), _ptr(out_tokens), _ptr(out_len),
                            _ptr(text), int(text.stride(0)), _ptr(length),
                            _ptr(prefix) if prefix is not None and prefix.numel() else None, _ptr(start_pos),
                            _ptr(n_active), _stream(stream)))


def toy_logits(params: Params, lm: ToyLM, gamma: int, start_pos, drafts: bool = True, stream=None):
    """psd_toy_logits -> (target rows [B][gamma+1][V], draft rows [B][K][gamma][V] or None)."""
    B, V, K = int(start_pos.shape[0]), params.vocab, params.num_drafts
    dt = torch.bfloat16 if params.dtype == PSD_BF16 else torch.float32
    tl = torch.empty((B, gamma + 1, V), dtype=dt, device=start_pos.device)
    dl = torch.empty((B, K, gamma, V), dtype=dt, device=start_pos.device) if drafts else None
    _check(_lib.psd_toy_logits(ctypes.byref(params), ctypes.byref(lm), B, gamma, _ptr(start_pos), _ptr(tl), _ptr(dl),
                               _stream(stream)))
    return tl, dl


def generate_workspace_bytes(params: Params, batch: int, gamma: int) -> int:
    return int(_lib.psd_generate_workspace_bytes(ctypes.byref(params), batch, gamma))


def generate(params: Params, lm: ToyLM, prompts, n_pos: int, gamma: int, check_every: int = 16,
             use_graph: bool = False, ws=None, stream=None):
    """psd_generate: n_pos tokens after each prompt (int32 [B][m], m = ctx_window) on the device.
    Returns (text int32 [B][m + n_pos], blocks, error bits)."""
    B, m = int(prompts.shape[0]), params.ctx_window
    assert prompts.shape[1] == m
    text = torch.full((B, m + n_pos), -1, dtype=torch.int32, device=prompts.device)
    text[:, :m] = prompts
    if ws is None:
        n = generate_workspace_bytes(params, B, gamma)
        if n == 0:
            raise PsdError(PSD_E_ARG, "invalid parameters for generation")
        ws = torch.empty(n, dtype=torch.uint8, device=prompts.device)
    blocks = ctypes.c_int32(0)
    bits = ctypes.c_uint32(0)
    _check(_lib.psd_generate(ctypes.byref(params), ctypes.byref(lm), B, gamma, n_pos, _ptr(text), int(text.stride(0)),
                             _ptr(ws), ws.numel(), check_every, 1 if use_graph else 0, ctypes.byref(blocks),
                             ctypes.byref(bits), _stream(stream)))
    return text, int(blocks.value), int(bits.value)

