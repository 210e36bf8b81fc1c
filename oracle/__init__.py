"""Plain CPU oracle of the keyed Poisson race (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may import this package.  It shares no code with the HIP library
(``paper_2609_21858_amd``) and never imports it; the two meet only through the
seeded input generator in ``workloads.py``.

The arithmetic lives in ``psd_oracle.c`` (double precision, exhaustive); this
module adds the block-level orchestration in plain Python:

* draft path k of a speculative block drafts depth s with the race of its own
  slot k over its draft row, keyed by the context (key, t, last m tokens of
  prefix || x^(k)_{<s}) -- Sec. 4.3 / Sec. 5 algorithms and the non-identical
  proposal construction (Prop. "heterogeneous PML bound");
* the target chain races all K slots at every depth s = 0..gamma, keyed by the
  context of its own chain prefix || y_{<s} (stopping-time drafter invariance,
  Prop. on stopping-time invariance: the chain never looks at the drafts);
* the walk emits target tokens while they belong to the drafts of the still
  active paths, then the bonus token (Alg. "Multi-Draft ... (Formal)").
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "psd_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

LAYOUT_TREE = 0
LAYOUT_FLAT = 1
NEAR_TIE = 1e-6  # gap (natural-log score units = relative gap of E/p) below which either token is accepted


def build() -> str:
    """Compile the oracle with gcc into oracle/liboracle.so."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-o", _LIB, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


class _RaceResult(ctypes.Structure):
    _fields_ = [
        ("token", ctypes.c_int32),
        ("slot", ctypes.c_int32),
        ("best", ctypes.c_double),
        ("second", ctypes.c_double),
        ("lse", ctypes.c_double),
    ]


_lib_handle = None


def _lib():
    global _lib_handle
    if _lib_handle is not None:
        return _lib_handle
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    i32p = ctypes.POINTER(ctypes.c_int32)
    f32p = ctypes.POINTER(ctypes.c_float)
    f64p = ctypes.POINTER(ctypes.c_double)
    lib.oracle_philox.argtypes = [u32p, u32p, u32p]
    lib.oracle_philox.restype = None
    lib.oracle_fold.argtypes = [u32p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, u32p]
    lib.oracle_fold.restype = None
    lib.oracle_context_key.argtypes = [ctypes.c_uint64, ctypes.c_int64, i32p, ctypes.c_int, u32p]
    lib.oracle_context_key.restype = None
    lib.oracle_uniform.argtypes = [ctypes.c_uint32]
    lib.oracle_uniform.restype = ctypes.c_double
    lib.oracle_clocks.argtypes = [u32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, f64p]
    lib.oracle_clocks.restype = ctypes.c_int
    lib.oracle_clock.argtypes = [u32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    lib.oracle_clock.restype = ctypes.c_double
    lib.oracle_lse.argtypes = [f32p, ctypes.c_int, ctypes.c_float]
    lib.oracle_lse.restype = ctypes.c_double
    lib.oracle_race.argtypes = [f32p, ctypes.c_int, ctypes.c_float, u32p, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, ctypes.POINTER(_RaceResult)]
    lib.oracle_race.restype = ctypes.c_int
    lib.oracle_mpfr.argtypes = [f32p, ctypes.c_int, ctypes.c_float, u32p, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, i32p, i32p, f64p]
    lib.oracle_mpfr.restype = ctypes.c_int
    lib.oracle_detect_term.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_int, i32p, ctypes.c_int64]
    lib.oracle_detect_term.restype = ctypes.c_double
    lib.oracle_detect_clock.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, i32p, ctypes.c_int64]
    lib.oracle_detect_clock.restype = ctypes.c_double
    lib.oracle_detect_sequence.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_int, i32p, ctypes.c_int, ctypes.c_int, i32p, f64p]
    lib.oracle_detect_sequence.restype = ctypes.c_double
    _lib_handle = lib
    return lib


def _u32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.uint32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))


def _i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


# ---------------------------------------------------------------- primitives

def philox(ctr, key):
    """Philox4x32-10 block: 4 counter words, 2 key words -> 4 words."""
    c, cp = _u32(ctr)
    k, kp = _u32(key)
    out, op = _u32(np.zeros(4, np.uint32))
    _lib().oracle_philox(cp, kp, op)
    return [int(x) for x in out]


def fold(kappa, a, b, tag):
    k, kp = _u32(kappa)
    out, op = _u32(np.zeros(2, np.uint32))
    _lib().oracle_fold(kp, a & 0xFFFFFFFF, b & 0xFFFFFFFF, tag & 0xFFFFFFFF, op)
    return (int(out[0]), int(out[1]))


def context_key(key: int, t: int, window) -> tuple:
    """kappa = H(key, absolute position t, window of previous tokens, oldest first)."""
    w, wp = _i32(window if len(window) else np.zeros(1, np.int32))
    out, op = _u32(np.zeros(2, np.uint32))
    _lib().oracle_context_key(ctypes.c_uint64(key & 0xFFFFFFFFFFFFFFFF), int(t), wp, len(window), op)
    return (int(out[0]), int(out[1]))


def uniform(word: int) -> float:
    return _lib().oracle_uniform(word & 0xFFFFFFFF)


def clocks(kappa, slot: int, V: int, layout: int = LAYOUT_TREE) -> np.ndarray:
    """All V clocks E_slot[v] of the keyed source kappa (double)."""
    k, kp = _u32(kappa)
    out = np.empty(V, np.float64)
    rc = _lib().oracle_clocks(kp, slot, V, layout, out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError("oracle_clocks: bad arguments")
    return out


def clock(kappa, slot: int, V: int, v: int, layout: int = LAYOUT_TREE) -> float:
    """One clock E_slot[v] (tree walk root -> token, or one flat word)."""
    k, kp = _u32(kappa)
    return _lib().oracle_clock(kp, slot, V, layout, v)


def lse(logits, T: float) -> float:
    x, xp = _f32(logits)
    return _lib().oracle_lse(xp, x.size, T)


def race(logits, T: float, kappa, slot0: int, nslots: int, layout: int = LAYOUT_TREE) -> dict:
    """Exhaustive race of one row over slots [slot0, slot0+nslots)."""
    x, xp = _f32(logits)
    k, kp = _u32(kappa)
    res = _RaceResult()
    rc = _lib().oracle_race(xp, x.size, T, kp, slot0, nslots, layout, ctypes.byref(res))
    if rc != 0:
        raise ValueError("oracle_race failed (%d)" % rc)
    return {"token": res.token, "slot": res.slot, "best": res.best, "second": res.second, "lse": res.lse}


def mpfr(logits, T: float, kappa, nu: int, layout: int = LAYOUT_TREE, n_out: int = None) -> dict:
    """The nu MPFR samples of one row under the keyed source kappa (exhaustive, double):
    the labels of the smallest ln G_{v,j} - l_v/T over (v, j < nu), G_{v,j} the sum of
    the clocks of slots 0..j of token v.  Returns the first n_out (default nu + 4)
    sorted (token, arrival, score) entries; the samples are the first nu tokens."""
    n_out = nu + 4 if n_out is None else n_out
    x, xp = _f32(logits)
    k, kp = _u32(kappa)
    tok, tp = _i32(np.zeros(n_out, np.int32))
    arr, ap = _i32(np.zeros(n_out, np.int32))
    sc = np.zeros(n_out, np.float64)
    rc = _lib().oracle_mpfr(xp, x.size, T, kp, nu, layout, n_out, tp, ap,
                            sc.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError("oracle_mpfr failed (%d)" % rc)
    return {"tokens": [int(t) for t in tok], "arrivals": [int(a) for a in arr], "scores": [float(v) for v in sc],
            "samples": [int(t) for t in tok[:nu]]}


def token_score(logits, T: float, kappa, slot0: int, nslots: int, v: int, layout: int = LAYOUT_TREE) -> float:
    """Score min_j ln E_j[v] - l_v/T of one token (used to classify near-ties)."""
    x = float(np.float32(logits[v]))
    if x == -np.inf:
        return np.inf
    e = min(clock(kappa, j, len(logits), v, layout) for j in range(slot0, slot0 + nslots))
    return float(np.log(e) - np.float64(x) / np.float64(np.float32(T)))


def detect_term(key: int, m: int, K: int, V: int, tokens, t: int, layout: int = LAYOUT_TREE) -> float:
    tk, tp = _i32(tokens)
    return _lib().oracle_detect_term(ctypes.c_uint64(key), m, K, V, layout, tp, int(t))


def detect_sequence(key: int, m: int, K: int, V: int, tokens, n0: int, layout: int = LAYOUT_TREE):
    """(S_A, M, per-token A_t) of one sequence, scored positions t in [n0, n)."""
    tk, tp = _i32(tokens)
    per = np.empty(tk.size, np.float64)
    cnt = ctypes.c_int32(0)
    S = _lib().oracle_detect_sequence(ctypes.c_uint64(key), m, K, V, layout, tp, tk.size, n0,
                                      ctypes.byref(cnt), per.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return S, int(cnt.value), per


def gamma_tail_log_p(S: float, M: int) -> float:
    """ln p_A with p_A = P(Gamma(M, 1) >= S_A) = Gamma(M, S_A) / Gamma(M) (App. "Gumbel
    Watermark": under the null the M scored A_t are iid Exp(1), so S_A ~ Gamma(M, 1)).

    M is a count, so the regularised upper incomplete gamma is the Poisson sum
    Q(M, S) = sum_{k<M} e^{-S} S^k / k!  (the M-th arrival of a unit-rate Poisson
    process comes after S iff fewer than M arrivals fall in [0, S]); it is summed here
    in the log domain, ln k! from the C library's lgamma (a running sum of ln i drifts
    by ~1e-7 at M = 1e6).  M = 0 (nothing scored) gives
    p = 1; S <= 0 gives p = 1; NaN S or negative M give NaN.
    """
    M = int(M)
    S = float(S)
    if M < 0 or np.isnan(S):
        return float("nan")
    if M == 0 or S <= 0.0:
        return 0.0
    if np.isinf(S):
        return float("-inf")
    k = np.arange(M, dtype=np.float64)
    log_fact = np.array([math.lgamma(i + 1.0) for i in range(M)])
    terms = -S + k * np.log(S) - log_fact
    top = terms.max()
    # a probability: rounding of a sum that is 1 to double precision stays at ln 1
    return min(0.0, float(top + np.log(np.exp(terms - top).sum())))


def anlppt(S: float, M: int) -> float:
    """ANLPPT_A = -(1/M) ln p_A (App. "Gumbel Watermark"); NaN when M = 0."""
    M = int(M)
    if M <= 0:
        return float("nan")
    return -gamma_tail_log_p(S, M) / M


# ---------------------------------------------------------------- block level

def window_of(prefix, path, m: int):
    """Last m tokens of prefix || path, oldest first, padded with -1 in front."""
    seq = list(prefix) + list(path)
    w = seq[-m:] if m > 0 else []
    return [-1] * (m - len(w)) + [int(a) for a in w]


def walk(draft_tokens, chain, K: int, gamma: int, per_path: bool = False):
    """Realised-path walk of one speculative block.

    draft_tokens[k][s]: drafts of path k.  chain[s] (shared target rows) or
    chain[k][s] (per-path target rows, the row of the lowest active path is read).
    Emit the target token of the current depth; stop after it if it is not among
    the drafts of the active paths (correction); otherwise narrow the active set to
    the paths that drafted it.  All gamma accepted -> emit the bonus token.
    Returns the emitted tokens (tau = len)."""
    active = list(range(K))
    out = []
    for s in range(gamma):
        y = int(chain[min(active)][s]) if per_path else int(chain[s])
        out.append(y)
        proposals = {int(draft_tokens[k][s]) for k in active}
        if y < 0 or y not in proposals:
            return out
        active = [k for k in active if int(draft_tokens[k][s]) == y]
    out.append(int(chain[min(active)][gamma]) if per_path else int(chain[gamma]))
    return out


def _check(tag, got, res, logits, T, kappa, slot0, nslots, layout, stats):
    """Compare a GPU-chosen token with the oracle race: exact, near-tie or mismatch."""
    if got == res["token"]:
        stats["exact"] += 1
        return
    if res["token"] >= 0 and got >= 0:
        s_got = token_score(logits, T, kappa, slot0, nslots, got, layout)
        if s_got - res["best"] < NEAR_TIE:
            stats["near_tie"] += 1
            return
    stats["mismatch"] += 1
    stats["mismatches"].append((tag, got, res["token"], res["best"], res["second"]))


def verify_block(*, key, K, gamma, m, T_target, T_draft, prefix, start_pos, target_logits,
                 draft_logits=None, draft_tokens=None, target_rows=1, layout=LAYOUT_TREE,
                 gpu=None, seqs=None):
    """Oracle of one speculative block for sequences `seqs` (default all).

    target_logits: float32 [B][gamma+1][V] (target_rows=1) or [B][K][gamma+1][V].
    draft_logits:  float32 [B][K][gamma][V], or None when draft_tokens [B][K][gamma]
    are given.  gpu: optional dict of the HIP results (draft_tokens, target_tokens,
    out_tokens, out_len, target_lse, draft_lse); when given, every race is run in
    the GPU's context (teacher forcing) and classified exact / near-tie / mismatch,
    so a near-tie cannot derail the rest of the comparison.
    Returns a dict with the oracle's tokens, LSEs and the comparison counts."""
    B = target_logits.shape[0]
    V = target_logits.shape[-1]
    seqs = list(range(B)) if seqs is None else list(seqs)
    stats = {"exact": 0, "near_tie": 0, "mismatch": 0, "mismatches": []}
    out = {"draft_tokens": {}, "target_tokens": {}, "out_tokens": {}, "out_len": {},
           "draft_lse": {}, "target_lse": {}, "stats": stats}
    per_path = target_rows != 1
    for b in range(B):
        if b not in seqs:
            continue
        pre = [int(a) for a in prefix[b]]
        t0 = int(start_pos[b])
        # --- drafts: path k races slot k, sequential over depth
        drafts = np.zeros((K, gamma), np.int64)
        for k in range(K):
            for s in range(gamma):
                if draft_logits is None:
                    drafts[k, s] = int(draft_tokens[b][k][s])
                    continue
                ctx_path = (gpu["draft_tokens"][b][k][:s] if gpu is not None else drafts[k, :s])
                kappa = context_key(key, t0 + s, window_of(pre, ctx_path, m))
                row = draft_logits[b][k][s]
                res = race(row, T_draft, kappa, k, 1, layout)
                out["draft_lse"][(b, k, s)] = res["lse"]
                if gpu is not None:
                    _check(("draft", b, k, s), int(gpu["draft_tokens"][b][k][s]), res, row, T_draft, kappa,
                           k, 1, layout, stats)
                    drafts[k, s] = int(gpu["draft_tokens"][b][k][s])
                else:
                    drafts[k, s] = res["token"]
        out["draft_tokens"][b] = drafts
        # --- target: all K slots; shared chain or one chain per path
        chains = []
        paths = range(K) if per_path else [None]
        for k in paths:
            chain = np.zeros(gamma + 1, np.int64)
            for s in range(gamma + 1):
                if per_path:
                    ctx_path = drafts[k, :s]
                    row = target_logits[b][k][s]
                    gtok = None if gpu is None else int(gpu["target_tokens"][b][k][s])
                else:
                    ctx_path = (gpu["target_tokens"][b][:s] if gpu is not None else chain[:s])
                    row = target_logits[b][s]
                    gtok = None if gpu is None else int(gpu["target_tokens"][b][s])
                kappa = context_key(key, t0 + s, window_of(pre, ctx_path, m))
                res = race(row, T_target, kappa, 0, K, layout)
                out["target_lse"][(b, k, s) if per_path else (b, s)] = res["lse"]
                if gtok is not None:
                    _check(("target", b, k, s), gtok, res, row, T_target, kappa, 0, K, layout, stats)
                    chain[s] = gtok
                else:
                    chain[s] = res["token"]
            chains.append(chain)
        chain_arr = np.stack(chains) if per_path else chains[0]
        out["target_tokens"][b] = chain_arr
        emitted = walk(drafts, chain_arr, K, gamma, per_path)
        out["out_tokens"][b] = emitted
        out["out_len"][b] = len(emitted)
    return out


def verify_block_parallel(workers: int, seqs=None, mpfr_mode: bool = False, **kw) -> dict:
    """verify_block over `seqs` (default all), one sequence per task on `workers`
    threads.  The C oracle runs with the interpreter lock released (ctypes), so the
    sequences are checked in parallel; results and comparison counts are merged."""
    import concurrent.futures

    _lib()  # load (or build) the library once, before the threads start
    B = kw["target_logits"].shape[0]
    seqs = list(range(B)) if seqs is None else list(seqs)
    with concurrent.futures.ThreadPoolExecutor(max_workers=max(1, workers)) as ex:
        fn = verify_block_mpfr if mpfr_mode else verify_block
        parts = list(ex.map(lambda b: fn(seqs=[b], **kw), seqs))
    out = {"draft_tokens": {}, "target_tokens": {}, "out_tokens": {}, "out_len": {}, "draft_lse": {},
           "target_lse": {}, "stats": {"exact": 0, "near_tie": 0, "mismatch": 0, "mismatches": []}}
    for part in parts:
        for k in ("draft_tokens", "target_tokens", "out_tokens", "out_len", "draft_lse", "target_lse"):
            out[k].update(part[k])
        for k in ("exact", "near_tie", "mismatch"):
            out["stats"][k] += part["stats"][k]
        out["stats"]["mismatches"] += part["stats"]["mismatches"]
    return out


# ---------------------------------------------------------------- identical drafters (MPFR)

def context_groups(paths):
    """Paths with equal draft prefixes share a context (Alg. "Multi-Draft ... (Formal)":
    the context tree with multiplicities).  Returns the groups as lists of path
    indices in increasing order, ordered by their lowest index."""
    groups = {}
    for k, pre in enumerate(paths):
        groups.setdefault(tuple(int(t) for t in pre), []).append(k)
    return sorted(groups.values(), key=lambda g: g[0])


def _check_mpfr(tag, got, res, stats):
    """GPU samples of one context (member order) against the oracle's sorted list:
    exact, or each differing sample inside a run of oracle scores closer than
    NEAR_TIE to the one at its rank (either order of near-tied arrivals is valid)."""
    want = res["tokens"][:len(got)]
    if list(got) == want:
        stats["exact"] += 1
        return
    sc = res["scores"]
    for i, g in enumerate(got):
        if g == want[i]:
            continue
        lo = hi = i
        while lo > 0 and sc[lo] - sc[lo - 1] < NEAR_TIE:
            lo -= 1
        while hi + 1 < len(sc) and sc[hi + 1] - sc[hi] < NEAR_TIE:
            hi += 1
        if g not in res["tokens"][lo:hi + 1]:
            stats["mismatch"] += 1
            stats["mismatches"].append((tag, list(got), want, sc))
            return
    stats["near_tie"] += 1


def verify_block_mpfr(*, key, K, gamma, m, T_target, T_draft, prefix, start_pos, target_logits,
                      draft_logits=None, draft_tokens=None, target_rows=1, layout=LAYOUT_TREE, gpu=None, seqs=None):
    """Oracle of one speculative block with K identical drafters (MPFR mode).

    Paths stand for the K drafts of Alg. "Multi-Draft ... (Formal)": at depth s the
    paths whose drafts so far are equal form one context c with multiplicity nu(c)
    = the group's size; the context's proposal row is the draft row of its lowest
    path, its keyed source Pi(c) = the context key of (key, t, last m tokens), and
    its nu(c) drafts are MPFR(Q(.|c), Pi(c), nu(c)) -- the i-th smallest score goes
    to the group's i-th path, so equal draft tokens move to one child context with
    their count as its multiplicity.  The target at a context is MPFR(P(.|c), Pi(c), 1),
    the race of slot 0 alone; the walk is the HET walk (emit y(c*), stop unless it is
    among the drafts D(c*) of the active paths).  Arguments as verify_block."""
    B = target_logits.shape[0]
    seqs = list(range(B)) if seqs is None else list(seqs)
    stats = {"exact": 0, "near_tie": 0, "mismatch": 0, "mismatches": []}
    out = {"draft_tokens": {}, "target_tokens": {}, "out_tokens": {}, "out_len": {},
           "draft_lse": {}, "target_lse": {}, "stats": stats}
    per_path = target_rows != 1
    for b in seqs:
        pre = [int(a) for a in prefix[b]]
        t0 = int(start_pos[b])
        drafts = np.zeros((K, gamma), np.int64)
        for s in range(gamma):
            if draft_logits is None:
                drafts[:, s] = [int(draft_tokens[b][k][s]) for k in range(K)]
                continue
            for k in range(K):
                out["draft_lse"][(b, k, s)] = lse(draft_logits[b][k][s], T_draft)
            for members in context_groups([drafts[k, :s] for k in range(K)]):
                rep = members[0]
                kappa = context_key(key, t0 + s, window_of(pre, drafts[rep, :s], m))
                res = mpfr(draft_logits[b][rep][s], T_draft, kappa, len(members), layout)
                if gpu is not None:
                    got = [int(gpu["draft_tokens"][b][k][s]) for k in members]
                    _check_mpfr(("draft", b, s, tuple(members)), got, res, stats)
                    for k, g in zip(members, got):
                        drafts[k, s] = g
                else:
                    for k, v in zip(members, res["samples"]):
                        drafts[k, s] = v
        out["draft_tokens"][b] = drafts
        chains = []
        for k in (range(K) if per_path else [None]):
            chain = np.zeros(gamma + 1, np.int64)
            for s in range(gamma + 1):
                if per_path:
                    ctx_path, row = drafts[k, :s], target_logits[b][k][s]
                    gtok = None if gpu is None else int(gpu["target_tokens"][b][k][s])
                else:
                    ctx_path = gpu["target_tokens"][b][:s] if gpu is not None else chain[:s]
                    row = target_logits[b][s]
                    gtok = None if gpu is None else int(gpu["target_tokens"][b][s])
                kappa = context_key(key, t0 + s, window_of(pre, ctx_path, m))
                res = race(row, T_target, kappa, 0, 1, layout)
                out["target_lse"][(b, k, s) if per_path else (b, s)] = res["lse"]
                if gtok is not None:
                    _check(("target", b, k, s), gtok, res, row, T_target, kappa, 0, 1, layout, stats)
                    chain[s] = gtok
                else:
                    chain[s] = res["token"]
            chains.append(chain)
        chain_arr = np.stack(chains) if per_path else chains[0]
        out["target_tokens"][b] = chain_arr
        emitted = walk(drafts, chain_arr, K, gamma, per_path)
        out["out_tokens"][b] = emitted
        out["out_len"][b] = len(emitted)
    return out


# ---------------------------------------------------------------- further detection scores

def detect_clocks(key: int, m: int, K: int, V: int, tokens, n0: int, layout: int = LAYOUT_TREE) -> np.ndarray:
    """c_t = K min_j E_j[w_t] for every position (NaN before n0 and for tokens outside
    [0, V)): the pivot is r_t = exp(-c_t), uniform under the null."""
    tk, tp = _i32(tokens)
    out = np.full(tk.size, np.nan)
    for t in range(n0, tk.size):
        out[t] = _lib().oracle_detect_clock(ctypes.c_uint64(key), m, K, V, layout, tp, t)
    return out


def li_params(delta: float):
    """k_Delta = floor(1/(1-Delta)), q_Delta = 1 - k_Delta (1-Delta) (App. on Li et al.'s score).
    1/(1-Delta) within 1e-12 (relative) of an integer counts as that integer, and then q = 0:
    binary rounding (1/(1 - 0.9) = 10.000000000000002) must not leave a spurious q ~ 1e-16."""
    x = 1.0 / (1.0 - delta)
    k = math.floor(x + 1e-12 * x)
    q = 1.0 - k * (1.0 - delta)
    if q < 1e-12:
        q = 0.0
    return k, q


def score_terms(c, delta: float, eps: float) -> dict:
    """Per-token scores of the pivot r = exp(-c) (App. "Gumbel Watermark" and the two
    following appendices): Aaronson's A = -log(1 - r), the U-score U = r, Li et al.'s
    h*_{gum,Delta}(r) = log(k r^{Delta/(1-Delta)} + [q > 0] r^{(1-q)/q}) and Lattimore's
    h_{PL,eps}(r) = min(eps^{-1/2}, (1 - r)^{-1/2}) - (2 - sqrt(eps))."""
    c = np.asarray(c, np.float64)
    r = np.exp(-c)
    one_minus_r = -np.expm1(-c)
    k, q = li_params(delta)
    li = np.log(k * r ** (delta / (1.0 - delta)) + (r ** ((1.0 - q) / q) if q > 0 else 0.0))
    pl = np.minimum(eps ** -0.5, one_minus_r ** -0.5) - (2.0 - math.sqrt(eps))
    return {"A": -np.log(one_minus_r), "U": r, "Li": li, "PL": pl}


def _null_log_mgf(kind: str, lam: float, delta: float, eps: float):
    """(ln E[e^{lam h(U)}], E_lam[h]) under U ~ Unif(0, 1), by adaptive quadrature (the
    tilted mean is the derivative of the log-MGF)."""
    from scipy import integrate
    if kind == "U":
        if lam == 0.0:
            return 0.0, 0.5
        return math.log(math.expm1(lam) / lam), 1.0 / (-math.expm1(-lam)) - 1.0 / lam
    if kind == "Li":
        k, q = li_params(delta)
        h = lambda u: math.log(k * u ** (delta / (1.0 - delta)) + (u ** ((1.0 - q) / q) if q > 0 else 0.0))
        hmax = math.log(k + (1 if q > 0 else 0))
        pts = None
    else:
        c0 = 2.0 - math.sqrt(eps)
        h = lambda u: min(eps ** -0.5, (1.0 - u) ** -0.5) - c0
        hmax = eps ** -0.5 - c0
        pts = [1.0 - eps]
    import warnings
    kw = dict(epsabs=1e-15, epsrel=1e-12, limit=400)
    if pts is not None and 0.0 < pts[0] < 1.0:
        kw["points"] = pts
    with warnings.catch_warnings():
        warnings.simplefilter("ignore", integrate.IntegrationWarning)
        z = integrate.quad(lambda u: math.exp(lam * (h(u) - hmax)), 0.0, 1.0, **kw)[0]
        zh = integrate.quad(lambda u: h(u) * math.exp(lam * (h(u) - hmax)), 0.0, 1.0, **kw)[0]
    return lam * hmax + math.log(z), zh / z


def chernoff_log_p(kind: str, S: float, M: int, delta: float = 0.5, eps: float = 0.01) -> float:
    """Chernoff bound on the null tail of a sum of M iid per-token scores:
    ln p <= min_{lam >= 0} M ln E[e^{lam h(U)}] - lam S (App. "Gumbel Watermark" for the
    U-score; the same construction for Li et al.'s and Lattimore's scores, whose null
    p-values the paper leaves unstated).  0 when S is at most the null mean."""
    from scipy import optimize
    M = int(M)
    if M <= 0 or not math.isfinite(S):
        return float("nan") if (M < 0 or math.isnan(S)) else 0.0
    mean0 = _null_log_mgf(kind, 0.0, delta, eps)[1]
    if S <= M * mean0:
        return 0.0
    dphi = lambda lam: M * _null_log_mgf(kind, lam, delta, eps)[1] - S
    hi = 1.0
    while dphi(hi) < 0.0 and hi < 1e4:
        hi *= 2.0
    lam = optimize.brentq(dphi, 0.0, min(hi, 1e4), xtol=1e-14, rtol=1e-14, maxiter=400) if dphi(min(hi, 1e4)) > 0 \
        else min(hi, 1e4)
    return min(0.0, M * _null_log_mgf(kind, lam, delta, eps)[0] - lam * S)


# ---------------------------------------------------------------- logit processing before the race

def truncation_mask(logits, T: float, top_k: int = 0, top_p: float = 1.0) -> np.ndarray:
    """Tokens kept by top-k, then top-p, truncation (the paper's experiments race the
    processed distribution P_k: temperature, top-k = 50, top-p; Alg. "Batched-target
    direct-top-k MPFR speculative sampling").  Order: logit descending, ties to the
    lowest index; top-k keeps the first min(k, #finite) (k = 0: all finite); top-p then
    keeps the shortest prefix of those whose softmax mass (at T, over the top-k set)
    reaches top_p.  Returns a boolean mask over the vocabulary."""
    x = np.asarray(logits, np.float32)
    finite = np.flatnonzero(x != -np.inf)
    order = finite[np.lexsort((finite, -x[finite].astype(np.float64)))]  # by -x, then index
    if top_k > 0:
        order = order[:top_k]
    if top_p < 1.0 and order.size:
        z = x[order].astype(np.float64) / np.float64(np.float32(T))
        p = np.exp(z - z.max())
        p /= p.sum()
        cum = np.cumsum(p)
        n = int(np.searchsorted(cum, top_p, side="left")) + 1
        order = order[:min(n, order.size)]
    mask = np.zeros(x.size, bool)
    mask[order] = True
    return mask


def truncate(logits, T: float, top_k: int = 0, top_p: float = 1.0) -> np.ndarray:
    """The row with every token outside the kept set at -inf (probability 0)."""
    x = np.array(logits, np.float32, copy=True)
    if top_k > 0 or top_p < 1.0:
        x[~truncation_mask(x, T, top_k, top_p)] = -np.inf
    return x


def truncate_block(arr, T: float, top_k: int, top_p: float):
    """truncate() on every row (last axis) of a logits array."""
    if top_k <= 0 and top_p >= 1.0:
        return arr
    flat = np.asarray(arr, np.float32).reshape(-1, arr.shape[-1])
    return np.stack([truncate(r, T, top_k, top_p) for r in flat]).reshape(arr.shape)

