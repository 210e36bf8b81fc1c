"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function include/psd.h declares, and rejects invalid arguments before launching."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def psd():
    from paper_2609_21858_amd import psd as m
    return m


def _declared():
    txt = open(os.path.join(ROOT, "include", "psd.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(psd_[a-z_]+)\s*\(", txt, re.M)))


def test_library_exports_every_declared_symbol(psd):
    names = _declared()
    assert len(names) >= 11
    for n in names:
        assert hasattr(psd.lib(), n), n
        assert n in psd.EXPORTS
    assert psd.lib().psd_abi_version() == 4


def test_workspace_bytes(psd):
    p = psd.make_params(1, 128256, 4, 4, 0.7, 0.7)
    n = psd.workspace_bytes(p, 64, 4)
    assert n > 0 and n % 256 == 0
    assert psd.workspace_bytes(p, 128, 4) > n
    bad = psd.make_params(1, 0, 4, 4)
    assert psd.workspace_bytes(bad, 64, 4) == 0
    assert psd.workspace_bytes(psd.make_params(1, 1 << 20, 4, 4), 1, 1) == 0
    assert psd.workspace_bytes(p, 0, 4) == 0 and psd.workspace_bytes(p, 1, 33) == 0


FAKE = 4096  # a non-NULL, 256-aligned dummy address: never dereferenced by rejected calls


def _verify(psd, params, B=2, gamma=3, target_rows=1, ws_bytes=None, tl=FAKE, dt=FAKE, ot=FAKE, ol=FAKE,
            sp=FAKE, pre=FAKE, ws=FAKE):
    if ws_bytes is None:
        ws_bytes = max(psd.workspace_bytes(params, B, gamma), 1)
    blk = psd.Block(B, gamma, pre, sp, ws, ws_bytes)
    return psd.lib().psd_verify(ctypes.byref(params), ctypes.byref(blk), target_rows, tl, None, dt, ot, ol, None,
                                None, None, None)


@pytest.mark.parametrize("field,value", [("vocab", 0), ("vocab", (1 << 19) + 1), ("num_drafts", 0),
                                         ("num_drafts", 33), ("ctx_window", -1), ("ctx_window", 17),
                                         ("temp_target", 0.0), ("temp_target", float("inf")),
                                         ("temp_draft", -1.0), ("temp_draft", float("nan")), ("dtype", 2),
                                         ("clocks", 5), ("mode", 7)])
def test_verify_rejects_bad_params(psd, field, value):
    p = psd.make_params(1, 1000, 2, 4)
    setattr(p, field, value)
    assert _verify(psd, p) == psd.PSD_E_ARG
    assert psd.lib().psd_last_error()


def test_verify_rejects_bad_block(psd):
    p = psd.make_params(1, 1000, 2, 4)
    assert _verify(psd, p, B=0) == psd.PSD_E_ARG
    assert _verify(psd, p, gamma=0) == psd.PSD_E_ARG
    assert _verify(psd, p, gamma=33) == psd.PSD_E_ARG
    assert _verify(psd, p, sp=None) == psd.PSD_E_ARG
    assert _verify(psd, p, pre=None) == psd.PSD_E_ARG
    assert _verify(psd, p, tl=None) == psd.PSD_E_ARG
    assert _verify(psd, p, dt=None) == psd.PSD_E_ARG
    assert _verify(psd, p, ot=None) == psd.PSD_E_ARG
    assert _verify(psd, p, target_rows=3) == psd.PSD_E_ARG
    assert _verify(psd, p, ws=None) == psd.PSD_E_WORKSPACE
    assert _verify(psd, p, ws_bytes=100) == psd.PSD_E_WORKSPACE
    assert _verify(psd, p, ws=FAKE + 16) == psd.PSD_E_WORKSPACE
    assert "workspace" in psd.lib().psd_last_error().decode()


def test_mode_mpfr_validated_like_het(psd):
    """Identical-drafter mode takes the same arguments and is checked the same way."""
    p = psd.make_params(1, 1000, 2, 4, mode=psd.PSD_MODE_MPFR)
    assert _verify(psd, p, B=0) == psd.PSD_E_ARG
    assert _verify(psd, p, tl=None) == psd.PSD_E_ARG
    assert _verify(psd, p, target_rows=3) == psd.PSD_E_ARG
    assert _verify(psd, p, ws=None) == psd.PSD_E_WORKSPACE
    blk = psd.Block(2, 3, FAKE, FAKE, FAKE, psd.workspace_bytes(p, 2, 3), None)
    assert psd.lib().psd_draft(ctypes.byref(p), ctypes.byref(blk), 0, 4, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    p.mode = 2
    assert _verify(psd, p) == psd.PSD_E_ARG


@pytest.mark.parametrize("top_k,top_p", [(-1, 1.0), (257, 1.0), (50, 0.0), (50, -0.5), (50, 1.5),
                                         (50, float("nan")), (0, 0.9)])
def test_truncation_params_validated(psd, top_k, top_p):
    """top_k in [0, 256]; top_p in (0, 1]; top_p < 1 needs top_k >= 1 (the nucleus is
    taken inside the top-k set)."""
    p = psd.make_params(1, 1000, 2, 4, top_k=top_k, top_p=top_p)
    assert _verify(psd, p, ws_bytes=1 << 30) == psd.PSD_E_ARG
    assert "top_" in psd.lib().psd_last_error().decode()


def test_truncation_workspace(psd):
    """Truncated calls need room for the kept lists: the workspace grows with top_k and a
    block sized for untruncated calls is rejected."""
    base = psd.make_params(1, 32000, 4, 4)
    n0 = psd.workspace_bytes(base, 16, 5)
    n50 = psd.workspace_bytes(psd.make_params(1, 32000, 4, 4, top_k=50), 16, 5)
    n256 = psd.workspace_bytes(psd.make_params(1, 32000, 4, 4, top_k=256, top_p=0.9), 16, 5)
    rows = 16 * 4 * 5 + 16 * 4 * 6  # draft rows and per-path target rows
    assert n0 < n50 < n256 and n50 - n0 >= rows * 50 * 8 and n256 % 256 == 0
    assert psd.workspace_bytes(psd.make_params(1, 32000, 4, 4, top_k=300), 16, 5) == 0
    p = psd.make_params(1, 32000, 4, 4, top_k=50)
    assert _verify(psd, p, B=16, gamma=5, ws_bytes=n0) == psd.PSD_E_WORKSPACE
    for mode in (psd.PSD_MODE_HET, psd.PSD_MODE_MPFR):
        p = psd.make_params(1, 1000, 2, 4, mode=mode, top_k=5, top_p=0.5)
        assert _verify(psd, p, tl=None) == psd.PSD_E_ARG
        assert _verify(psd, p, target_rows=3) == psd.PSD_E_ARG


def test_generation_entry_points_reject_bad_args(psd):
    """psd_advance, psd_toy_logits and psd_generate validate every argument before any
    launch (dummy device addresses are never dereferenced)."""
    L = psd.lib()
    p = psd.make_params(1, 1000, 2, 3)
    i64 = ctypes.c_int64

    def adv(B=2, G=3, max_len=10, stride=12, ot=FAKE, ol=FAKE, text=FAKE, length=FAKE, prefix=FAKE, start=FAKE,
            act=FAKE, params=p):
        return L.psd_advance(ctypes.byref(params), B, G, i64(max_len), ot, ol, text, i64(stride), length, prefix,
                             start, act, None)
    assert adv(B=0) == psd.PSD_E_ARG and adv(G=0) == psd.PSD_E_ARG and adv(G=33) == psd.PSD_E_ARG
    assert adv(max_len=3) == psd.PSD_E_ARG          # max_len must exceed the prompt (m = 3)
    assert adv(stride=9) == psd.PSD_E_ARG           # rows shorter than max_len
    for k in ("text", "length", "prefix", "start", "act"):
        assert adv(**{k: None}) == psd.PSD_E_ARG, k
    assert adv(ot=None) == psd.PSD_E_ARG            # out_len without out_tokens
    lm = psd.make_toy_lm(1, 2, 3.0, 1.2)
    assert L.psd_toy_logits(ctypes.byref(p), None, 2, 3, FAKE, FAKE, FAKE, None) == psd.PSD_E_ARG
    bad = psd.make_toy_lm(1, 2, float("nan"), 1.2)
    assert L.psd_toy_logits(ctypes.byref(p), ctypes.byref(bad), 2, 3, FAKE, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_toy_logits(ctypes.byref(p), ctypes.byref(lm), 2, 3, None, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_toy_logits(ctypes.byref(p), ctypes.byref(lm), 2, 3, FAKE, None, FAKE, None) == psd.PSD_E_ARG
    n = psd.generate_workspace_bytes(p, 2, 3)
    assert n > psd.workspace_bytes(p, 2, 3) and n % 256 == 0
    assert psd.generate_workspace_bytes(psd.make_params(1, 2000, 2, 3), 2, 3) > n
    assert psd.generate_workspace_bytes(psd.make_params(1, 0, 2, 3), 2, 3) == 0
    blocks, bits = ctypes.c_int32(0), ctypes.c_uint32(0)

    def gen(n_pos=8, stride=11, ws=FAKE, nb=n, every=4, text=FAKE, lmp=lm):
        return L.psd_generate(ctypes.byref(p), ctypes.byref(lmp) if lmp else None, 2, 3, n_pos, text, i64(stride),
                              ws, nb, every, 0, ctypes.byref(blocks), ctypes.byref(bits), None)
    assert gen(n_pos=0) == psd.PSD_E_ARG and gen(stride=10) == psd.PSD_E_ARG and gen(every=0) == psd.PSD_E_ARG
    assert gen(text=None) == psd.PSD_E_ARG and gen(lmp=None) == psd.PSD_E_ARG
    assert gen(ws=None) == psd.PSD_E_WORKSPACE and gen(nb=n - 1) == psd.PSD_E_WORKSPACE
    assert gen(ws=FAKE + 16) == psd.PSD_E_WORKSPACE


def test_draft_and_detect_reject_bad_args(psd):
    p = psd.make_params(1, 1000, 2, 4)
    blk = psd.Block(2, 3, FAKE, FAKE, FAKE, psd.workspace_bytes(p, 2, 3))
    L = psd.lib()
    assert L.psd_draft(ctypes.byref(p), ctypes.byref(blk), -1, 1, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_draft(ctypes.byref(p), ctypes.byref(blk), 2, 2, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_draft(ctypes.byref(p), ctypes.byref(blk), 0, 0, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_draft(ctypes.byref(p), ctypes.byref(blk), 0, 1, None, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_detect(ctypes.byref(p), -1, 4, FAKE, FAKE, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_detect(ctypes.byref(p), 2, 4, None, FAKE, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_detect_pvalue(-1, FAKE, FAKE, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_detect_pvalue(2, FAKE, None, FAKE, None, None) == psd.PSD_E_ARG
    assert L.psd_detect_pvalue(2, FAKE, FAKE, None, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_detect_pvalue(0, None, None, None, None, None) == psd.PSD_OK
    assert L.psd_philox(-1, None, None, None, None) == psd.PSD_E_ARG
    assert L.psd_philox(3, None, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_context_keys(None, 1, FAKE, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_clock_values(ctypes.byref(p), 2, None, FAKE, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_workspace_clear(None, 16, None) == psd.PSD_E_ARG


def test_verify_static_rejects_before_launch(psd):
    """The allocation-free entry point takes no workspace and refuses shapes beyond its
    fixed 32 MiB scratch, before touching the device."""
    L = psd.lib()
    p = psd.make_params(1, 128256, 4, 4, 0.7, 0.7)
    ok_blk = psd.Block(64, 4, FAKE, FAKE, None, 0, None)
    with_ws = psd.Block(64, 4, FAKE, FAKE, FAKE, 1 << 20, None)
    args = (1, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None)
    assert L.psd_verify_static(ctypes.byref(p), ctypes.byref(with_ws), *args) == psd.PSD_E_ARG
    assert L.psd_verify_static(ctypes.byref(p), None, *args) == psd.PSD_E_ARG
    big = psd.make_params(1, 256000, 16, 4)
    big_blk = psd.Block(256, 4, FAKE, FAKE, None, 0, None)
    assert psd.workspace_bytes(big, 256, 4) > 32 << 20
    assert L.psd_verify_static(ctypes.byref(big), ctypes.byref(big_blk), *args) == psd.PSD_E_WORKSPACE
    assert b"fixed scratch" in L.psd_last_error()
    assert psd.workspace_bytes(p, 64, 4) <= 32 << 20  # the headline block fits
    bad = psd.make_params(1, 0, 4, 4)
    assert L.psd_verify_static(ctypes.byref(bad), ctypes.byref(ok_blk), *args) == psd.PSD_E_ARG


def test_detect_scores_reject_bad_args(psd):
    p = psd.make_params(1, 1000, 2, 4)
    L = psd.lib()
    good = psd.ScoreParams(0.3, 0.05)
    for bad in (psd.ScoreParams(0.0, 0.05), psd.ScoreParams(1.0, 0.05), psd.ScoreParams(0.3, 0.0),
                psd.ScoreParams(0.3, 1.5), psd.ScoreParams(float("nan"), 0.05)):
        assert L.psd_detect_scores(ctypes.byref(p), ctypes.byref(bad), 2, 4, 4, FAKE, FAKE, FAKE, FAKE,
                                   None) == psd.PSD_E_ARG
        assert L.psd_detect_scores_pvalue(ctypes.byref(bad), 2, FAKE, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_detect_scores(ctypes.byref(p), ctypes.byref(good), 2, 8, 4, FAKE, FAKE, FAKE, FAKE,
                               None) == psd.PSD_E_ARG  # row stride shorter than the scored length
    assert L.psd_detect_scores(ctypes.byref(p), None, 2, 4, 4, FAKE, FAKE, FAKE, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_detect_scores(ctypes.byref(p), ctypes.byref(good), 2, 4, 4, None, FAKE, FAKE, FAKE,
                               None) == psd.PSD_E_ARG
    assert L.psd_detection_rate(3, FAKE, 0, 0.01, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_detection_rate(3, FAKE, 1, 0.0, FAKE, None) == psd.PSD_E_ARG
    assert L.psd_detection_rate(3, None, 1, 0.01, FAKE, None) == psd.PSD_E_ARG
