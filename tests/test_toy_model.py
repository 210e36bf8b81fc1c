"""Host checks of the position-indexed toy model (workloads.ToyModel), the synthetic
stand-in for the models in the multi-block generation loop: its rank map is a
bijection, its rank term tracks -alpha ln(1 + rank), its noise has the stated
moments, its bf16 rows are the round-to-nearest-even of its fp32 rows, and its rows
are distinct functions of (b, t) and of (b, k, t)."""
import math
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

torch = pytest.importorskip("torch")
import workloads  # noqa: E402

TM = workloads.ToyModel(seed=31, draft_seed=32, sigma=3.0, alpha=1.2, tau=(0.5, 2.0), tau_split=4)


def _rank_term(r, alpha):
    q = ((r + 1).astype(np.float32).view(np.uint32) - np.uint32(0x3F800000)).astype(np.int32).astype(np.float32)
    return np.float32(-float(np.float32(alpha)) * math.log(2.0) * 2.0 ** -23) * q


@pytest.mark.parametrize("V", [1, 2, 3, 97, 1024, 32000, 128256, 151936])
def test_rank_is_a_bijection(V):
    z0 = TM.target_row(0, 9, V, fp32_values=True)
    z1 = TM.target_row(0, 9, V, fp32_values=True)
    assert np.array_equal(z0.view(np.uint32), z1.view(np.uint32))
    # with sigma = 0 the row is the rank term alone: its values are the rank term of a permutation
    flat = workloads.ToyModel(seed=31, draft_seed=32, sigma=0.0, alpha=1.2)
    z = flat.target_row(0, 9, V, fp32_values=True)
    want = _rank_term(np.arange(V, dtype=np.int64), 1.2)
    assert np.array_equal(np.sort(z), np.sort(want))


def test_rank_term_tracks_zipf():
    r = np.arange(1 << 19, dtype=np.int64)
    got = _rank_term(r, 1.0).astype(np.float64)
    want = -np.log1p(r.astype(np.float64))
    # the bit-level log2 of 1 + r is within 0.0861 of log2(1 + r) (a chord of log2 on each octave)
    assert np.max(np.abs(got - want)) <= 0.0861 * math.log(2.0) + 1e-6
    assert got[0] == 0.0 and np.all(np.diff(got) <= 0)


def test_noise_moments_and_bf16_rounding():
    V = 1 << 18
    flat = workloads.ToyModel(seed=5, draft_seed=6, sigma=1.0, alpha=0.0, tau=(1.0, 1.0))
    n = flat.target_row(2, 40, V, fp32_values=True).astype(np.float64)  # = sigma * n exactly
    assert abs(n.mean()) < 0.01 and abs(n.var() - 1.0) < 0.01 and n.min() >= -2 * math.sqrt(3) - 1e-6
    d = flat.draft_row(2, 3, 40, V, bf16=False).astype(np.float64) - n
    assert abs(d.mean()) < 0.01 and abs(d.var() - 1.0) < 0.01 and np.abs(d).max() <= math.sqrt(6) + 1e-5
    z = TM.target_row(3, 7, 50000, fp32_values=True)
    assert np.array_equal(TM.target_row(3, 7, 50000), torch.from_numpy(z).to(torch.bfloat16).float().numpy())


def test_rows_depend_on_position_drafter_and_half():
    V = 4096
    rows = [TM.target_row(b, t, V) for b in range(3) for t in range(5, 8)]
    for i in range(len(rows)):
        for j in range(i):
            assert not np.array_equal(rows[i], rows[j])
    t = TM.target_row(1, 11, V, fp32_values=True)
    drafts = [TM.draft_row(1, k, 11, V, bf16=False) for k in range(4)]
    for k in range(4):
        assert not np.array_equal(drafts[k], t)
        for j in range(k):
            assert not np.array_equal(drafts[k], drafts[j])
    # tau[0] below tau_split, tau[1] from it on
    lo = np.std(TM.draft_row(1, 0, 11, V, bf16=False) - TM.target_row(1, 11, V, fp32_values=True))
    hi = np.std(TM.draft_row(5, 0, 11, V, bf16=False) - TM.target_row(5, 11, V, fp32_values=True))
    assert abs(lo - 0.5) < 0.05 and abs(hi - 2.0) < 0.15
