"""The allocation-free entry point psd_verify_static against psd_verify (GPU).

Both run the same kernels; the static one uses the library's fixed per-device
scratch instead of a caller workspace.  Two calls in a row (the second with a
smaller block, reusing the scratch the first left behind) must give exactly the
workspace path's outputs, and healthy status words."""
import os
import sys

import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

DEV = "cuda"


@pytest.fixture(scope="module")
def psd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_21858_amd import psd as m
    return m


def _outputs(w, dev, with_lse):
    o = dict(draft_tokens=torch.full((w.B, w.K, w.gamma), -7, dtype=torch.int32, device=dev),
             out_tokens=torch.full((w.B, w.gamma + 1), -7, dtype=torch.int32, device=dev),
             out_len=torch.full((w.B,), -7, dtype=torch.int32, device=dev),
             target_tokens=torch.full((w.B, w.gamma + 1), -7, dtype=torch.int32, device=dev))
    if with_lse:
        o["target_lse"] = torch.full((w.B, w.gamma + 1), 7.0, dtype=torch.float32, device=dev)
        o["draft_lse"] = torch.full((w.B, w.K, w.gamma), 7.0, dtype=torch.float32, device=dev)
    return o


@pytest.mark.parametrize("layout", [0, 1])
def test_verify_static_matches_workspace_path(psd, layout):
    big = workloads.WORKLOADS[3]                                   # 19.98 MB of scratch
    small = workloads.custom(20000, 3, 2, 5, dtype="bf16", m=3, sigma=3.0, alpha=1.2, tau=0.5)
    for i, w in enumerate((big, small)):
        print(f"[no-alloc] call {i}: {w.name} V={w.V} K={w.K} g={w.gamma} B={w.B} layout={layout}", flush=True)
        blk = workloads.make_block(w, 90 + i, device=DEV)
        params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=layout)
        ws = psd.new_workspace(params, w.B, w.gamma, DEV)
        st_ws = torch.full((1,), -1, dtype=torch.int32, device=DEV)
        st_static = torch.full((1,), -1, dtype=torch.int32, device=DEV)
        ref = psd.verify(params, ws, blk["prefix_tokens"], blk["start_pos"], blk["target_logits"],
                         blk["draft_logits"], out=_outputs(w, DEV, True), status=st_ws)
        got = psd.verify_static(params, blk["prefix_tokens"], blk["start_pos"], blk["target_logits"],
                                blk["draft_logits"], out=_outputs(w, DEV, True), status=st_static)
        torch.cuda.synchronize()
        assert int(st_ws[0]) == 0 and int(st_static[0]) == 0
        for k in ref:
            assert torch.equal(ref[k], got[k]), (i, k)
        assert bool((got["out_len"] >= 1).all()) and bool((got["out_len"] <= w.gamma + 1).all())
