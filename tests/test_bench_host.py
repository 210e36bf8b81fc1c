"""Host-side logic of bench.py, on the CPU: which kernel-trace rows are the headline
race launches, and the refusal of more than one GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

RACE = "void psd::(anonymous namespace)::race_kernel<true, true, 0>(psd::RaceArgs)"


def _row(i, name):
    return {"Dispatch_Id": str(i), "Kernel_Name": name}


def test_headline_rows_stop_at_the_identical_drafter_leg():
    """The headline leg's race launches come first.  The identical-drafter leg then
    enqueues its streaming launch, its race kernel on a second stream, its sampling
    launch and a walk launch per call: none of its race launches may count, although
    each is dispatched before that call's sampling launch."""
    rows = [_row(i, RACE) for i in range(1, 56)]
    i = 56
    for _ in range(3):
        for name in ("void psd::(anonymous namespace)::mpfr_stream_kernel<true, true>(psd::MpfrArgs)", RACE,
                     "void psd::(anonymous namespace)::mpfr_draft_kernel<true, true, 0>(psd::MpfrArgs)",
                     "psd::(anonymous namespace)::topk_walk_kernel(psd::TopkRaceArgs)"):
            rows.append(_row(i, name))
            i += 1
    rows.append(_row(i, "void psd::(anonymous namespace)::topk_select_kernel<true>(psd::TopkSelectArgs)"))
    got = bench.headline_race_rows(list(reversed(rows)))  # any order in, dispatch order out
    assert [int(r["Dispatch_Id"]) for r in got] == list(range(1, 56))


def test_headline_rows_without_an_identical_drafter_leg():
    rows = [_row(i, RACE) for i in range(1, 11)] + [_row(11, "other_kernel")]
    assert len(bench.headline_race_rows(rows)) == 10


def test_more_than_one_gpu_is_refused():
    """bench.py runs on one GPU: --gpus 2 exits with an error before touching a device."""
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert p.returncode != 0
    assert "one GPU" in p.stderr
