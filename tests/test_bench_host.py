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


def _pmc_csv(path, race_values, copy_value):
    import csv
    rows = []
    i = 1
    rows.append(dict(Dispatch_Id=i, Kernel_Name="__amd_rocclr_copyBuffer", Grid_Size=1 << 20, Counter_Value=7.0))
    for v in race_values:
        i += 1
        rows.append(dict(Dispatch_Id=i, Kernel_Name=RACE, Grid_Size=262144, Counter_Value=v))
    for name, grid, v in (("void psd::(anonymous namespace)::mpfr_stream_kernel<true, true>(psd::MpfrArgs)", 131072, 5.0),
                          (RACE, 262144, 99999.0),  # the identical-drafter leg's race: not a headline launch
                          ("__amd_rocclr_copyBuffer", 1024, 3.0),  # a small copy: not the calibration
                          ("__amd_rocclr_copyBuffer", 1 << 22, copy_value),
                          ("__amd_rocclr_copyBuffer", 1 << 22, copy_value)):
        i += 1
        rows.append(dict(Dispatch_Id=i, Kernel_Name=name, Grid_Size=grid, Counter_Value=v))
    with open(path, "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=list(rows[0]))
        wr.writeheader()
        wr.writerows(rows)


def test_traffic_scaling_from_the_copy_calibration(tmp_path):
    """HBM bytes per launch = mean FETCH_SIZE of the headline race launches, scaled by
    1 GiB over what FETCH_SIZE reads for the 1 GiB calibration copy, plus WRITE_SIZE
    scaled the same way (counters in KiB).  Copies before the race launches, small
    copies and the identical-drafter leg's race launch do not count."""
    fetch, write, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "t.json"
    _pmc_csv(fetch, [100000.0, 110000.0, 120000.0], 524288.0)  # fetch reads half a copy's bytes
    _pmc_csv(write, [10000.0, 10000.0, 10000.0], 1048576.0)
    rec = bench.write_traffic(str(fetch), str(write), str(out))
    assert rec["race_dispatches"] == [3, 3] and rec["copy_dispatches"] == [2, 2]
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["hbm_bytes_per_launch"] == (110000 * 2 + 10000) * 1024
    assert rec["clocks"] == "tree"
