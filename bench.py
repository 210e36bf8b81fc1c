"""Benchmark of one fused draft+verify step of the keyed Poisson race on one MI355X.

A step is one psd_verify call with fused drafting over one block of the
V=128256, K=4, gamma=4, B=64 bf16 workload (Llama-3-sized vocabulary): every
draft row is streamed, its LSE computed and raced on its own slot, every target
row is raced over all K slots, and the walk emits the accepted tokens.  Inputs
are resident in HBM before timing and rotate over enough sets that the 256 MB
Infinity Cache cannot serve them.  Prints one JSON line.

  python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--clocks tree|flat] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0   # MI355X HBM3E, vendor figure
MALL_BYTES = 256 << 20
KERNEL_SOURCES = ["psd_race.hip", "psd_device.hpp", "psd_layout.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "race_kernel_c3_traffic.json")
COUNTERS_FILE = os.path.join(ROOT, "profiles", "race_kernel_c3_counters.json")


def kernel_digest() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_21858_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(clocks: str):
    """HBM bytes per launch from the committed PMC summary, if it was taken on this kernel."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_digest") != kernel_digest() or rec.get("clocks") != clocks:
        return None
    return rec.get("hbm_bytes_per_launch")


def measured_counters(clocks: str):
    """VALU-busy and related derived counters of the race kernel from the committed PMC
    summary, if it was taken on this kernel."""
    try:
        with open(COUNTERS_FILE) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_digest") != kernel_digest() or rec.get("clocks") != clocks:
        return None
    return rec.get("per_dispatch")


def write_counters(csv_path: str, out: str = COUNTERS_FILE) -> dict:
    """Average per race-kernel dispatch of each counter in a rocprofv3 --pmc run."""
    import csv
    import collections

    vals = collections.defaultdict(list)
    clocks = "tree"
    for r in headline_race_rows(list(csv.DictReader(open(csv_path)))):
        clocks = "flat" if r["Kernel_Name"].split("race_kernel<")[1].split(">")[0].endswith("1") else "tree"
        vals[r["Counter_Name"]].append(float(r["Counter_Value"]))
    if not vals:
        raise SystemExit(f"{csv_path}: no race_kernel dispatches")
    rec = {"kernel": "race_kernel", "workload": "V=128256 K=4 gamma=4 B=64 bf16", "clocks": clocks,
           "kernel_digest": kernel_digest(), "dispatches": max(len(v) for v in vals.values()),
           "per_dispatch": {k: sum(v) / len(v) for k, v in sorted(vals.items())}}
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    return rec


def headline_race_rows(rows):
    """Race-kernel rows of the headline (distinct-drafter) step: those dispatched before
    the first identical-drafter kernel (the bench's MPFR leg runs afterwards, and its
    streaming launch comes before its own race kernel on the side stream)."""
    rows = sorted(rows, key=lambda r: int(r["Dispatch_Id"]))
    first_mpfr = min((int(r["Dispatch_Id"]) for r in rows if "mpfr_" in r["Kernel_Name"]), default=1 << 62)
    return [r for r in rows if "race_kernel<" in r["Kernel_Name"] and int(r["Dispatch_Id"]) < first_mpfr]


def write_traffic(fetch_csv: str, write_csv: str, out: str = TRAFFIC_FILE) -> dict:
    """HBM bytes per launch of the race kernel from two rocprofv3 --pmc runs of
    `bench.py --pmc-copy-calibration` (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch).

    Each counter is scaled by what it reads for the plain 1 GiB device copy that the
    calibration run issues after the timed steps (1 GiB read, 1 GiB written)."""
    import csv

    def per_dispatch(path):
        rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
        race = headline_race_rows(rows)
        last = int(race[-1]["Dispatch_Id"])
        copy = [r for r in rows if int(r["Dispatch_Id"]) > last and "copyBuffer" in r["Kernel_Name"]
                and int(r["Grid_Size"]) >= 65536]
        if not race or not copy:
            raise SystemExit(f"{path}: no race_kernel or calibration copy dispatches")
        kib = sum(float(r["Counter_Value"]) for r in race) / len(race)
        cal = sum(float(r["Counter_Value"]) for r in copy) / len(copy)
        clocks = "flat" if race[0]["Kernel_Name"].split("race_kernel<")[1].split(">")[0].endswith("1") else "tree"
        return kib, cal, len(race), len(copy), clocks

    fk, fc, fn, fcn, clocks = per_dispatch(fetch_csv)
    wk, wc, wn, wcn, _ = per_dispatch(write_csv)
    copy_kib = float(1 << 20)  # 1 GiB each way
    f_scale, w_scale = copy_kib / fc, copy_kib / wc
    rec = {"kernel": "race_kernel", "workload": "V=128256 K=4 gamma=4 B=64 bf16", "clocks": clocks,
           "kernel_digest": kernel_digest(),
           "fetch_kib_per_dispatch": fk, "write_kib_per_dispatch": wk,
           "copy_fetch_kib": fc, "copy_write_kib": wc, "fetch_scale": f_scale, "write_scale": w_scale,
           "race_dispatches": [fn, wn], "copy_dispatches": [fcn, wcn],
           "hbm_bytes_per_launch": int(round((fk * f_scale + wk * w_scale) * 1024))}
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    return rec


def cpu_baseline(blk, w, clocks_id, n_seq, n_seq_single):
    """The oracle as it stands, on the host cores of this machine: all n_seq sequences of
    the block split over one thread per available core (the C oracle runs without the
    interpreter lock), and the first n_seq_single sequences on one thread."""
    import oracle
    import workloads

    tl = workloads.as_f32_numpy(blk["target_logits"][:n_seq])
    dl = workloads.as_f32_numpy(blk["draft_logits"][:n_seq])
    pre = blk["prefix_tokens"][:n_seq].cpu().numpy()
    sp = blk["start_pos"][:n_seq].cpu().numpy()
    kw = dict(key=w.key, K=w.K, gamma=w.gamma, m=w.m, T_target=w.T_target, T_draft=w.T_draft, prefix=pre,
              start_pos=sp, target_logits=tl, draft_logits=dl, layout=clocks_id)
    affinity = len(os.sched_getaffinity(0))
    workers = max(1, min(affinity, int(os.environ.get("OMP_NUM_THREADS", affinity))))
    t0 = time.perf_counter()
    oracle.verify_block(seqs=list(range(n_seq_single)), **kw)
    dt1 = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.verify_block_parallel(workers, seqs=list(range(n_seq)), **kw)
    dt = time.perf_counter() - t0
    rows = w.K * w.gamma + w.gamma + 1
    return {"value": n_seq * w.gamma / dt, "unit": "positions/s", "cores": workers, "kind": "oracle",
            "affinity_cpus": affinity, "single_thread_value": n_seq_single * w.gamma / dt1,
            "sample": f"all-cores leg: sequences 0..{n_seq - 1} of the B={w.B} block ({n_seq * rows} rows), one "
                      f"thread per sequence on {workers} threads, {dt:.1f} s; single-thread leg: sequences "
                      f"0..{n_seq_single - 1} ({n_seq_single * rows} rows), {dt1:.1f} s; exhaustive "
                      f"double-precision clocks, two-pass LSE, race and walk in plain C"}


def detect_leg(psd, torch, clocks_id, dev, launches=20, replicate=1):
    """Detection throughput on the stress workload's text shape: 256 sequences of
    512 scored tokens after a 4-token prompt, K=16, V=256000 (replicate: that many
    times more sequences).  The per-token work (context key plus K keyed clocks)
    does not depend on the token values, so uniform tokens stand in for generated
    text (parity on generated text is a test)."""
    import workloads
    w5 = workloads.WORKLOADS[5]
    n_seq, n_pos = w5.B * replicate, 512
    toks = workloads.uniform_tokens(n_seq, w5.m + n_pos, w5.V, seed=5).to(dev)
    n0 = torch.full((n_seq,), w5.m, dtype=torch.int32, device=dev)
    p5 = psd.make_params(w5.key, w5.V, w5.K, w5.m, dtype=w5.torch_dtype, clocks=clocks_id)
    for _ in range(3):
        psd.detect(p5, toks, n0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(launches):
        psd.detect(p5, toks, n0)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / launches
    # the Gamma-tail p-value and ANLPPT of the scores (one fp64 wavefront per sequence)
    score, count, _ = psd.detect(p5, toks, n0)
    for _ in range(3):
        psd.detect_pvalue(score, count)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(launches):
        psd.detect_pvalue(score, count)
    e1.record()
    torch.cuda.synchronize()
    ms_p = e0.elapsed_time(e1) / launches
    draws = 6 if clocks_id == psd.PSD_CLOCKS_TREE else 1
    # key folds, the K float clocks, and the exact rebuild of the smallest one
    calls = (w5.m + 1) + w5.K * draws + draws
    return {"workload": f"detection: {n_seq} sequences x {n_pos} scored tokens, K={w5.K}, V={w5.V}, m={w5.m}",
            "tokens_per_s": n_seq * n_pos / (ms / 1e3), "ms_per_launch": ms, "launches": launches,
            "philox_calls_per_token": calls,
            "philox_calls_per_s": n_seq * n_pos * calls / (ms / 1e3),
            "pvalue_ms_per_launch": ms_p}


def mpfr_leg(psd, torch, w, sets, clocks_id, dev, launches=20):
    """The same block with identical drafters (MPFR mode): contexts drafted one launch
    per depth (multi-sample PFR), then the fused kernel races the target rows on
    slot 0.  Same algorithmic bytes as the distinct-drafter step."""
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=clocks_id,
                             mode=psd.PSD_MODE_MPFR)
    ws = psd.new_workspace(params, w.B, w.gamma, dev)
    status = torch.zeros((1,), dtype=torch.int32, device=dev)
    outs = [dict(out_tokens=torch.empty((w.B, w.gamma + 1), dtype=torch.int32, device=dev),
                 out_len=torch.empty((w.B,), dtype=torch.int32, device=dev)) for _ in sets]
    dts = [torch.empty((w.B, w.K, w.gamma), dtype=torch.int32, device=dev) for _ in sets]

    def step(i):
        s = sets[i % len(sets)]
        psd.verify(params, ws, s["prefix_tokens"], s["start_pos"], s["target_logits"], s["draft_logits"],
                   dts[i % len(sets)], out=outs[i % len(sets)], status=status)

    for i in range(3):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(launches):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    if int(status[0]) or psd.workspace_errors(ws):
        raise RuntimeError("MPFR step reported errors")
    ms = e0.elapsed_time(e1) / launches
    nbytes = w.algorithmic_bytes()
    return {"workload": w.name + ", identical drafters (MPFR)", "ms_per_step": ms,
            "positions_per_s": w.B * w.gamma / (ms / 1e3), "achieved_gbps": nbytes / (ms / 1e3) / 1e9,
            "frac_of_hbm_peak": nbytes / (ms / 1e3) / 1e9 / PEAK_HBM_GBPS, "launches": launches,
            "mean_tau": float(outs[(launches - 1) % len(sets)]["out_len"].float().mean())}


def topk_leg(psd, torch, w, sets, clocks_id, dev, mpfr=False, top_k=50, top_p=1.0, launches=20):
    """The same block with every row truncated to its top_k logits (the paper's
    experiments use top-k = 50): one selection launch over the draft rows and one over
    the target rows, then the list races and the walk.  Algorithmic bytes: every row
    read once, as in the untruncated step."""
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=clocks_id,
                             mode=psd.PSD_MODE_MPFR if mpfr else psd.PSD_MODE_HET, top_k=top_k, top_p=top_p)
    ws = psd.new_workspace(params, w.B, w.gamma, dev)
    status = torch.zeros((1,), dtype=torch.int32, device=dev)
    outs = [dict(out_tokens=torch.empty((w.B, w.gamma + 1), dtype=torch.int32, device=dev),
                 out_len=torch.empty((w.B,), dtype=torch.int32, device=dev)) for _ in sets]
    dts = [torch.empty((w.B, w.K, w.gamma), dtype=torch.int32, device=dev) for _ in sets]

    def step(i):
        s = sets[i % len(sets)]
        psd.verify(params, ws, s["prefix_tokens"], s["start_pos"], s["target_logits"], s["draft_logits"],
                   dts[i % len(sets)], out=outs[i % len(sets)], status=status)

    for i in range(3):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(launches):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    if int(status[0]) or psd.workspace_errors(ws):
        raise RuntimeError("top-k step reported errors")
    ms = e0.elapsed_time(e1) / launches
    nbytes = w.algorithmic_bytes()
    return {"workload": w.name + (", identical drafters (MPFR)" if mpfr else "") + f", top-k {top_k}"
            + (f", top-p {top_p}" if top_p < 1.0 else ""), "ms_per_step": ms,
            "positions_per_s": w.B * w.gamma / (ms / 1e3), "achieved_gbps": nbytes / (ms / 1e3) / 1e9,
            "frac_of_hbm_peak": nbytes / (ms / 1e3) / 1e9 / PEAK_HBM_GBPS, "launches": launches,
            "mean_tau": float(outs[(launches - 1) % len(sets)]["out_len"].float().mean())}


def generation_leg(psd, torch, clocks_id, dev, n_pos=512):
    """The stress workload's generation statement on the device: 256 sequences x 512
    positions, V=256000, K=16, gamma=4, bf16, with the position-indexed toy model
    (psd_generate: toy rows -> fused verify -> commit, the active count read every 16
    blocks), once as captured-graph replays and once eagerly; and, for comparison, the
    same blocks driven from Python with a host synchronisation per block."""
    import workloads
    w = workloads.WORKLOADS[5]
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=clocks_id)
    lm = psd.make_toy_lm(2026, 12, w.sigma, w.alpha, w.tau, w.B // 2)
    g = torch.Generator().manual_seed(77)
    prompts = torch.randint(0, w.V, (w.B, w.m), generator=g, dtype=torch.int64).to(torch.int32).to(dev)
    ws = torch.empty(psd.generate_workspace_bytes(params, w.B, w.gamma), dtype=torch.uint8, device=dev)
    out = {"workload": f"{w.name}, {w.B} x {n_pos} positions, position-indexed toy model", "tokens": w.B * n_pos}
    texts = {}
    for name, graph in (("graph", True), ("eager", False)):
        psd.generate(params, lm, prompts, 32, w.gamma, check_every=16, use_graph=graph, ws=ws)  # warm-up
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        text, blocks, bits = psd.generate(params, lm, prompts, n_pos, w.gamma, check_every=16, use_graph=graph, ws=ws)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        if bits:
            raise RuntimeError(f"generation reported error bits {bits}")
        texts[name] = text
        out[name] = {"wall_s": dt, "blocks": blocks, "tokens_per_s": w.B * n_pos / dt, "ms_per_block": dt / blocks * 1e3}
    # host-driven loop: the same calls, a synchronisation and a host read per block
    m = w.m
    text = torch.full((w.B, m + n_pos), -1, dtype=torch.int32, device=dev)
    text[:, :m] = prompts
    length = torch.empty(w.B, dtype=torch.int64, device=dev)
    start = torch.empty(w.B, dtype=torch.int64, device=dev)
    prefix = torch.empty((w.B, m), dtype=torch.int32, device=dev)
    act = torch.empty(1, dtype=torch.int32, device=dev)
    bws = psd.new_workspace(params, w.B, w.gamma, dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    psd.advance(params, w.gamma, m + n_pos, text, length, prefix, start, act)
    blocks = 0
    while True:
        tl, dl = psd.toy_logits(params, lm, w.gamma, start)
        o = psd.verify(params, bws, prefix, start, tl, dl)
        psd.advance(params, w.gamma, m + n_pos, text, length, prefix, start, act, o["out_tokens"], o["out_len"])
        blocks += 1
        if int(act[0]) == 0:  # the host read synchronises
            break
    dt = time.perf_counter() - t0
    out["host_loop"] = {"wall_s": dt, "blocks": blocks, "tokens_per_s": w.B * n_pos / dt,
                        "ms_per_block": dt / blocks * 1e3}
    out["same_text"] = bool(torch.equal(texts["graph"], texts["eager"]) and torch.equal(texts["graph"], text))
    out["positions_per_block"] = n_pos / float(blocks)  # of the sequence that needed the most blocks
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--clocks", choices=["tree", "flat"], default="tree")
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seqs", type=int, default=64, help="sequences of the all-cores oracle leg")
    ap.add_argument("--cpu-seqs-single", type=int, default=16, help="sequences of the single-thread leg")
    ap.add_argument("--no-detect-100x", action="store_true")
    ap.add_argument("--no-generation", action="store_true")
    ap.add_argument("--pmc-copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (for FETCH/WRITE_SIZE scaling)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the HBM traffic record from two rocprofv3 --pmc counter files and exit")
    ap.add_argument("--counters-from", metavar="CSV",
                    help="write the race kernel's derived-counter record from a rocprofv3 --pmc file and exit")
    args = ap.parse_args()
    if args.traffic_from:
        print(json.dumps(write_traffic(*args.traffic_from)))
        return
    if args.counters_from:
        print(json.dumps(write_counters(args.counters_from)))
        return
    if args.gpus != 1:
        print(f"bench.py: the race kernel runs on one GPU only (asked for --gpus {args.gpus}); it has no "
              f"inter-GPU collectives.  Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    import workloads
    from paper_2609_21858_amd import psd

    w = workloads.WORKLOADS[args.config]
    clocks_id = psd.PSD_CLOCKS_TREE if args.clocks == "tree" else psd.PSD_CLOCKS_FLAT
    dev = "cuda:0"
    torch.cuda.set_device(0)
    bytes_per_launch = w.algorithmic_bytes()
    n_sets = max(2, math.ceil(2.3 * MALL_BYTES / bytes_per_launch))
    sets = [workloads.make_block(w, seed=1000 + i, device=dev) for i in range(n_sets)]
    params = psd.make_params(w.key, w.V, w.K, w.m, w.T_target, w.T_draft, dtype=w.torch_dtype, clocks=clocks_id)
    ws = psd.new_workspace(params, w.B, w.gamma, dev)
    outs = [dict(draft_tokens=torch.empty((w.B, w.K, w.gamma), dtype=torch.int32, device=dev),
                 out_tokens=torch.empty((w.B, w.gamma + 1), dtype=torch.int32, device=dev),
                 out_len=torch.empty((w.B,), dtype=torch.int32, device=dev)) for _ in range(n_sets)]

    def step(i):
        s = sets[i % n_sets]
        o = outs[i % n_sets]
        psd.verify(params, ws, s["prefix_tokens"], s["start_pos"], s["target_logits"], s["draft_logits"],
                   o["draft_tokens"], out=o)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    if psd.workspace_errors(ws):
        raise RuntimeError("kernel reported errors during warmup")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        step(i)
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    total_ms = ev[0].elapsed_time(ev[-1])
    if psd.workspace_errors(ws):
        raise RuntimeError("kernel reported errors during timing")
    ms_step = total_ms / args.steps
    positions = w.B * w.gamma
    value = positions / (ms_step / 1e3)
    avg_launch_ms = sum(per) / len(per)
    achieved = bytes_per_launch / (avg_launch_ms / 1e3) / 1e9
    mean_tau = float(outs[(args.steps - 1) % n_sets]["out_len"].float().mean())

    if args.pmc_copy_calibration:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    res = {
        "metric": "verified draft positions/sec and achieved HBM GB/s (V=128256, K=4, B=64)",
        "value": value,
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "V": w.V, "K": w.K, "gamma": w.gamma, "B": w.B, "logits": w.dtype,
                   "T": w.T_target, "clocks": args.clocks, "fused_drafting": True, "input_sets": n_sets},
        "hbm_gbps": achieved,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBPS,
                     "traffic": measured_traffic(args.clocks) if args.config == 3 else None,
                     "counters": measured_counters(args.clocks) if args.config == 3 else None,
                     "algorithmic_bytes_per_launch": bytes_per_launch, "avg_launch_ms": avg_launch_ms,
                     "min_launch_ms": min(per), "max_launch_ms": max(per)},
        "mean_tau": mean_tau,
        "wall_s": wall,
    }
    res["mpfr"] = mpfr_leg(psd, torch, w, sets, clocks_id, dev)
    res["topk"] = [topk_leg(psd, torch, w, sets, clocks_id, dev),
                   topk_leg(psd, torch, w, sets, clocks_id, dev, mpfr=True),
                   topk_leg(psd, torch, w, sets, clocks_id, dev, top_p=0.9)]
    res["detect"] = detect_leg(psd, torch, clocks_id, dev)
    if not args.no_generation:
        res["generation"] = generation_leg(psd, torch, clocks_id, dev)
    if not args.no_detect_100x:
        res["detect_100x"] = detect_leg(psd, torch, clocks_id, dev, launches=5, replicate=100)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(sets[0], w, clocks_id, min(args.cpu_seqs, w.B),
                                           min(args.cpu_seqs_single, w.B))
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
