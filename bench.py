#!/usr/bin/env python3
"""Candidate validity checks/s of the EPIC hot path on one MI355X.

One step = one denoising step of the workload over its whole batch: the
lexing memo build, epic_validate_batch over every proposal, then
epic_select_compatible (Alg. 4), on inputs already resident in device memory.
The workload's own step sequence (its evolving partial outputs and proposals)
is generated first, untimed, by running the same path with the harness commit
policy; timed steps then cycle through it.

Prints one JSON line (see the driver contract); `roofline` is reported for the
kernel that takes the most time, with its bytes per launch counted by the
library's work counters (chart rows written and read, memo entries read) and
HIP-event durations; `traffic` comes from the committed rocprofv3 PMC summary
when it was taken on the current kernel sources, else null.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "candidate validity checks/sec on 1 MI355X; % of HBM/LDS roofline"
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")


def source_hash() -> str:
    h = hashlib.sha256()
    for f in ("epic.hip", "walker.inc", "tables.cpp", "tables.h"):
        with open(os.path.join(ROOT, "paper_2606_00722_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def pmc_summary(kernel: str, preset: int):
    """The committed rocprofv3 counter summary of a kernel kind on a workload
    (profiles/<kernel>_preset<p>_pmc.json: HBM bytes per launch, LDS and VALU
    figures) if it was taken on the current kernel sources, else None."""
    path = os.path.join(PROFILES, f"{kernel}_preset{preset}_pmc.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_hash") != source_hash():
        return None
    return d


def copy_calibration(mib: int) -> int:
    import torch

    n = mib << 20
    src = torch.empty(n // 4, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.neg(src, out=dst)  # reads n bytes, writes n bytes
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read": n, "bytes_written": n, "launches": 5}}))
    return 0


KERNEL_KIND = {"lexmemo_kernel": "lexmemo", "base_kernel": "base", "validate_kernel": "validate",
               "select_kernel": "select", "fallback_kernel": "fallback", "spec_clear_kernel": "spec_bookkeeping",
               "spec_account_kernel": "spec_bookkeeping", "base_validate_kernel": "validate"}
LDS_COUNTERS = ("SQ_INSTS_LDS_LOAD_BANDWIDTH", "SQ_INSTS_LDS_STORE_BANDWIDTH", "SQ_INSTS_LDS_ATOMIC_BANDWIDTH")
XCDS = 8  # GRBM_GUI_ACTIVE is summed over the eight accelerator dies
CUS = 256
PEAK_CLOCK_GHZ = 2.4


def lds_peak(configs=((2, 1024), (1, 1024), (2, 512), (4, 256)), iters: int = 1 << 15) -> dict:
    """LDS read bandwidth of the device from the library's streaming
    microbenchmark, over a few launch shapes (workgroups per CU, threads):
    bytes per clock per CU (shader clock measured in the kernel against the
    constant-rate wall clock) and GB/s; the best shape gives the peak used by
    the roofline (times 256 CUs and the 2.4 GHz peak engine clock)."""
    import torch

    from paper_2606_00722_amd import epic

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.zeros(8, dtype=torch.int32, device="cuda:0")
    shader_khz, wall_khz = epic.clock_rates()
    runs = []
    for per_cu, threads in configs:
        blocks = per_cu * cus
        epic.lds_stream(blocks, threads, 256, sink)  # warm
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        epic.lds_stream(blocks, threads, iters, sink)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        s = [int(v) & 0xFFFFFFFF for v in sink.cpu().tolist()]
        ticks, wall = s[2] | (s[3] << 32), s[4] | (s[5] << 32)
        clk_hz = ticks / (wall / (wall_khz * 1e3)) if wall else shader_khz * 1e3
        nbytes = float(blocks) * threads * iters * 16
        runs.append({"workgroups_per_cu": per_cu, "threads": threads, "bytes": nbytes, "ms": round(ms, 4),
                     "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1), "clock_mhz_measured": round(clk_hz / 1e6, 1),
                     "bytes_per_clk_per_cu": round(nbytes / (ms * 1e-3) / clk_hz / cus, 2)})
    best = max(r["bytes_per_clk_per_cu"] for r in runs)
    return {"runs": runs, "cus": cus, "clock_mhz_rated": shader_khz / 1e3, "bytes_per_clk_per_cu": best,
            "peak_gbs": round(best * CUS * PEAK_CLOCK_GHZ, 1), "iters": iters}


def lds_peak_record():
    """The committed LDS peak (profiles/lds_peak.json, the output of
    --lds-peak): bytes per clock per CU from the streaming microbenchmark,
    times 256 CUs and the 2.4 GHz peak engine clock (peak_gbs)."""
    path = os.path.join(PROFILES, "lds_peak.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        return json.load(f).get("lds_peak")


def _counter_csv(run_dir: str) -> dict:
    """Per kernel kind: dispatches, summed counter values and summed
    durations (ns) of one rocprofv3 --pmc run (csv output)."""
    import csv
    import glob

    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    out, seen = {}, set()
    with open(files[0]) as fh:
        for row in csv.DictReader(fh):
            name = row["Kernel_Name"]
            kind = next((v for k, v in KERNEL_KIND.items() if k in name), "copy" if "elementwise" in name else None)
            if kind is None:
                continue
            d = out.setdefault(kind, {"dispatches": 0, "ns": 0.0, "counters": {}, "name": name.split("(")[0],
                                      "scratch": int(float(row.get("Scratch_Size") or 0)),
                                      "vgpr": int(float(row.get("VGPR_Count") or 0)),
                                      "lds_block": int(float(row.get("LDS_Block_Size") or 0))})
            key = (row["Dispatch_Id"], kind)
            if key not in seen:
                seen.add(key)
                d["dispatches"] += 1
                d["ns"] += int(row["End_Timestamp"]) - int(row["Start_Timestamp"])
            c = row["Counter_Name"]
            d["counters"][c] = d["counters"].get(c, 0.0) + float(row["Counter_Value"])
    return out


def _run_source_hash(log_path: str):
    """The source hash a bench run printed in its JSON line (None if absent)."""
    try:
        with open(log_path) as f:
            for line in f:
                if line.startswith("{") and '"source_hash"' in line:
                    return json.loads(line).get("source_hash")
    except OSError:
        pass
    return None


def pmc_summarize(pmc_dir: str, preset: int, hash_override=None) -> int:
    """Turn the rocprofv3 counter runs of one workload into
    profiles/<kernel>_preset<preset>_pmc.json per kernel kind, and print a
    markdown table.  Expected run directories under pmc_dir: p<preset>_lds,
    p<preset>_valu, p<preset>_fetch, p<preset>_write (one counter set each),
    copy_fetch and copy_write (the --copy-calibration 256 runs).  Values are
    averages per dispatch; LDS bytes = 64 x the three LDS bandwidth counters
    (units of 64 bytes); HBM bytes = FETCH_SIZE and WRITE_SIZE (KiB) scaled by
    the plain copy's readings; VALU busy = SQ_ACTIVE_INST_VALU / CUs / one
    die's GRBM_GUI_ACTIVE."""
    from paper_2606_00722_amd import workloads as W

    runs = {k: _counter_csv(os.path.join(pmc_dir, f"p{preset}_{k}")) for k in ("lds", "valu", "fetch", "write")}
    cf = _counter_csv(os.path.join(pmc_dir, "copy_fetch"))["copy"]
    cw = _counter_csv(os.path.join(pmc_dir, "copy_write"))["copy"]
    copy_bytes = 256 << 20
    f_fac = copy_bytes / (cf["counters"]["FETCH_SIZE"] / cf["dispatches"] * 1024)
    w_fac = copy_bytes / (cw["counters"]["WRITE_SIZE"] / cw["dispatches"] * 1024)
    peak = lds_peak_record()
    # the sources the counters were taken on, as the profiled run printed them
    sh = hash_override or _run_source_hash(os.path.join(pmc_dir, f"p{preset}_lds.log")) or source_hash()
    rows = []
    for kind in ("validate", "select", "base", "fallback", "lexmemo"):
        if kind not in runs["lds"]:
            continue
        per = {}
        for name, run in runs.items():
            d = run.get(kind)
            if not d:
                continue
            for c, v in d["counters"].items():
                per[f"{c}@{name}" if c == "GRBM_GUI_ACTIVE" else c] = v / d["dispatches"]
        d0 = runs["lds"][kind]
        us = d0["ns"] / d0["dispatches"] / 1e3
        lds_b = 64.0 * sum(per.get(c, 0.0) for c in LDS_COUNTERS)
        hbm_b = per.get("FETCH_SIZE", 0.0) * 1024 * f_fac + per.get("WRITE_SIZE", 0.0) * 1024 * w_fac
        grbm_valu = per.get("GRBM_GUI_ACTIVE@valu", 0.0) / XCDS
        valu_busy = per.get("SQ_ACTIVE_INST_VALU", 0.0) / CUS / grbm_valu if grbm_valu else None
        valu_util = (per["SQ_THREAD_CYCLES_VALU"] / (per["SQ_ACTIVE_INST_VALU"] * 64)
                     if per.get("SQ_ACTIVE_INST_VALU") else None)
        conflict = per.get("SQ_LDS_BANK_CONFLICT", 0.0) / max(per.get("SQ_LDS_IDX_ACTIVE", 0.0), 1.0)
        hit, miss = per.get("TCC_HIT_sum", 0.0), per.get("TCC_MISS_sum", 0.0)
        lds_gbs = lds_b / (us * 1e-6) / 1e9 if us else None
        rec = {"kernel": kind, "kernel_name": d0["name"], "preset": preset, "workload": W.PRESET_NAMES[preset],
               "source_hash": sh, "dispatches": d0["dispatches"], "us_per_dispatch_counter_run": round(us, 2),
               "hbm_bytes_per_launch": round(hbm_b), "fetch_factor": round(f_fac, 4), "write_factor": round(w_fac, 4),
               "lds_bytes_per_launch": round(lds_b), "lds_gbs_counter_run": round(lds_gbs, 2) if lds_gbs else None,
               "lds_peak_gbs": peak["peak_gbs"] if peak else None,
               "lds_bank_conflict_per_active_cycle": round(conflict, 4),
               "valu_busy": round(valu_busy, 5) if valu_busy is not None else None,
               "valu_thread_utilization": round(valu_util, 4) if valu_util is not None else None,
               "waves": per.get("SQ_WAVES"), "tcc_hit_rate": round(hit / (hit + miss), 4) if hit + miss else None,
               "scratch_bytes_per_lane": d0["scratch"], "vgpr": d0["vgpr"], "lds_block_bytes": d0["lds_block"],
               "counters_per_dispatch": {k: round(v, 1) for k, v in sorted(per.items())}}
        with open(os.path.join(PROFILES, f"{kind}_preset{preset}_pmc.json"), "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
        rows.append(rec)
    print("| kernel | dispatches | us/dispatch | LDS MB | LDS GB/s | of LDS peak | bank-conflict cycles per "
          "LDS-active cycle | VALU busy | VALU thread util | HBM MB | L2 hit rate | scratch B/lane |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|")
    for r in rows:
        frac = (r["lds_gbs_counter_run"] / r["lds_peak_gbs"]
                if r["lds_peak_gbs"] and r["lds_gbs_counter_run"] else None)
        print(f"| {r['kernel_name']} | {r['dispatches']} | {r['us_per_dispatch_counter_run']} | "
              f"{r['lds_bytes_per_launch'] / 1e6:.2f} | {r['lds_gbs_counter_run']} | "
              f"{None if frac is None else round(frac, 5)} | {r['lds_bank_conflict_per_active_cycle']} | "
              f"{r['valu_busy']} | {r['valu_thread_utilization']} | {r['hbm_bytes_per_launch'] / 1e6:.2f} | "
              f"{r['tcc_hit_rate']} | {r['scratch_bytes_per_lane']} |")
    print(f"\nsource_hash {sh}; copy factors FETCH {f_fac:.4f}, WRITE {w_fac:.4f}")
    return 0


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inst, traj, budget_s: float) -> dict:
    """The oracle, untuned, on the host cores: validity checks of the first
    step's candidates (cycled) on one thread and on all threads of the CPU
    share, Alg. 4 selections of its sequences the same way, the prior
    pipeline's checks (the paper's Con. baseline, by phase) on one thread, and
    one memo build, within about `budget_s` seconds in all."""
    import numpy as np

    import oracle

    p = oracle.problem_from(inst.lang, inst.vocab)
    host_cpus = len(os.sched_getaffinity(0))
    nall = max(1, min(16, host_cpus))  # one GPU's share of the host
    x0, pr0 = traj[0]["host"]
    v0 = traj[0]["ref"][0]

    def checks(nth: int, secs: float):
        done, spent = 0, 0.0
        while spent < secs and done < 50 * pr0.C:
            idx = (done + np.arange(max(1, 2 * nth))) % pr0.C
            ts = time.perf_counter()
            oracle.validate_batch(p, x0, pr0.seq[idx], pr0.pos[idx], pr0.tok[idx], nth)
            spent += time.perf_counter() - ts
            done += len(idx)
        return done, spent

    def selections(nth: int, secs: float):
        done, spent, b = 0, 0.0, 0
        while spent < secs and done < 4 * inst.B:
            seqs = [(b + i) % inst.B for i in range(max(1, nth))]
            b += len(seqs)
            idx = np.flatnonzero(np.isin(pr0.seq, seqs))
            ts = time.perf_counter()
            oracle.select(p, x0, pr0.seq[idx], pr0.pos[idx], pr0.tok[idx], pr0.conf[idx], v0[idx], nth)
            spent += time.perf_counter() - ts
            done += len(seqs)
        return done, spent

    def con_checks(secs: float):
        """The prior pipeline (lexing automaton, subset construction, Hopcroft,
        intersection emptiness) on one thread, candidate by candidate."""
        done, spent, ms = 0, 0.0, np.zeros(3)
        while (spent < secs or done == 0) and done < 50 * pr0.C:
            k = np.array([done % pr0.C])
            ts = time.perf_counter()
            _, m = oracle.con_validate_batch(p, x0, pr0.seq[k], pr0.pos[k], pr0.tok[k], 1)
            spent += time.perf_counter() - ts
            ms += m
            done += 1
        return done, spent, ms

    ts = time.perf_counter()
    oracle.memo(p)
    memo_s = time.perf_counter() - ts
    share = max(0.0, budget_s - memo_s) / 5
    c1, s1 = checks(1, share)
    cn, sn = checks(nall, share)
    q1, t1 = selections(1, share)
    qn, tn = selections(nall, share)
    k1, u1, kms = con_checks(share)
    return {"value": round(cn / sn, 3), "unit": "checks/s", "cores": nall, "kind": "oracle",
            "sample": f"{cn} validity checks of the first step of the same workload (its {pr0.C} candidates "
                      f"cycled), {nall} threads, {sn:.1f} s",
            "one_core": {"value": round(c1 / s1, 3), "unit": "checks/s", "sample": f"{c1} checks, {s1:.1f} s"},
            "select": {"unit": "sequences/s", "one_core": round(q1 / t1, 4),
                       "all_cores": round(qn / tn, 4),
                       "sample": f"Alg. 4 on {q1} and {qn} sequences of the first step, {t1:.1f} s and {tn:.1f} s"},
            "prior_pipeline": {"kind": "Con. (lexing automaton, subset construction, Hopcroft minimisation, "
                                       "intersection emptiness)", "unit": "checks/s", "cores": 1,
                               "value": round(k1 / u1, 3),
                               "ms_per_check": {"lex": round(kms[0] / k1, 3), "dfa": round(kms[1] / k1, 3),
                                                "val": round(kms[2] / k1, 3)},
                               "sample": f"{k1} validity checks of the first step, one thread, {u1:.1f} s"},
            "memo_build_s": round(memo_s, 3), "cpu_model": cpu_model(), "host_cpus": host_cpus,
            "threads_note": "all cores = the host CPUs this process may use, at most 16 (one GPU's share)"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--preset", type=int, default=5,
                    help="workload preset 1..5 (default 5: C-like, 64 x 1024 tokens, the largest configuration)")
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--saturate", type=int, default=1, metavar="K",
                    help="saturated variant: the same configuration with K times the batch (same grammar and "
                         "vocabulary; K = 16 gives every CU several walks); reports the step loop only")
    ap.add_argument("--cpu-seconds", type=float, default=24.0,
                    help="time budget of the oracle baseline (all legs together)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lds-peak", action="store_true",
                    help="run only the LDS streaming microbenchmark and print its bandwidth")
    ap.add_argument("--pmc-summary", metavar="DIR",
                    help="summarise the rocprofv3 counter runs under DIR for --preset into profiles/ (no GPU)")
    ap.add_argument("--source-hash", default=None,
                    help="with --pmc-summary: the source hash of the profiled run, when its log does not print it")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run only a plain device copy of MIB MiB, 5 launches (the reference kernel that "
                         "scales rocprofv3 FETCH_SIZE / WRITE_SIZE readings to bytes)")
    args = ap.parse_args()
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
    if args.lds_peak:
        print(json.dumps({"lds_peak": lds_peak()}))
        return 0
    if args.pmc_summary:
        return pmc_summarize(args.pmc_summary, args.preset, args.source_hash)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(sequences shard across GPUs with no collectives in the step)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2606_00722_amd import epic
    from paper_2606_00722_amd import workloads as W

    dev = torch.device("cuda:0")
    base_B = W.PRESETS[args.preset]["B"]
    inst = W.make_instance(args.preset, args.seed, B=base_B * args.saturate if args.saturate > 1 else None)
    arr = W.arrays(inst.lang, inst.vocab)
    props_per_step = inst.cfg["props"] * inst.B
    ctx = epic.Context.from_problem(arr, inst.B, inst.n, props_per_step)
    ws = ctx.alloc_workspace(dev)
    ctx.lexmemo_build()
    t = lambda a, dt=torch.int32: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    # the workload's own step sequence, generated by the same path (untimed)
    traj = []
    for si in range(inst.cfg["steps"]):
        log(f"generating step {si}")
        pr = W.propose(inst)
        if pr.C == 0:
            break
        d = dict(seqs=t(inst.seqs), cs=t(pr.seq), cp=t(pr.pos), ct=t(pr.tok), cf=t(pr.conf, torch.float32),
                 verdict=torch.zeros(pr.C, dtype=torch.uint8, device=dev),
                 selected=torch.zeros(pr.C, dtype=torch.uint8, device=dev), C=pr.C,
                 host=(inst.seqs.copy(), pr))
        ctx.validate(d["seqs"], d["cs"], d["cp"], d["ct"], d["verdict"], ws)
        ctx.select(d["seqs"], d["cs"], d["cp"], d["ct"], d["cf"], d["verdict"], d["selected"], ws)
        torch.cuda.synchronize()
        v, s = d["verdict"].cpu().numpy(), d["selected"].cpu().numpy()
        d["ref"] = (v.copy(), s.copy())
        W.commit(inst, pr, v, s)
        traj.append(d)
    err = ctx.device_error()
    if err != 0:
        print(f"device error flags set while generating the workload: {err:#x}", file=sys.stderr)
        return 1

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]

    def step(d, e=None):
        if e:
            e[0].record()
        ctx.lexmemo_build()
        if e:
            e[1].record()
        ctx.validate(d["seqs"], d["cs"], d["cp"], d["ct"], d["verdict"], ws)
        if e:
            e[2].record()
        ctx.select(d["seqs"], d["cs"], d["cp"], d["ct"], d["cf"], d["verdict"], d["selected"], ws)
        if e:
            e[3].record()

    log("warmup")
    for k in range(args.warmup):
        step(traj[k % len(traj)])
    torch.cuda.synchronize()
    ctx.set_timing(True)  # HIP events around every kernel, on its stream
    ctx.kernel_stats()  # clear
    log("timing")
    checks = 0
    t0 = time.perf_counter()
    for k in range(args.steps):
        d = traj[k % len(traj)]
        step(d, ev[k])
        checks += d["C"]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kstats = ctx.kernel_stats()
    ctx.set_timing(False)
    # outputs of the timed steps equal the generation run (deterministic path)
    for d in traj:
        if not (np.array_equal(d["verdict"].cpu().numpy(), d["ref"][0])
                and np.array_equal(d["selected"].cpu().numpy(), d["ref"][1])):
            print("timed outputs differ from the generation run", file=sys.stderr)
            return 1
    if ctx.device_error() != 0:
        print("device error flags set", file=sys.stderr)
        return 1

    fb_ms, fb_commits, wit_ms, wit_ok = [], 0, [], 0
    if args.saturate == 1:
        # the sequential fallback after the batch (Alg. 1), timed on its own over
        # the same steps: per sequence a budget of all its proposals, so that the
        # loop checks every valid candidate the batch left
        fb_ms, fb_commits = [], 0
        for d in traj:
            nc = np.bincount(d["host"][1].seq, minlength=inst.B).astype(np.int32)
            d["nc"] = t(nc)
            d["accepted"] = torch.zeros(d["C"], dtype=torch.uint8, device=dev)
        for d in traj[:2]:  # warm
            ctx.fallback(d["seqs"], d["cs"], d["cp"], d["ct"], d["cf"], d["verdict"], d["selected"], d["nc"],
                         d["accepted"], ws)
        torch.cuda.synchronize()
        for k in range(args.steps):
            d = traj[k % len(traj)]
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            ctx.fallback(d["seqs"], d["cs"], d["cp"], d["ct"], d["cf"], d["verdict"], d["selected"], d["nc"],
                         d["accepted"], ws)
            e1.record()
            fb_ms.append((e0, e1))
        torch.cuda.synchronize()
        for k in range(args.steps):
            fb_commits += int(traj[k % len(traj)]["accepted"].sum().item())
        if ctx.device_error() != 0:
            print("device error flags set by the fallback", file=sys.stderr)
            return 1

        # witness extraction (failure recovery) for every sequence of the first
        # steps, timed on its own: one call per step over the whole batch
        wws = ctx.alloc_witness_workspace(inst.B, dev)
        wbytes = torch.zeros((inst.B, 1 << 14), dtype=torch.uint8, device=dev)
        wlen = torch.zeros((inst.B, inst.n), dtype=torch.int32, device=dev)
        wst = torch.zeros(inst.B, dtype=torch.int32, device=dev)
        ctx.witness(traj[0]["seqs"], wbytes, wlen, wst, wws, ws)  # warm
        torch.cuda.synchronize()
        wit_ms, wit_ok = [], 0
        for d in traj[:4]:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            ctx.witness(d["seqs"], wbytes, wlen, wst, wws, ws)
            e1.record()
            torch.cuda.synchronize()
            wit_ms.append(e0.elapsed_time(e1))
            wit_ok += int((wst == 1).sum().item())
        del wws
        if ctx.device_error() != 0:
            print("device error flags set by the witness extraction", file=sys.stderr)
            return 1

    ms = {"lexmemo": [], "validate": [], "select": []}
    for e in ev:
        ms["lexmemo"].append(e[0].elapsed_time(e[1]))
        ms["validate"].append(e[1].elapsed_time(e[2]))
        ms["select"].append(e[2].elapsed_time(e[3]))
    phase = {k: float(np.mean(v)) for k, v in ms.items()}
    fallback_ms = float(np.mean([a.elapsed_time(b) for a, b in fb_ms])) if fb_ms else None

    # algorithmic bytes of the walks of one kernel kind, from its work
    # counters over the timed steps: chart entries written (4W B of items,
    # 8 B expected nonterminals, 8 B expected terminals, 4 B origin), memo
    # entries read (16 B), chart entries pulled by row tasks (origin, summary
    # and items: 12 + 4W B), one sequence row per walk (4n B)
    Wd = ctx.item_words

    def walk_bytes(c):
        return float(c[1] * (4 * Wd + 20) + c[2] * 16 + c[4] * (12 + 4 * Wd) + c[0] * 4 * inst.n)

    V, Q = ctx.vocab_size, ctx.num_states
    kern = {}
    for k, st in kstats.items():
        if st["launches"] == 0:
            continue
        by = (16.0 * V * Q + 4.0 * (V + 1) + float(arr.voffs[-1]) + 512.0 * Q) * st["launches"] \
            if k == "lexmemo" else walk_bytes(st["work"])
        kern[k] = {"ms_per_launch": st["ms"] / st["launches"], "launches_per_step": st["launches"] / args.steps,
                   "ms_per_step": st["ms"] / args.steps, "bytes": by, "launches": st["launches"],
                   "walks_per_step": int(st["work"][0]) / args.steps}
    # "select" counts the checks Alg. 4 asks for (walked by the selection's
    # workgroup, or by a helper whose result it took); speculated checks whose
    # results it did not take count apart
    hw = kstats.get("spec_unused", {}).get("work")
    spec = None
    if hw is not None and "select" in kern:
        spec = {"unused_walks_per_step": round(int(hw[0]) / args.steps, 1),
                "unused_bytes_per_select_launch": round(walk_bytes(hw) / kern["select"]["launches"], 1)}
    dom = max(kern, key=lambda k: kern[k]["ms_per_step"])
    kd = kern[dom]
    ms_launch = kd["ms_per_launch"]
    hbm_launch = kd["bytes"] / kd["launches"]
    hbm_gbs = hbm_launch / (ms_launch * 1e-3) / 1e9
    pmc = pmc_summary(dom, args.preset) if args.saturate == 1 else None  # counters are of the default workload
    peak = lds_peak_record()
    lds_peak_gbs = peak["peak_gbs"] if peak else None
    if dom == "lexmemo":  # the one HBM-bound kernel: no LDS traffic
        roof = {"bound": "hbm", "kernel": dom, "achieved": round(hbm_gbs, 3), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(hbm_gbs / HBM_PEAK_GBS, 6), "traffic": pmc.get("hbm_bytes_per_launch") if pmc else None,
                "bytes_per_launch": round(hbm_launch, 1), "ms_per_launch": round(ms_launch, 4)}
    else:
        # walk kernels: the chart's item sets are combined in LDS; algorithmic
        # LDS bytes per applied (task, entry) pair: advance mask, slot words
        # read and ORed (3 x 4W), per chart entry written: its slot words (4W);
        # for the selection, its own checks only (the helpers' speculated
        # checks are reported apart)
        w = kstats[dom]["work"]
        lds_launch = float(w[5] * 12 * Wd + w[1] * 4 * Wd) / kd["launches"]
        lds_gbs = lds_launch / (ms_launch * 1e-3) / 1e9
        roof = {"bound": "lds", "kernel": dom, "achieved": round(lds_gbs, 3), "peak": lds_peak_gbs, "unit": "GB/s",
                "frac": round(lds_gbs / lds_peak_gbs, 7) if lds_peak_gbs else None,
                "traffic": pmc.get("hbm_bytes_per_launch") if pmc else None,
                "bytes_per_launch": round(lds_launch, 1), "ms_per_launch": round(ms_launch, 4),
                "lds_traffic": pmc.get("lds_bytes_per_launch") if pmc else None,
                "lds_traffic_frac": (round(pmc["lds_bytes_per_launch"] / (ms_launch * 1e-3) / 1e9 / lds_peak_gbs, 6)
                                     if pmc and lds_peak_gbs else None),
                "hbm": {"achieved": round(hbm_gbs, 3), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(hbm_gbs / HBM_PEAK_GBS, 7), "bytes_per_launch": round(hbm_launch, 1)},
                "valu": {"busy": pmc.get("valu_busy"), "thread_utilization": pmc.get("valu_thread_utilization")}
                if pmc else None,
                "peak_source": "LDS streaming microbenchmark (profiles/lds_peak.json) x 256 CUs x 2.4 GHz"}
    if pmc:
        roof["counters"] = {"source_hash": pmc["source_hash"], "scratch_bytes_per_lane": pmc.get("scratch_bytes_per_lane"),
                            "tcc_hit_rate": pmc.get("tcc_hit_rate"),
                            "lds_bank_conflict_per_active_cycle": pmc.get("lds_bank_conflict_per_active_cycle")}

    cpu = None
    if not args.no_cpu_baseline and args.saturate == 1:
        log("cpu baseline")
        cpu = cpu_baseline(inst, traj, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": round(checks / elapsed, 2), "unit": "checks/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(1e3 * elapsed / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "source_hash": source_hash(),
        "config": {"workload": W.PRESET_NAMES[args.preset] + (
                       f"; saturated: the batch x{args.saturate} ({inst.B} sequences, same grammar and vocabulary)"
                       if args.saturate > 1 else ""),
                   "preset": args.preset, "batch": inst.B, "seq_len": inst.n,
                   "candidates_per_step": props_per_step, "steps_cycled": len(traj), "seed": args.seed,
                   "saturated": args.saturate > 1, "parallelism": "none (1 GPU)"},
        "phases_ms": {**{k: round(v, 4) for k, v in phase.items()},
                      "fallback": round(fallback_ms, 4) if fallback_ms is not None else None},
        "kernels_ms": {k: {"ms_per_launch": round(v["ms_per_launch"], 4),
                           "launches_per_step": round(v["launches_per_step"], 3),
                           "walks_per_step": round(v["walks_per_step"], 1)} for k, v in kern.items()},
        "select_speculation": spec,
        "fallback": {"ms_per_call": round(fallback_ms, 4), "commits_per_call": round(fb_commits / args.steps, 2),
                     "budget": "per sequence, all of its proposals", "in_step": False} if fb_ms else None,
        "witness": {"ms_per_call": round(float(np.mean(wit_ms)), 4), "sequences_per_call": inst.B,
                    "completions": wit_ok, "calls": len(wit_ms)} if wit_ms else None,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))
    return 0


if __name__ == "__main__":
    sys.exit(main())
