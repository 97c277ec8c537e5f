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
    share, Alg. 4 selections of its sequences the same way, and one memo
    build, within about `budget_s` seconds in all."""
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

    ts = time.perf_counter()
    oracle.memo(p)
    memo_s = time.perf_counter() - ts
    share = max(0.0, budget_s - memo_s) / 4
    c1, s1 = checks(1, share)
    cn, sn = checks(nall, share)
    q1, t1 = selections(1, share)
    qn, tn = selections(nall, share)
    return {"value": round(cn / sn, 3), "unit": "checks/s", "cores": nall, "kind": "oracle",
            "sample": f"{cn} validity checks of the first step of the same workload (its {pr0.C} candidates "
                      f"cycled), {nall} threads, {sn:.1f} s",
            "one_core": {"value": round(c1 / s1, 3), "unit": "checks/s", "sample": f"{c1} checks, {s1:.1f} s"},
            "select": {"unit": "sequences/s", "one_core": round(q1 / t1, 4),
                       "all_cores": round(qn / tn, 4),
                       "sample": f"Alg. 4 on {q1} and {qn} sequences of the first step, {t1:.1f} s and {tn:.1f} s"},
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
    ap.add_argument("--cpu-seconds", type=float, default=24.0,
                    help="time budget of the oracle baseline (all legs together)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run only a plain device copy of MIB MiB, 5 launches (the reference kernel that "
                         "scales rocprofv3 FETCH_SIZE / WRITE_SIZE readings to bytes)")
    args = ap.parse_args()
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
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
    inst = W.make_instance(args.preset, args.seed)
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

    ms = {"lexmemo": [], "validate": [], "select": []}
    for e in ev:
        ms["lexmemo"].append(e[0].elapsed_time(e[1]))
        ms["validate"].append(e[1].elapsed_time(e[2]))
        ms["select"].append(e[2].elapsed_time(e[3]))
    phase = {k: float(np.mean(v)) for k, v in ms.items()}
    fallback_ms = float(np.mean([a.elapsed_time(b) for a, b in fb_ms]))

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
    dom = max(kern, key=lambda k: kern[k]["ms_per_step"])
    kd = kern[dom]
    bytes_per_launch = kd["bytes"] / kd["launches"]
    achieved = bytes_per_launch / (kd["ms_per_launch"] * 1e-3) / 1e9
    pmc = pmc_summary(dom, args.preset)
    roof = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 3), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 6),
            "traffic": pmc.get("hbm_bytes_per_launch") if pmc else None,
            "bytes_per_launch": round(bytes_per_launch, 1), "ms_per_launch": round(kd["ms_per_launch"], 4)}
    if pmc:
        for key in ("lds", "valu", "occupancy"):
            if key in pmc:
                roof[key] = pmc[key]

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline")
        cpu = cpu_baseline(inst, traj, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": round(checks / elapsed, 2), "unit": "checks/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(1e3 * elapsed / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": W.PRESET_NAMES[args.preset], "preset": args.preset, "batch": inst.B,
                   "seq_len": inst.n, "candidates_per_step": props_per_step, "steps_cycled": len(traj),
                   "seed": args.seed, "parallelism": "none (1 GPU)"},
        "phases_ms": {**{k: round(v, 4) for k, v in phase.items()}, "fallback": round(fallback_ms, 4)},
        "kernels_ms": {k: {"ms_per_launch": round(v["ms_per_launch"], 4),
                           "launches_per_step": round(v["launches_per_step"], 3),
                           "walks_per_step": round(v["walks_per_step"], 1)} for k, v in kern.items()},
        "fallback": {"ms_per_call": round(fallback_ms, 4), "commits_per_call": round(fb_commits / args.steps, 2),
                     "budget": "per sequence, all of its proposals", "in_step": False},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))
    return 0


if __name__ == "__main__":
    sys.exit(main())
