#!/usr/bin/env python3
"""Write the oracle's multi-step decoding trajectories of the seeded workloads.

For each workload preset and seed, the oracle alone drives the denoising
steps: proposals are drawn from the seeded generator, the oracle decides every
candidate's verdict (Sec. 3 Valid), runs Alg. 4 on the valid ones, and the
harness commit policy (the selected subset, else the single most confident
valid candidate) updates the partial outputs.  At every step the oracle also
runs the sequential fallback after the batch (Alg. 1 in App. C.1) with a
seeded commit budget per sequence, after the step's Alg. 4 subset and after
an empty one; its commits are recorded, not applied.

Output: ``traj_p<preset>_s<seed>.jsonl``, a header line, then one line per
step with digests of the partial outputs and proposals (so that a drift of the
generator is detected), the verdicts, selections and fallback commits as digit
strings (one character per candidate) and the (cover, exact) check counts.

The GPU parity tests replay the same steps through the C ABI and compare
every step with these lines.  Nothing here calls the HIP library.

    python tests/golden/make_trajectories.py [--presets 3 4 5] [--seeds 42 43 44]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2606_00722_amd import workloads as W  # noqa: E402

# steps replayed per preset (the preset's own step count)
STEPS = {1: 1, 2: 8, 3: 16, 4: 4, 5: 32}


def digest(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()[:24]


def budgets(preset: int, seed: int, step: int, B: int, props: int) -> np.ndarray:
    """Seeded per-sequence commit budget n_t of one step (the model's choice
    in the paper; a harness input here)."""
    rng = np.random.default_rng([seed, preset, step, 7])
    return rng.integers(1, props + 2, size=B).astype(np.int32)


def digits(a) -> str:
    return "".join(str(int(v)) for v in a)


def path(preset: int, seed: int) -> str:
    return os.path.join(HERE, f"traj_p{preset}_s{seed}.jsonl")


def make(preset: int, seed: int, nthreads: int) -> str:
    inst = W.make_instance(preset, seed)
    p = oracle.problem_from(inst.lang, inst.vocab)
    steps = STEPS[preset]
    lines = [json.dumps({"preset": preset, "seed": seed, "B": inst.B, "n": inst.n, "steps": steps,
                         "workload": W.PRESET_NAMES[preset],
                         "policy": "commit the Alg. 4 subset, else the most confident valid candidate; "
                                   "fallback commits recorded, not applied"})]
    for k in range(steps):
        t0 = time.time()
        x = inst.seqs.copy()
        pr = W.propose(inst)
        if pr.C == 0:
            break
        v = oracle.validate_batch(p, x, pr.seq, pr.pos, pr.tok, nthreads)
        sel, counts, st = oracle.select(p, x, pr.seq, pr.pos, pr.tok, pr.conf, v, nthreads)
        if st != 0:
            raise RuntimeError(f"oracle select status {st} at preset {preset} seed {seed} step {k}")
        nc = budgets(preset, seed, k, inst.B, inst.cfg["props"])
        acc, st = oracle.fallback(p, x, pr.seq, pr.pos, pr.tok, pr.conf, v, sel, nc, nthreads)
        if st != 0:
            raise RuntimeError(f"oracle fallback status {st} at preset {preset} seed {seed} step {k}")
        # the loop alone (an empty batch): every commit of the step decided by exact checks
        acc0, st = oracle.fallback(p, x, pr.seq, pr.pos, pr.tok, pr.conf, v, np.zeros(pr.C, np.uint8), nc, nthreads)
        if st != 0:
            raise RuntimeError(f"oracle fallback status {st} at preset {preset} seed {seed} step {k}")
        lines.append(json.dumps({"step": k, "seqs": digest(x), "props": digest(pr.seq, pr.pos, pr.tok, pr.conf),
                                 "C": pr.C, "verdict": digits(v), "selected": digits(sel),
                                 "counts": [int(counts[0]), int(counts[1])], "num_commit": nc.tolist(),
                                 "fallback": digits(acc), "fallback_empty": digits(acc0)}))
        W.commit(inst, pr, v, sel)
        print(f"preset {preset} seed {seed} step {k}: C={pr.C} valid={int((v == 1).sum())} "
              f"selected={int(sel.sum())} fallback={int(acc.sum())}/{int(acc0.sum())} {time.time() - t0:.1f}s", flush=True)
    out = path(preset, seed)
    with open(out + ".tmp", "w") as f:
        f.write("\n".join(lines) + "\n")
    os.replace(out + ".tmp", out)
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--presets", type=int, nargs="+", default=[1, 2, 3, 4, 5])
    ap.add_argument("--seeds", type=int, nargs="+", default=[42, 43, 44])
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    args = ap.parse_args()
    oracle.build(force=False)
    for preset in args.presets:
        for seed in args.seeds:
            print("wrote", make(preset, seed, args.threads), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
