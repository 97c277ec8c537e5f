"""Every candidate of every step of the seeded workloads, through the C ABI,
against the oracle's stored trajectories (tests/golden/traj_*.jsonl, written
by tests/golden/make_trajectories.py, which calls only the oracle).

Each workload is replayed step by step on the GPU, in the launch
configuration the benchmark times: the step's proposals are drawn from the
seeded generator, the device decides every candidate (Sec. 3 Valid), runs
Alg. 4 on its own verdicts, and the harness commit policy updates the
partial outputs, exactly as the oracle's run did.  At every step the partial
outputs and proposals must hash as recorded, and the verdicts, the selected
subset, the (cover, exact) check counts and the commits of the sequential
fallback (Alg. 1 in App. C.1; after the selected subset and after an empty
one, seeded budgets) must be bit-exact.  Because each step's inputs follow
from the previous step's outputs, a single differing bit anywhere stops the
replay at that step."""
import glob
import json
import os
import re

import numpy as np
import pytest

from paper_2606_00722_amd import workloads as W
from tests.golden import make_trajectories as MT

pytestmark = pytest.mark.gpu

# every stored trajectory (presets 1-5, seeds 42-44)
CASES = sorted((int(m.group(1)), int(m.group(2))) for m in
               (re.search(r"traj_p(\d)_s(\d+)\.jsonl$", f) for f in glob.glob(os.path.join(os.path.dirname(MT.__file__),
                                                                                        "traj_p*_s*.jsonl"))) if m)


@pytest.fixture(scope="module")
def gpu_mod():
    import torch

    if not torch.cuda.is_available():
        pytest.fail("no GPU visible to the gpu-marked tests")
    from tests import gpu_util

    return gpu_util


def load(preset, seed):
    with open(MT.path(preset, seed)) as f:
        rows = [json.loads(l) for l in f if l.strip()]
    return rows[0], rows[1:]


@pytest.mark.parametrize("preset,seed", CASES)
def test_trajectory_bit_exact(preset, seed, gpu_mod):
    head, steps = load(preset, seed)
    inst = W.make_instance(preset, seed)
    assert (head["B"], head["n"], head["steps"]) == (inst.B, inst.n, len(steps))
    g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), inst.B, inst.n, max(inst.cfg["props"] * inst.B, 64))
    for rec in steps:
        k = rec["step"]
        x = inst.seqs.copy()
        pr = W.propose(inst)
        assert MT.digest(x) == rec["seqs"], f"step {k}: partial outputs differ from the oracle's run"
        assert MT.digest(pr.seq, pr.pos, pr.tok, pr.conf) == rec["props"], f"step {k}: proposals differ"
        v = g.validate(x, pr.seq, pr.pos, pr.tok)
        assert g.errors() == 0
        assert MT.digits(v) == rec["verdict"], f"step {k}: verdicts"
        sel, counts = g.select(x, pr.seq, pr.pos, pr.tok, pr.conf, v)
        assert g.errors() == 0
        assert MT.digits(sel) == rec["selected"], f"step {k}: selection"
        assert list(counts) == rec["counts"], f"step {k}: (cover, exact) checks"
        nc = np.array(rec["num_commit"], np.int32)
        acc = g.fallback(x, pr.seq, pr.pos, pr.tok, pr.conf, v, sel, nc)
        assert MT.digits(acc) == rec["fallback"], f"step {k}: fallback after the subset"
        acc0 = g.fallback(x, pr.seq, pr.pos, pr.tok, pr.conf, v, np.zeros(pr.C, np.uint8), nc)
        assert MT.digits(acc0) == rec["fallback_empty"], f"step {k}: fallback after an empty subset"
        assert g.errors() == 0
        W.commit(inst, pr, v, sel)
