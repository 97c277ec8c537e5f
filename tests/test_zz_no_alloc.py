"""epic_validate_batch_noalloc, the entry point for callers that cannot
allocate device memory, through the C ABI: its verdicts equal
epic_validate_batch's on the same inputs, on two calls in a row (the second
smaller), and sizes beyond the context are rejected."""
import numpy as np
import pytest

from paper_2606_00722_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu_mod():
    import torch

    if not torch.cuda.is_available():
        pytest.fail("no GPU visible to the gpu-marked tests")
    from tests import gpu_util

    return gpu_util


def noalloc(g, seqs, seq, pos, tok):
    torch = g.torch
    C = len(seq)
    out = torch.full((max(C, 1),), 7, dtype=torch.uint8, device=g.dev)
    g.ctx.validate_noalloc(g.t(seqs), g.t(seq), g.t(pos), g.t(tok), out[:C])
    torch.cuda.synchronize()
    return out[:C].cpu().numpy()


@pytest.mark.parametrize("preset", [2, 4, 5])
def test_noalloc_equals_validate_batch(preset, gpu_mod):
    from paper_2606_00722_amd import epic

    inst = W.make_instance(preset, 42)
    pr = W.propose(inst)
    g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), inst.B, inst.n, max(pr.C, 64))
    want = g.validate(inst.seqs, pr.seq, pr.pos, pr.tok)
    got = noalloc(g, inst.seqs, pr.seq, pr.pos, pr.tok)
    assert g.errors() == 0
    assert np.array_equal(got, want) and 0 < int(want.sum()) < len(want)
    # a second, smaller call: half the sequences and their candidates
    half = inst.B // 2
    keep = pr.seq < half
    seqs2 = np.ascontiguousarray(inst.seqs[:half])
    want2 = g.validate(seqs2, pr.seq[keep], pr.pos[keep], pr.tok[keep])
    got2 = noalloc(g, seqs2, pr.seq[keep], pr.pos[keep], pr.tok[keep])
    assert g.errors() == 0
    assert np.array_equal(got2, want2) and len(got2) < len(got)
    # sizes beyond what the context was created for are rejected
    n = max(pr.C, 64) + 1
    with pytest.raises(epic.EpicError) as e:
        noalloc(g, inst.seqs, np.zeros(n, np.int32), np.zeros(n, np.int32), np.zeros(n, np.int32))
    assert e.value.code == -3
