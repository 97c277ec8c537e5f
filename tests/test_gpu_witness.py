"""Witness extraction on the device (failure recovery, Sec. 4), through the C
ABI.  Several completions can be correct, so the device's completion is not
compared with the oracle's: its status must equal the oracle's Valid, and with
status 1 the sequence with every masked run replaced by the device's bytes must
keep the fixed tokens and lex into a sentence of L(G), checked by the oracle's
Valid on the plain byte string, and on short texts also by regex maximal munch
with CYK recognition (tests/refimpl.py)."""
import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests import refimpl
from tests.util import custom_vocab, fill

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu_mod():
    import torch

    if not torch.cuda.is_available():
        pytest.fail("no GPU visible to the gpu-marked tests")
    from tests import gpu_util

    return gpu_util


def run_witness(gpu_mod, lang, vocab, seqs, max_cands=64, lds=None):
    import torch

    B, n = seqs.shape
    g = gpu_mod.Gpu(W.arrays(lang, vocab), B, n, max(max_cands, B))
    if lds is not None:
        g.ctx.set_witness_lds(*lds)
    wws = g.ctx.alloc_witness_workspace(B, g.dev)
    cap, max_gaps = 1 << 14, n
    out = torch.zeros((B, cap), dtype=torch.uint8, device=g.dev)
    lens = torch.zeros((B, max_gaps), dtype=torch.int32, device=g.dev)
    st = torch.full((B,), 9, dtype=torch.int32, device=g.dev)
    g.ctx.witness(g.t(seqs), out, lens, st, wws, g.ws)
    torch.cuda.synchronize()
    st, out, lens = st.cpu().numpy(), out.cpu().numpy(), lens.cpu().numpy()
    res = []
    for b in range(B):
        ngaps = sum(1 for i in range(n) if seqs[b, i] < 0 and (i == 0 or seqs[b, i - 1] >= 0))
        gaps, k = [], 0
        for j in range(ngaps):
            gaps.append(bytes(out[b, k:k + lens[b, j]]))
            k += int(lens[b, j])
        res.append((int(st[b]), gaps))
    return res, g.errors()


def check(oracle_lib, p, lang, strings, x, st, gaps, independent):
    want = oracle_lib.valid(p, x)
    assert st == want, (x, st, want)
    if st != 1:
        return
    text = fill(strings, x, gaps)
    assert oracle_lib.valid_text(p, text) == 1, (x, gaps)
    if independent:
        toks = refimpl.munch_lex(lang.name, text.decode("latin-1"))
        assert toks is not None and refimpl.derives(lang.grammar, toks), (x, gaps, text)


@pytest.mark.parametrize("preset", [1, 2, 3, 4, 5])
def test_witness_workload_sequences(preset, gpu_mod, oracle_lib):
    """The step-1 partial outputs of each workload (all completable), plus
    corrupted copies of some (a fixed token replaced: mostly not completable)."""
    inst = W.make_instance(preset, 42, B={1: 4, 2: 8, 3: 8, 4: 6, 5: 6}[preset])
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    rng = np.random.default_rng(preset)
    bad = inst.seqs.copy()
    for b in range(inst.B):
        fixed = np.flatnonzero(bad[b] >= 0)
        bad[b, rng.choice(fixed, 2, replace=False)] = rng.integers(0, inst.vocab.size, 2)
    seqs = np.concatenate([inst.seqs, bad]).astype(np.int32)
    res, err = run_witness(gpu_mod, inst.lang, inst.vocab, seqs)
    assert err == 0
    sts = []
    for b in range(seqs.shape[0]):
        st, gaps = res[b]
        sts.append(st)
        check(oracle_lib, p, inst.lang, inst.vocab.strings, seqs[b], st, gaps, independent=preset <= 2)
    assert all(s == 1 for s in sts[:inst.B])


def test_witness_search_state_placement(gpu_mod, oracle_lib):
    """Where the witness search keeps its state (the back-trace's proof index:
    LDS throughout, moved to the workspace after 300 proofs, or the workspace
    from the start; the byte search's visited sets: LDS or the workspace) does
    not change the outcome: the statuses are equal and every completion
    parses.  (The bytes themselves can differ from call to call: the byte
    search's breadth-first records are appended by many threads at once.)"""
    inst = W.make_instance(3, 42, B=6)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    seqs = inst.seqs.astype(np.int32)
    for lds in (None, (300, 4096), (0, 0), (8192, 0)):
        res, err = run_witness(gpu_mod, inst.lang, inst.vocab, seqs, lds=lds)
        assert err == 0
        for b in range(seqs.shape[0]):
            st, gaps = res[b]
            check(oracle_lib, p, inst.lang, inst.vocab.strings, seqs[b], st, gaps, independent=False)
            assert st == 1, (lds, b)


def test_witness_lds_range(gpu_mod):
    from paper_2606_00722_amd import epic

    inst = W.make_instance(1, 42, B=2)
    g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), 2, inst.n, 64)
    for bad in ((-1, 0), (8193, 0), (0, -1), (0, 4097)):
        with pytest.raises(epic.EpicError):
            g.ctx.set_witness_lds(*bad)
    g.ctx.set_witness_lds(8192, 4096)
    g.ctx.set_witness_lds(0, 0)


@pytest.mark.parametrize("name", ["tiny_paren", "tiny_expr", "tiny_kw", "tiny_ab", "arith"])
def test_witness_tiny_languages(name, gpu_mod, oracle_lib):
    """Random short sequences over tiny languages (nullable start, three-class
    masked runs, keywords against identifiers), masks anywhere: status equals
    Valid and every completion parses."""
    lang = G.language(name)
    extra = {"tiny_expr": ["a+", "(a", "a)", " a"], "tiny_kw": ["if", "(x", "x)", " i"],
             "tiny_ab": ["ab", "ba", "cc"], "tiny_paren": ["((", "))", "()"], "arith": ["a+", "1*", "(a", " 1"]}[name]
    vocab = custom_vocab(lang, extra)
    rng = np.random.default_rng(77)
    n = 6
    seqs = rng.integers(0, vocab.size, size=(48, n)).astype(np.int32)
    seqs[rng.random(seqs.shape) < 0.4] = -1
    seqs[0] = -1  # all masked
    p = oracle_lib.problem_from(lang, vocab)
    res, err = run_witness(gpu_mod, lang, vocab, seqs)
    assert err == 0
    seen = set()
    for b in range(seqs.shape[0]):
        st, gaps = res[b]
        seen.add(st)
        check(oracle_lib, p, lang, vocab.strings, seqs[b], st, gaps, independent=True)
    assert seen == {0, 1}
