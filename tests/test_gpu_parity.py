"""Bit-exact parity of the HIP path (through the C ABI) with the CPU oracle."""
import os

import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests.util import custom_vocab, pad_language

pytestmark = pytest.mark.gpu
NTH = min(16, os.cpu_count() or 1)


@pytest.fixture(scope="module")
def gpu_mod():
    import torch

    if not torch.cuda.is_available():
        pytest.fail("no GPU visible to the gpu-marked tests")
    from tests import gpu_util

    return gpu_util


_cache = {}


def setup(preset, gpu_mod, oracle_lib, seed=42):
    key = (preset, seed)
    if key not in _cache:
        inst = W.make_instance(preset, seed)
        arr = W.arrays(inst.lang, inst.vocab)
        props = inst.cfg["props"] * inst.B
        g = gpu_mod.Gpu(arr, inst.B, inst.n, max(props, 64))
        _cache[key] = (inst, g, oracle_lib.problem_from(inst.lang, inst.vocab))
    return _cache[key]


@pytest.mark.parametrize("preset", [1, 2, 3, 4, 5])
def test_memo_table_bit_exact(preset, gpu_mod, oracle_lib):
    inst, g, p = setup(preset, gpu_mod, oracle_lib)
    got = g.ctx.memo_export()
    want = oracle_lib.memo(p)
    assert got.shape == want.shape
    assert np.array_equal(got, want)


@pytest.mark.parametrize("preset", [1, 2])
def test_verdicts_all_candidates(preset, gpu_mod, oracle_lib):
    inst = W.make_instance(preset, 42)
    _, g, p = setup(preset, gpu_mod, oracle_lib)
    pr = W.propose(inst)
    got = g.validate(inst.seqs, pr.seq, pr.pos, pr.tok)
    want = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH)
    assert g.errors() == 0
    assert np.array_equal(got, want)
    assert 0 < int(want.sum()) < len(want)


@pytest.mark.parametrize("preset,reps", [(2, 5), (3, 3), (1, 6)])
def test_prefix_sharing_bit_exact(preset, reps, gpu_mod, oracle_lib):
    """More candidates than CUs: each candidate resumes from its sequence's
    base walk at the start of its masked run.  The step-1 proposals, repeated
    (with every masked position of the first sequence added, so that
    candidates sit in the first and the last run), give the same verdicts as
    the oracle's candidate-by-candidate walks."""
    inst = W.make_instance(preset, 42)
    _, g, p = setup(preset, gpu_mod, oracle_lib)
    pr = W.propose(inst)
    masked = np.flatnonzero(inst.seqs[0] == W.MASK).astype(np.int32)
    seq = np.concatenate([np.tile(pr.seq, reps), np.zeros(len(masked), np.int32)])
    pos = np.concatenate([np.tile(pr.pos, reps), masked])
    tok = np.concatenate([np.tile(pr.tok, reps), inst.hidden[0, masked].astype(np.int32)])
    assert len(seq) > 256  # the prefix-sharing launch
    g2 = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), inst.B, inst.n, len(seq))
    got = g2.validate(inst.seqs, seq, pos, tok)
    assert g2.errors() == 0
    want_u = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH)
    want_m = oracle_lib.validate_batch(p, inst.seqs, seq[-len(masked):], pos[-len(masked):], tok[-len(masked):], NTH)
    assert np.array_equal(got, np.concatenate([np.tile(want_u, reps), want_m]))


@pytest.mark.parametrize("preset", [1, 2])
def test_selection_matches_alg4(preset, gpu_mod, oracle_lib):
    inst = W.make_instance(preset, 42)
    _, g, p = setup(preset, gpu_mod, oracle_lib)
    pr = W.propose(inst)
    v = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH)
    got, counts = g.select(inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v)
    want, ocounts, status = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, NTH)
    assert status == 0 and g.errors() == 0
    assert np.array_equal(got, want)
    assert counts == ocounts


@pytest.mark.parametrize("preset", [1, 2])
def test_multistep_evolution(preset, gpu_mod, oracle_lib):
    """Every step: verdicts, selections and the committed sequences agree."""
    _, g, p = setup(preset, gpu_mod, oracle_lib)
    a, b = W.make_instance(preset, 43), W.make_instance(preset, 43)
    ra = W.run_steps(a, lambda x, pr: g.validate(x, pr.seq, pr.pos, pr.tok),
                     lambda x, pr, v: g.select(x, pr.seq, pr.pos, pr.tok, pr.conf, v)[0])
    rb = W.run_steps(b, lambda x, pr: oracle_lib.validate_batch(p, x, pr.seq, pr.pos, pr.tok, NTH),
                     lambda x, pr, v: oracle_lib.select(p, x, pr.seq, pr.pos, pr.tok, pr.conf, v, NTH)[0])
    for sa, sb in zip(ra, rb):
        assert np.array_equal(sa.seqs, sb.seqs)
        assert np.array_equal(sa.verdict, sb.verdict)
        assert np.array_equal(sa.selected, sb.selected)
    assert np.array_equal(a.seqs, b.seqs)


def test_multistep_prefix_reuse(gpu_mod, oracle_lib):
    """1024-token sequences decoded in blocks: base walks are reused across
    calls (each resumes at the last masked run before the first changed
    token) and by the selection; several steps agree with the oracle."""
    inst_g = W.make_instance(5, 44, B=6)
    inst_o = W.make_instance(5, 44, B=6)
    p = oracle_lib.problem_from(inst_g.lang, inst_g.vocab)
    g = gpu_mod.Gpu(W.arrays(inst_g.lang, inst_g.vocab), inst_g.B, inst_g.n, inst_g.B * inst_g.cfg["props"])
    ra = W.run_steps(inst_g, lambda x, pr: g.validate(x, pr.seq, pr.pos, pr.tok),
                     lambda x, pr, v: g.select(x, pr.seq, pr.pos, pr.tok, pr.conf, v)[0], steps=3)
    rb = W.run_steps(inst_o, lambda x, pr: oracle_lib.validate_batch(p, x, pr.seq, pr.pos, pr.tok, NTH),
                     lambda x, pr, v: oracle_lib.select(p, x, pr.seq, pr.pos, pr.tok, pr.conf, v, NTH)[0], steps=3)
    assert g.errors() == 0
    for sa, sb in zip(ra, rb):
        assert np.array_equal(sa.seqs, sb.seqs)
        assert np.array_equal(sa.verdict, sb.verdict)
        assert np.array_equal(sa.selected, sb.selected)


@pytest.mark.parametrize("preset,words", [(1, 2), (2, 8)])
def test_padded_grammar_item_widths(preset, words, gpu_mod, oracle_lib):
    """2- and 8-word item sets, which no workload grammar packs into: the
    workload's grammar padded with equivalent productions, verdicts and Alg. 4
    selections against the oracle on the padded grammar, and verdicts equal
    to the unpadded grammar's (the language is the same)."""
    inst = W.make_instance(preset, 42)
    pr = W.propose(inst)
    lang = pad_language(inst.lang)
    g = gpu_mod.Gpu(W.arrays(lang, inst.vocab), inst.B, inst.n, max(pr.C, 64))
    assert g.ctx.item_words == words
    p = oracle_lib.problem_from(lang, inst.vocab)
    got = g.validate(inst.seqs, pr.seq, pr.pos, pr.tok)
    want = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH)
    assert np.array_equal(got, want)
    p0 = oracle_lib.problem_from(inst.lang, inst.vocab)
    assert np.array_equal(want, oracle_lib.validate_batch(p0, inst.seqs, pr.seq, pr.pos, pr.tok, NTH))
    gs, gc = g.select(inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, want)
    ws, wc, st = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, want)
    assert st == 0 and g.errors() == 0
    assert np.array_equal(gs, ws) and gc == wc


@pytest.mark.parametrize("batch", ["alg4", "empty"])
@pytest.mark.parametrize("preset,B", [(1, None), (2, None), (3, 6), (4, 1), (5, 4)])
def test_commit_fallback_matches_oracle(preset, B, batch, gpu_mod, oracle_lib):
    """The sequential fallback after the relaxed batch, with the oracle's
    verdicts as input and a seeded commit budget per sequence; the batch is
    Alg. 4's selection, or empty (the case where the loop decides every
    commit, accepting and rejecting candidates against the updated x).  The
    candidates the device commits equal the oracle's, which checks every
    candidate it reaches (the device walks verdict-1 ones only).  The
    1024-token workload takes the launch whose checks resume from the base
    walks of the sequences."""
    import torch

    inst = W.make_instance(preset, 42, B=B)
    pr = W.propose(inst)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    v = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH)
    if batch == "alg4":
        sel, _, st = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, NTH)
        assert st == 0
    else:
        sel = np.zeros(pr.C, np.uint8)
    rng = np.random.default_rng(100 + preset)
    nc = rng.integers(1, 6 if preset == 4 else inst.cfg["props"] + 2, size=inst.B).astype(np.int32)
    want, st = oracle_lib.fallback(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, sel, nc)
    assert st == 0
    if batch == "empty":
        assert want.sum() > 0
    g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), inst.B, inst.n, max(pr.C, 64))
    acc = torch.full((pr.C,), 7, dtype=torch.uint8, device=g.dev)
    g.ctx.fallback(g.t(inst.seqs), g.t(pr.seq), g.t(pr.pos), g.t(pr.tok), g.t(pr.conf, torch.float32),
                   g.t(v, torch.uint8), g.t(sel, torch.uint8), g.t(nc), acc, g.ws)
    torch.cuda.synchronize()
    assert g.errors() == 0
    assert np.array_equal(acc.cpu().numpy(), want)


def test_commit_fallback_edge_cases(gpu_mod, oracle_lib):
    """Zero budget, a budget above the candidate count, a repeated position
    among one sequence's valid candidates (that sequence commits nothing and
    sets EPIC_DEV_BAD_SELECT, the others match the oracle), and C = 0."""
    import torch

    from paper_2606_00722_amd import epic

    inst = W.make_instance(1, 42)
    pr = W.propose(inst)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    v = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH)
    g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), inst.B, inst.n, max(pr.C, 64))
    none = np.zeros(pr.C, np.uint8)

    def run(pos, nc, C=None):
        C = pr.C if C is None else C
        acc = torch.full((max(C, 1),), 7, dtype=torch.uint8, device=g.dev)
        g.ctx.fallback(g.t(inst.seqs), g.t(pr.seq[:C]), g.t(pos[:C]), g.t(pr.tok[:C]),
                       g.t(pr.conf[:C], torch.float32), g.t(v[:C], torch.uint8), g.t(none[:C], torch.uint8),
                       g.t(nc), acc[:C], g.ws)
        torch.cuda.synchronize()
        return acc[:C].cpu().numpy()

    assert not run(pr.pos, np.zeros(inst.B, np.int32)).any() and g.errors() == 0
    big = np.full(inst.B, 64, np.int32)
    want, st = oracle_lib.fallback(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, none, big)
    assert st == 0 and want.sum() > 0
    assert np.array_equal(run(pr.pos, big), want) and g.errors() == 0
    b0 = next(b for b in range(inst.B) if ((pr.seq == b) & (v == 1)).sum() >= 2)
    c1, c2 = np.flatnonzero((pr.seq == b0) & (v == 1))[:2]
    pos2 = pr.pos.copy()
    pos2[c2] = pos2[c1]
    want2, st2 = oracle_lib.fallback(p, inst.seqs, pr.seq, pos2, pr.tok, pr.conf, v, none, big)
    assert st2 == -4 and not want2[pr.seq == b0].any()
    got2 = run(pos2, big)
    assert np.array_equal(got2, want2)
    assert g.errors() & epic.DEV_BAD_SELECT
    assert run(pr.pos, big, C=0).size == 0 and g.errors() == 0


@pytest.mark.parametrize("name,extra", [("tiny_paren", ["((", "))", "()"]), ("tiny_expr", ["a+", "(a", "a)", " a"]),
                                        ("tiny_kw", ["if", "(x", "x)", " i"]), ("tiny_ab", ["ab", "ba", "cc"]),
                                        ("arith", ["a+", "1*", "(a", " 1"])])
def test_tiny_languages(name, extra, gpu_mod, oracle_lib):
    """Small random sequences: nullable start, multi-class gaps (no
    whitespace), keyword/identifier boundaries spanning masks."""
    lang = G.language(name)
    vocab = custom_vocab(lang, extra)
    arr = W.arrays(lang, vocab)
    p = oracle_lib.problem_from(lang, vocab)
    g = gpu_mod.Gpu(arr, 64, 10, 512)
    rng = np.random.default_rng(4)
    B, n = 48, 10
    seqs = rng.integers(0, vocab.size, size=(B, n)).astype(np.int32)
    seqs[rng.random((B, n)) < 0.5] = -1
    for b in range(B):
        seqs[b, rng.integers(0, n)] = -1
    cs, cp, ct, cf = [], [], [], []
    for b in range(B):
        m = np.flatnonzero(seqs[b] == -1)
        for pos in rng.choice(m, min(len(m), 4), replace=False):
            cs.append(b), cp.append(pos), ct.append(rng.integers(0, vocab.size)), cf.append(rng.random())
    cs, cp, ct = (np.array(a, np.int32) for a in (cs, cp, ct))
    cf = np.array(cf, np.float32)
    got = g.validate(seqs, cs, cp, ct)
    want = oracle_lib.validate_batch(p, seqs, cs, cp, ct)
    assert np.array_equal(got, want)
    gs, gc = g.select(seqs, cs, cp, ct, cf, want)
    ws, wc, st = oracle_lib.select(p, seqs, cs, cp, ct, cf, want)
    assert st == 0 and g.errors() == 0
    assert np.array_equal(gs, ws) and gc == wc


def test_edge_cases(gpu_mod, oracle_lib):
    """Single-token sequences, all-masked rows, candidates at both ends, the
    longest row (every token of a 10-token row fixed but one), and C = 0."""
    lang = G.language("arith")
    vocab = custom_vocab(lang, ["a+", " 1", "((", "))"])
    arr = W.arrays(lang, vocab)
    p = oracle_lib.problem_from(lang, vocab)
    g = gpu_mod.Gpu(arr, 8, 10, 64)
    idx = {s: i for i, s in enumerate(vocab.strings)}
    rows = [[-1] * 10, [-1] + [idx[b"a"]] * 9, [idx[b"("]] * 9 + [-1], [-1, idx[b"a+"], -1, -1, idx[b"))"], -1, -1, -1, -1, -1]]
    seqs = np.array(rows, np.int32)
    cs = np.array([0, 0, 1, 2, 3, 3], np.int32)
    cp = np.array([0, 9, 0, 9, 0, 9], np.int32)
    ct = np.array([idx[b"a"], idx[b")"], idx[b"("], idx[b")"], idx[b"(("], idx[b"1"]], np.int32)
    got = g.validate(seqs, cs, cp, ct)
    want = oracle_lib.validate_batch(p, seqs, cs, cp, ct)
    assert np.array_equal(got, want)
    one = np.array([[-1]], np.int32)
    for t in range(vocab.size):
        assert g.validate(one, [0], [0], [t])[0] == oracle_lib.validate_batch(p, one, [0], [0], [t])[0]
    assert g.validate(seqs, np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32)).size == 0


def test_malformed_candidates_and_host_errors(gpu_mod, oracle_lib):
    from paper_2606_00722_amd import epic

    inst, g, p = setup(1, gpu_mod, oracle_lib)
    x = inst.seqs
    fixed = int(np.flatnonzero(x[0] != -1)[0])
    masked = int(np.flatnonzero(x[0] == -1)[0])
    seq = [0, 0, 5, 0, 0, -1]
    pos = [fixed, masked, masked, 999, masked, masked]
    tok = [1, inst.vocab.size, 1, 1, 3, 3]
    got = g.validate(x, seq, pos, tok)
    assert got.tolist()[:4] == [2, 2, 2, 2] and got[5] == 2
    assert got[4] == oracle_lib.validate_batch(p, x, [0], [masked], [3])[0]
    assert g.errors() & epic.DEV_BAD_CANDIDATE
    assert g.errors() == 0  # reading clears
    with pytest.raises(epic.EpicError) as e:  # more candidates than the context was sized for
        n = 10_000
        g.validate(x, np.zeros(n, np.int32), np.full(n, masked, np.int32), np.zeros(n, np.int32))
    assert e.value.code == -3
    # duplicate positions among valid candidates: nothing selected, flag set
    v = np.array([1, 1], np.uint8)
    sel, _ = g.select(x, [0, 0], [masked, masked], [3, 4], [0.5, 0.4], v)
    assert sel.tolist() == [0, 0] and g.errors() & epic.DEV_BAD_SELECT


def test_deterministic(gpu_mod, oracle_lib):
    inst = W.make_instance(2, 42)
    _, g, p = setup(2, gpu_mod, oracle_lib)
    pr = W.propose(inst)
    a = g.validate(inst.seqs, pr.seq, pr.pos, pr.tok)
    b = g.validate(inst.seqs, pr.seq, pr.pos, pr.tok)
    assert np.array_equal(a, b)
    sa, _ = g.select(inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, a)
    sb, _ = g.select(inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, a)
    assert np.array_equal(sa, sb)


def test_two_contexts_share_one_workspace(gpu_mod, oracle_lib):
    """Walk records carry an owner tag derived from the context's tables and
    workspace layout: two contexts with different grammars (JSON-like and
    arithmetic) alternate over one workspace, each with more candidates than
    CUs so that its base walks record and later calls resume, and every call
    agrees with the oracle."""
    import torch

    runs = []
    for preset in (2, 1):
        inst = W.make_instance(preset, 42)
        pr = W.propose(inst)
        reps = 300 // pr.C + 1
        cand = (np.tile(pr.seq, reps), np.tile(pr.pos, reps), np.tile(pr.tok, reps))
        g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), inst.B, inst.n, len(cand[0]))
        p = oracle_lib.problem_from(inst.lang, inst.vocab)
        want = np.tile(oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, NTH), reps)
        runs.append((inst, g, cand, want))
    ws = torch.zeros(max(r[1].ctx.workspace_bytes for r in runs) + 256, dtype=torch.uint8, device=runs[0][1].dev)
    for r in runs:
        r[1].ws = ws
    for _ in range(3):
        for inst, g, cand, want in runs:
            assert np.array_equal(g.validate(inst.seqs, *cand), want)
            assert g.errors() == 0


def test_more_than_64_valid_candidates(gpu_mod, oracle_lib):
    """The device keeps a sequence's candidates in 64-bit subsets: with more
    than 64 verdict-1 candidates in one sequence, the selection and the
    fallback commit nothing for it and set EPIC_DEV_CAPACITY (the oracle has
    no such limit)."""
    from paper_2606_00722_amd import epic

    inst = W.make_instance(1, 42, B=1, n=200)
    masked = np.flatnonzero(inst.seqs[0] == W.MASK).astype(np.int32)
    C = len(masked)
    assert C > 64
    seq = np.zeros(C, np.int32)
    tok = inst.hidden[0, masked].astype(np.int32)
    conf = np.random.default_rng(7).random(C, dtype=np.float32)
    v = np.ones(C, np.uint8)
    g = gpu_mod.Gpu(W.arrays(inst.lang, inst.vocab), 1, 200, C)
    sel, _ = g.select(inst.seqs, seq, masked, tok, conf, v)
    assert not sel.any() and g.errors() & epic.DEV_CAPACITY
    acc = g.fallback(inst.seqs, seq, masked, tok, conf, v, np.zeros(C, np.uint8), np.array([70], np.int32))
    assert not acc.any() and g.errors() & epic.DEV_CAPACITY
    # 64 of them are within the limit: the fallback commits like the oracle
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    k = 64
    acc = g.fallback(inst.seqs, seq[:k], masked[:k], tok[:k], conf[:k], v[:k], np.zeros(k, np.uint8),
                     np.array([40], np.int32))
    want, st = oracle_lib.fallback(p, inst.seqs, seq[:k], masked[:k], tok[:k], conf[:k], v[:k],
                                   np.zeros(k, np.uint8), [40])
    assert st == 0 and g.errors() == 0
    assert np.array_equal(acc, want) and int(want.sum()) == 40
