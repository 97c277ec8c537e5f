"""Pins for the oracle's relaxed compatible-subset selection (Alg. 4, CPU only)."""
import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests.util import custom_vocab, encode


def _run(oracle_lib, lang_name, x_toks, cands):
    """cands: list of (pos, token string, confidence)."""
    lang = G.language(lang_name)
    vocab = custom_vocab(lang, [c[1] for c in cands] + [t for t in x_toks if t is not None])
    p = oracle_lib.problem_from(lang, vocab)
    x = encode(vocab, x_toks)[None, :]
    seq = np.zeros(len(cands), np.int32)
    pos = np.array([c[0] for c in cands], np.int32)
    tok = encode(vocab, [c[1] for c in cands])
    conf = np.array([c[2] for c in cands], np.float32)
    v = oracle_lib.validate_batch(p, x, seq, pos, tok)
    sel, stats, status = oracle_lib.select(p, x, seq, pos, tok, conf, v)
    return v, sel, stats, status


def test_worked_example_cover_false_positive_then_shrink(oracle_lib):
    """x = four masks; '(' '(' 'a' ')' at positions 0..3 with confidences
    .9 .8 .7 .6.  '((a)' passes the cover but not the exact check; the left
    half '((' is exact-valid; the right half is cover-compatible after it but
    fails exactly and shrinks to singletons, which are dropped.  B = {c0, c1}:
    2 cover calls, 3 exact calls."""
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 4,
                                 [(0, "(", .9), (1, "(", .8), (2, "a", .7), (3, ")", .6)])
    assert status == 0 and v.tolist() == [1, 1, 1, 1]
    assert sel.tolist() == [1, 1, 0, 0]
    assert stats == (2, 3)


def test_all_compatible_ties_keep_everything(oracle_lib):
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 5,
                                 [(0, "a", .5), (1, "+", .5), (2, "b", .5), (3, "*", .5), (4, "c", .5)])
    assert status == 0 and v.tolist() == [1] * 5
    assert sel.tolist() == [1] * 5 and stats == (1, 1)


def test_invalid_candidates_are_not_considered_and_exact_shrinks_to_nothing(oracle_lib):
    """'(' at the end is invalid on its own and is filtered out; 'a' ')' passes
    the cover but not the exact check, splits into singletons: B is empty."""
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 3, [(0, "a", .9), (1, ")", .8), (2, "(", .7)])
    assert v.tolist() == [1, 1, 0]
    assert sel.tolist() == [0, 0, 0] and stats == (1, 1) and status == 0


def test_cover_rejection_recurses_on_halves(oracle_lib):
    """'1a+2' fails the cover (NUM ID); the left half '1a' fails too and splits
    into singletons; the right half '+2' after nothing passes the cover and
    the exact check: B = {c2, c3}, with 3 cover calls and 1 exact call."""
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 4,
                                 [(0, "1", .9), (1, "a", .8), (2, "+", .7), (3, "2", .6)])
    assert v.tolist() == [1, 1, 1, 1]
    assert sel.tolist() == [0, 0, 1, 1] and stats == (3, 1) and status == 0


def test_confidence_order_not_index_order(oracle_lib):
    """The same four candidates as the worked example with confidences
    reversed: sorted order is c3, c2, c1, c0, so the halves are {')','a'} and
    {'(','('}.  Σ* 'a' ')' is exact-valid after nothing: B = {c2, c3}."""
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 4,
                                 [(0, "(", .6), (1, "(", .7), (2, "a", .8), (3, ")", .9)])
    assert v.tolist() == [1, 1, 1, 1]
    assert sel.tolist()[2:] == [1, 1]
    assert status == 0


def test_duplicate_positions_and_nan_are_rejected(oracle_lib):
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 3, [(0, "a", .9), (0, "b", .8)])
    assert v.tolist() == [1, 1] and status == -4 and sel.tolist() == [0, 0]
    v, sel, stats, status = _run(oracle_lib, "arith", [None] * 3, [(0, "a", float("nan")), (1, "+", .8)])
    assert status == -4 and sel.tolist() == [0, 0]


@pytest.mark.parametrize("preset,n", [(1, 32), (2, 64)])
def test_selection_invariants(oracle_lib, preset, n):
    """B is a subset of the individually valid candidates, is empty or has at
    least two elements, and x + B is exact-valid (App. D.4).  If the whole
    valid set passes both checks, B is all of it."""
    inst = W.make_instance(preset, 17, B=4, n=n)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    nonempty = 0
    for _ in range(2):
        pr = W.propose(inst)
        v = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok)
        sel, stats, status = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v)
        assert status == 0
        for b in range(inst.B):
            idx = np.flatnonzero(pr.seq == b)
            chosen = idx[sel[idx] == 1]
            valid = idx[v[idx] == 1]
            assert set(chosen) <= set(valid)
            assert chosen.size == 0 or chosen.size >= 2
            if chosen.size:
                nonempty += 1
                y = inst.seqs[b].copy()
                y[pr.pos[chosen]] = pr.tok[chosen]
                assert oracle_lib.valid(p, y) == 1
            if valid.size >= 2:
                y = inst.seqs[b].copy()
                y[pr.pos[valid]] = pr.tok[valid]
                if oracle_lib.valid(p, y) == 1:
                    assert set(chosen) == set(valid)
        W.commit(inst, pr, v, sel)
    assert nonempty >= 1


@pytest.mark.parametrize("preset,n", [(1, 32), (2, 64), (3, 64), (5, 96)])
def test_checks_are_monotone_in_the_filled_positions(oracle_lib, preset, n):
    """A masked run reads any bytes (R1), so filling more masked positions
    only shrinks the character language of x, and the regular cover's
    language contains L(G).  Hence, for candidate sets T ⊆ S of one
    sequence: x + S exact-valid => x + T exact-valid; x + S cover-valid =>
    x + T cover-valid; x + S exact-valid => x + S cover-valid.  The device
    selection answers a check that an answered check decides this way
    without walking it; the oracle never does, so this pins the property on
    the oracle's own checks."""
    rng = np.random.default_rng(5)
    inst = W.make_instance(preset, 23, B=6, n=n)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    seen = {(k, r): 0 for k in ("e", "c") for r in (0, 1)}
    for _ in range(2):
        pr = W.propose(inst)
        v = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok)
        for b in range(inst.B):
            idx = np.flatnonzero((pr.seq == b) & (v == 1))
            if idx.size < 2:
                continue
            for _ in range(6):
                S = idx[rng.random(idx.size) < 0.7]
                T = S[rng.random(S.size) < 0.5]
                res = {}
                for name, sub in (("S", S), ("T", T)):
                    y = inst.seqs[b].copy()
                    y[pr.pos[sub]] = pr.tok[sub]
                    res[name] = (oracle_lib.valid(p, y), oracle_lib.cover(p, y))
                for k, i in (("e", 0), ("c", 1)):
                    seen[(k, res["S"][i])] += 1
                    if res["S"][i] == 1:
                        assert res["T"][i] == 1, (preset, b, S, T, k)
                if res["S"][0] == 1:
                    assert res["S"][1] == 1
                if res["T"][1] == 0:
                    assert res["T"][0] == 0
        W.commit(inst, pr, v, oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v)[0])
    assert sum(seen.values()) >= 20, seen
    if preset == 2:  # the JSON-like workload's subsets fail both checks too
        assert all(seen[(k, r)] for k in ("e", "c") for r in (0, 1)), seen
