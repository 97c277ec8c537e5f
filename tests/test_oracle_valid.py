"""Pins for the oracle's Valid and relaxed (cover) checks (CPU only)."""
import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests import refimpl
from tests.util import custom_vocab, encode, golden


@pytest.mark.parametrize("row", golden("valid_cover.jsonl"), ids=lambda r: f"{r['lang']}:{r['x']}")
def test_golden_valid_and_cover(oracle_lib, row):
    lang = G.language(row["lang"])
    vocab = custom_vocab(lang, [t for t in row["x"] if t is not None])
    p = oracle_lib.problem_from(lang, vocab)
    x = encode(vocab, row["x"])
    assert oracle_lib.valid(p, x) == row["valid"], row["why"]
    if row["cover"] is not None:
        assert oracle_lib.cover(p, x) == row["cover"], row["why"]


def _instance(preset, seed=5, B=3, n=None):
    return W.make_instance(preset, seed, B=B, n=n)


@pytest.mark.parametrize("preset,n", [(1, 32), (2, 64), (3, 48), (4, 40)])
def test_unmasked_reduces_to_cfg_membership(oracle_lib, preset, n):
    """Fully unmasked x: Valid(x) = [lex(x) defined and in L(G)], decided here
    by regex maximal munch plus CYK-style recognition (Sec. 3 with M(x) empty)."""
    inst = _instance(preset, n=n)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    rng = np.random.default_rng(11)
    seqs = [inst.hidden[b] for b in range(inst.B)]
    for b in range(inst.B):  # corrupt one or two tokens: mostly invalid sequences
        for _ in range(4):
            x = inst.hidden[b].copy()
            for _ in range(int(rng.integers(1, 3))):
                x[rng.integers(0, len(x))] = rng.integers(0, inst.vocab.size)
            seqs.append(x)
    seen = set()
    for x in seqs:
        text = b"".join(inst.vocab.strings[t] for t in x).decode()
        toks = refimpl.munch_lex(inst.lang.name, text)
        want = int(toks is not None and refimpl.derives(inst.lang.grammar, toks))
        seen.add(want)
        assert oracle_lib.valid(p, x) == want, text
    assert seen == {0, 1}


@pytest.mark.parametrize("name", ["arith", "json", "smiles", "clike", "tiny_ab", "tiny_kw", "tiny_paren"])
def test_all_masked_is_valid(oracle_lib, name):
    lang = G.language(name)
    p = oracle_lib.problem_from(lang, custom_vocab(lang))
    for n in (1, 3, 10):
        assert oracle_lib.valid(p, np.full(n, -1, np.int32)) == 1
        assert oracle_lib.cover(p, np.full(n, -1, np.int32)) == 1


@pytest.mark.parametrize("preset", [1, 2, 3])
def test_monotone_under_unmasking(oracle_lib, preset):
    """R_{x+D} is contained in R_x, so Valid(x+D) = 1 implies Valid(x) = 1, and
    likewise for the cover check."""
    inst = _instance(preset, seed=9, B=2, n={1: 32, 2: 64, 3: 48}[preset])
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    rng = np.random.default_rng(5)
    for b in range(inst.B):
        x = inst.seqs[b].copy()
        for _ in range(6):
            masked = np.flatnonzero(x == -1)
            if masked.size == 0:
                break
            y = x.copy()
            pos = rng.choice(masked, min(3, masked.size), replace=False)
            y[pos] = np.where(rng.random(pos.size) < 0.5, inst.hidden[b, pos], rng.integers(0, inst.vocab.size, pos.size))
            vy, vx = oracle_lib.valid(p, y), oracle_lib.valid(p, x)
            assert not (vy == 1 and vx == 0)
            cy, cx = oracle_lib.cover(p, y), oracle_lib.cover(p, x)
            assert not (cy == 1 and cx == 0)
            assert not (vy == 1 and cy == 0)  # cover is a relaxation
            x = y if vy else x


def _tiny_cases(name, count, n_max, seed):
    lang = G.language(name)
    extra = {"tiny_expr": ["a+", "(a", "a)", " a"], "tiny_kw": ["if", "(x", "x)", " i"],
             "tiny_ab": ["ab", "ba", "cc"], "tiny_paren": ["((", "))", "()"], "arith": ["a+", "1*", "(a"]}[name]
    vocab = custom_vocab(lang, extra)
    rng = np.random.default_rng(seed)
    xs = []
    for _ in range(count):
        n = int(rng.integers(1, n_max + 1))
        x = rng.integers(0, vocab.size, size=n).astype(np.int32)
        x[rng.random(n) < 0.4] = -1
        xs.append(x)
    return lang, vocab, xs


@pytest.mark.parametrize("name", ["tiny_paren", "tiny_expr", "tiny_kw", "tiny_ab", "arith"])
def test_matches_bar_hillel_intersection(oracle_lib, name):
    """Second oracle: the prior pipeline's criterion as productive triples of
    the intersection grammar (App. A.2), over an automaton built in Python."""
    lang, vocab, xs = _tiny_cases(name, 40, 5, 21)
    p = oracle_lib.problem_from(lang, vocab)
    seen = set()
    for x in xs:
        want = int(refimpl.bar_hillel_valid(lang, vocab.strings, x))
        seen.add(want)
        assert oracle_lib.valid(p, x) == want, x
    assert seen == {0, 1}


@pytest.mark.parametrize("name,alpha,K", [("tiny_paren", "()", 6), ("tiny_ab", "abc", 4),
                                          ("tiny_kw", "fix() ", 3), ("tiny_expr", "a+() ", 3)])
def test_brute_force_fillings(oracle_lib, name, alpha, K):
    """Enumerated fillings of the masks: a filling that lexes into L(G) implies
    Valid = 1; and Valid = 0 implies that no filling up to K bytes works."""
    lang, vocab, xs = _tiny_cases(name, 25, 4, 33)
    p = oracle_lib.problem_from(lang, vocab)
    hits = 0
    for x in xs:
        bf = refimpl.brute_valid(lang, vocab.strings, x, alpha, K)
        v = oracle_lib.valid(p, x)
        if bf:
            assert v == 1, x
            hits += 1
        if v == 0:
            assert not bf
    assert hits > 3


@pytest.mark.parametrize("preset", [1, 2, 3, 4])
def test_cover_accepts_every_sentence(oracle_lib, preset):
    """L(G) is contained in L(F_G) (App. D.3): generated sentences, unmasked."""
    inst = _instance(preset, seed=3, B=3, n={1: 32, 2: 64, 3: 64, 4: 48}[preset])
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    for b in range(inst.B):
        assert oracle_lib.cover(p, inst.hidden[b]) == 1


def test_cover_is_exact_for_right_linear_grammar(oracle_lib):
    """For a right-linear grammar every call is a tail call, so flattening
    loses nothing: Relaxed = Valid."""
    from paper_2606_00722_amd import lexspec as lx

    prods = G._P("""
        S -> LP A | ID B | eps
        A -> RP S | ID A
        B -> PLUS S | ID
        """)
    g = G.Grammar(["PLUS", "LP", "RP", "ID"], G._nonterminals(prods), prods, "S")
    rules = [lx.LexerRule("PLUS", lx.lit("+"), 0), lx.LexerRule("LP", lx.lit("("), 1),
             lx.LexerRule("RP", lx.lit(")"), 2), lx.LexerRule("ID", lx.plus(lx.cls("a")), 3),
             lx.LexerRule("WS", lx.plus(lx.lit(" ")), lx.SKIP)]
    lang = G.Language("rl", g, rules, "a+() ", {})
    vocab = custom_vocab(lang, ["a+", "(a", "a)"])
    p = oracle_lib.problem_from(lang, vocab)
    rng = np.random.default_rng(2)
    seen = set()
    for _ in range(150):
        n = int(rng.integers(1, 7))
        x = rng.integers(0, vocab.size, size=n).astype(np.int32)
        x[rng.random(n) < 0.3] = -1
        v, c = oracle_lib.valid(p, x), oracle_lib.cover(p, x)
        assert v == c, x
        seen.add(v)
    assert seen == {0, 1}


def test_validate_batch_flags_malformed_candidates(oracle_lib):
    inst = _instance(1, B=2)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    x = inst.seqs
    fixed = int(np.flatnonzero(x[0] != -1)[0])
    masked = int(np.flatnonzero(x[0] == -1)[0])
    seq = [0, 0, 5, 0, 0, -1]
    pos = [fixed, masked, masked, 999, masked, masked]
    tok = [1, inst.vocab.size, 1, 1, 3, 3]
    v = oracle_lib.validate_batch(p, x, seq, pos, tok)
    assert v[:4].tolist() == [2, 2, 2, 2] and v[5] == 2
    assert v[4] in (0, 1)
