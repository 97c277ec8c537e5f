"""Pins for the oracle's witness (Sec. 4, failure recovery: the output of a
valid partial sequence is completed from a witness), CPU only.

A witness gives one byte string per maximal masked run.  It is checked with
procedures that share nothing with the oracle: the fixed tokens are kept, the
filled text is lexed by regex maximal munch and recognised by CYK-style
derivation (tests/refimpl.py), and it must be a sentence of L(G).  A witness
exists exactly when Valid holds, and every filling found by enumeration
implies one."""
import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests import refimpl
from tests.util import custom_vocab, fill


def check_witness(oracle_lib, p, lang, strings, x):
    st, gaps = oracle_lib.witness(p, x)
    v = oracle_lib.valid(p, x)
    assert st in (0, 1), st
    assert st == v, (x, st, v)
    if st == 1:
        assert len(gaps) == sum(1 for i, t in enumerate(x) if t < 0 and (i == 0 or x[i - 1] >= 0))
        text = fill(strings, x, gaps).decode("latin-1")
        toks = refimpl.munch_lex(lang.name, text)
        assert toks is not None and refimpl.derives(lang.grammar, toks), (x, gaps, text)
    return st


def _tiny(name, count, n_max, seed):
    lang = G.language(name)
    extra = {"tiny_expr": ["a+", "(a", "a)", " a"], "tiny_kw": ["if", "(x", "x)", " i"],
             "tiny_ab": ["ab", "ba", "cc"], "tiny_paren": ["((", "))", "()"], "arith": ["a+", "1*", "(a", " 1"]}[name]
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
def test_witness_iff_valid_and_parses(oracle_lib, name):
    """Random short sequences over tiny languages (masks at random places,
    runs at both ends): a witness is returned exactly for the valid ones, and
    each keeps the fixed tokens and lexes into L(G)."""
    lang, vocab, xs = _tiny(name, 60, 6, 41)
    p = oracle_lib.problem_from(lang, vocab)
    seen = {check_witness(oracle_lib, p, lang, vocab.strings, x) for x in xs}
    assert seen == {0, 1}


@pytest.mark.parametrize("name,alpha,K", [("tiny_paren", "()", 6), ("tiny_ab", "abc", 4), ("tiny_expr", "a+() ", 3)])
def test_witness_when_a_filling_exists(oracle_lib, name, alpha, K):
    """Every sequence for which enumeration finds a filling of at most K bytes
    has a witness; the witness itself parses."""
    lang, vocab, xs = _tiny(name, 30, 4, 57)
    p = oracle_lib.problem_from(lang, vocab)
    found = 0
    for x in xs:
        if refimpl.brute_valid(lang, vocab.strings, x, alpha, K):
            found += 1
            assert check_witness(oracle_lib, p, lang, vocab.strings, x) == 1
    assert found > 0


@pytest.mark.parametrize("name", ["arith", "json", "tiny_kw", "tiny_paren"])
def test_all_masked_witness_is_a_sentence(oracle_lib, name):
    """All positions masked: the witness is one byte string, a sentence of
    L(G) once lexed."""
    lang = G.language(name)
    vocab = custom_vocab(lang)
    p = oracle_lib.problem_from(lang, vocab)
    for n in (1, 4):
        x = np.full(n, -1, np.int32)
        assert check_witness(oracle_lib, p, lang, vocab.strings, x) == 1


def test_unmasked_valid_has_empty_witness(oracle_lib):
    """No masks: a valid sequence's witness fills nothing."""
    inst = W.make_instance(1, 7, B=2, n=16)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    for b in range(inst.B):
        st, gaps = oracle_lib.witness(p, inst.hidden[b])
        assert st == 1 and gaps == []


def test_workload_sequences(oracle_lib):
    """Partially masked sequences of the arithmetic workload (32 tokens, half
    masked) and of a short JSON-like one: every step-1 sequence is valid and
    its witness parses; corrupting a fixed token gives invalid ones too."""
    for preset, n in ((1, 32), (2, 24)):
        inst = W.make_instance(preset, 3, B=3, n=n)
        p = oracle_lib.problem_from(inst.lang, inst.vocab)
        rng = np.random.default_rng(preset)
        seen = set()
        for b in range(inst.B):
            x = inst.seqs[b]
            assert check_witness(oracle_lib, p, inst.lang, inst.vocab.strings, x) == 1
            for _ in range(3):
                y = x.copy()
                fixed = np.flatnonzero(y >= 0)
                if fixed.size:
                    y[rng.choice(fixed)] = rng.integers(0, inst.vocab.size)
                seen.add(check_witness(oracle_lib, p, inst.lang, inst.vocab.strings, y))
        assert 1 in seen


@pytest.mark.parametrize("preset,n", [(1, 24), (2, 32), (3, 24)])
def test_valid_text_is_lexing_then_cyk(oracle_lib, preset, n):
    """Valid of a plain byte string (what a completed output is checked with):
    equal to regex maximal munch followed by CYK-style recognition, on the
    hidden sentences of a workload and on corrupted copies of them."""
    inst = W.make_instance(preset, 11, B=3, n=n)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    rng = np.random.default_rng(preset)
    seen = set()
    for b in range(inst.B):
        text = b"".join(inst.vocab.strings[t] for t in inst.hidden[b])
        for k in range(4):
            t2 = bytearray(text)
            if k:
                t2[int(rng.integers(0, len(t2)))] = int(rng.choice(list(set(text))))
            toks = refimpl.munch_lex(inst.lang.name, t2.decode("latin-1"))
            want = int(toks is not None and refimpl.derives(inst.lang.grammar, toks))
            seen.add(want)
            assert oracle_lib.valid_text(p, bytes(t2)) == want
    assert seen == {0, 1}
