"""Pins for the oracle's lexing and memo (CPU only)."""
import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests import refimpl
from tests.util import custom_vocab, golden

LANGS = ["arith", "json", "smiles", "clike", "tiny_ab", "tiny_kw", "tiny_expr"]


def _problem(oracle_lib, lang, vocab=None):
    return oracle_lib.problem_from(lang, vocab or custom_vocab(lang))


@pytest.mark.parametrize("row", golden("lexing.jsonl"), ids=lambda r: f"{r['lang']}:{r['text']}")
def test_golden_lexing(oracle_lib, row):
    lang = G.language(row["lang"])
    p = _problem(oracle_lib, lang)
    r = oracle_lib.lex_bytes(p, 0, row["text"].encode(), flush=True)
    if row["terms"] is None:
        assert r is None
    else:
        assert r is not None
        assert [lang.grammar.terminals[t] for t in r[0]] == row["terms"]


@pytest.mark.parametrize("name", LANGS)
def test_lexing_matches_regex_maximal_munch(oracle_lib, name):
    """Greedy lexing equals maximal munch computed with Python's regex engine
    (our lexers are free of backtracking), on rendered sentences and on random
    byte strings over the alphabet."""
    lang = G.language(name)
    p = _problem(oracle_lib, lang)
    rng = np.random.default_rng(7)
    texts = []
    for _ in range(60):
        terms = [lang.grammar.terminals[i] for i in rng.integers(0, len(lang.grammar.terminals), size=6)]
        texts.append(G.render(lang, rng, terms, extra_space=0.3)[0])
    alpha = lang.alphabet
    for _ in range(200):
        L = int(rng.integers(0, 9))
        texts.append("".join(alpha[i] for i in rng.integers(0, len(alpha), size=L)))
    agree = 0
    for t in texts:
        ours = oracle_lib.lex_bytes(p, 0, t.encode(), flush=True)
        ref = refimpl.munch_lex(name, t)
        ours_names = None if ours is None else [lang.grammar.terminals[i] for i in ours[0]]
        assert ours_names == ref, t
        agree += ref is not None
    assert agree > 20


def test_golden_memo_arith(oracle_lib):
    lang = G.language("arith")
    rows = golden("memo_arith.jsonl")
    vocab = custom_vocab(lang, [r["token"] for r in rows])
    p = _problem(oracle_lib, lang, vocab)
    assert p.Q == 8
    m = oracle_lib.memo(p)
    ids = {s: i for i, s in enumerate(vocab.strings)}
    for r in rows:
        e = m[ids[r["token"].encode()], r["q"]]
        assert int(e[0]) | (int(e[1]) << 8) == r["next"]
        assert e[2] == len(r["labels"])
        assert e[3] == r["mask"]
        assert list(e[4:4 + len(r["labels"])]) == r["labels"]
        assert not e[4 + len(r["labels"]):].any()


def test_memo_dead_entry_is_canonical(oracle_lib):
    lang = G.language("json")
    vocab = custom_vocab(lang, ["{"])
    p = _problem(oracle_lib, lang, vocab)
    _, q_in_string = oracle_lib.lex_bytes(p, 0, b'"', flush=False)
    m = oracle_lib.memo(p)
    e = m[vocab.strings.index(b"{"), q_in_string]
    assert e.tolist() == [0xFF, 0xFF] + [0] * 14


@pytest.mark.parametrize("name", ["arith", "json", "smiles", "clike"])
def test_memo_composition_law(oracle_lib, name):
    """Lexing t1.t2 from q equals memo[t2] applied after memo[t1] (labels
    concatenate, masks shift by len(t1)); and a token from the start state
    followed by a flush equals standalone lexing of its bytes."""
    inst = W.make_instance({"arith": 1, "json": 2, "smiles": 3, "clike": 4}[name], 1, B=1, n=32)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    m = oracle_lib.memo(p)
    rng = np.random.default_rng(3)
    strings = inst.vocab.strings
    for _ in range(400):
        t1, t2 = (int(v) for v in rng.integers(0, inst.vocab.size, size=2))
        q = int(rng.integers(0, p.Q))
        e1 = m[t1, q]
        nxt = int(e1[0]) | (int(e1[1]) << 8)
        both = oracle_lib.lex_bytes(p, q, strings[t1] + strings[t2], flush=False)
        if nxt == 0xFFFF:
            assert both is None
            continue
        e2 = m[t2, nxt]
        nxt2 = int(e2[0]) | (int(e2[1]) << 8)
        if nxt2 == 0xFFFF:
            assert both is None
            continue
        labels = list(e1[4:4 + e1[2]]) + list(e2[4:4 + e2[2]])
        terms = [int(x) for x in labels if x != 0xFF]
        assert both is not None and both[0] == terms and both[1] == nxt2
        assert bin(int(e1[3])).count("1") == e1[2]
    for t in range(min(inst.vocab.size, 300)):
        e = m[t, 0]
        nxt = int(e[0]) | (int(e[1]) << 8)
        alone = oracle_lib.lex_bytes(p, 0, strings[t], flush=True)
        if nxt == 0xFFFF:
            assert alone is None
            continue
        ok = oracle_lib.lex_bytes(p, nxt, b"", flush=True)
        if ok is None:
            assert alone is None
        else:
            labels = [int(x) for x in e[4:4 + e[2]] if x != 0xFF] + ok[0]
            assert alone is not None and alone[0] == labels


@pytest.mark.parametrize("name", LANGS + ["tiny_paren"])
def test_lexer_tables_are_trim_minimal_bfs(name):
    """The shared DFA input: start state 0 never accepts, every state reaches
    acceptance, states are numbered breadth-first over increasing bytes."""
    tb = G.language(name).tables
    Q = tb.num_states
    assert tb.accept[0] == -1
    live = set(np.flatnonzero(tb.accept != -1).tolist())
    changed = True
    while changed:
        changed = False
        for q in range(Q):
            if q not in live and any(int(t) in live for t in tb.trans[q] if t >= 0):
                live.add(q)
                changed = True
    assert live == set(range(Q))
    order, seen = [0], {0}
    for q in order:
        for c in range(256):
            t = int(tb.trans[q, c])
            if t >= 0 and t not in seen:
                seen.add(t)
                order.append(t)
    assert order == list(range(Q))
