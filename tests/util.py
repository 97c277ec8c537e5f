"""Small shared test helpers (no validity arithmetic)."""
from __future__ import annotations

import json
import os
from typing import List, Optional, Sequence

import numpy as np

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def golden(name: str):
    with open(os.path.join(GOLDEN, name)) as f:
        rows = [json.loads(l) for l in f if l.strip()]
    return [r for r in rows if "_comment" not in r]


def custom_vocab(lang: G.Language, extra: Sequence[str] = ()) -> W.Vocab:
    """Single bytes of the alphabet first, then `extra` strings."""
    singles = sorted(set(lang.alphabet.encode()))
    strings = [bytes([c]) for c in singles]
    for s in extra:
        b = s.encode()
        if b not in strings:
            strings.append(b)
    return W.Vocab(strings)


def encode(vocab: W.Vocab, toks: Sequence[Optional[str]]) -> np.ndarray:
    idx = {s: i for i, s in enumerate(vocab.strings)}
    return np.array([-1 if t is None else idx[t.encode()] for t in toks], dtype=np.int32)


def pad_language(lang: G.Language) -> G.Language:
    """The same language with a larger grammar: every nonterminal A gets a
    fresh A' with A -> A' and A' -> each right-hand side of A.  L(G) is
    unchanged (A derives exactly what it did), while the dotted items grow
    enough to pack into more item words.  Terminals and their ids, hence the
    lexer, stay as they are."""
    import dataclasses

    g = lang.grammar
    extra_nts = [a + "'" for a in g.nonterminals]
    prods = list(g.productions)
    for a in g.nonterminals:
        prods.append((a, (a + "'",)))
        prods.extend((a + "'", rhs) for lhs, rhs in g.productions if lhs == a)
    pg = G.Grammar(list(g.terminals), list(g.nonterminals) + extra_nts, prods, g.start)
    return dataclasses.replace(lang, name=lang.name + "_padded", grammar=pg)


def packed_words(g: G.Grammar) -> int:
    """Item words of a grammar as the library packs it: productions (|rhs|+1
    items, plus 2 for the augmented start) first-fit by decreasing size into
    32-bit words, rounded up to a power of two."""
    bins: List[int] = []
    for s in sorted([len(r) + 1 for _, r in g.productions] + [2], reverse=True):
        for i, b in enumerate(bins):
            if b + s <= 32:
                bins[i] += s
                break
        else:
            bins.append(s)
    w = 1
    while w < len(bins):
        w *= 2
    return w


def fill(vocab_strings, x, gaps) -> bytes:
    """The bytes of x with its j-th maximal masked run replaced by gaps[j]."""
    out, g, prev_masked = [], 0, False
    for t in x:
        if t < 0:
            if not prev_masked:
                out.append(gaps[g])
                g += 1
            prev_masked = True
        else:
            out.append(vocab_strings[int(t)])
            prev_masked = False
    assert g == len(gaps)
    return b"".join(out)
