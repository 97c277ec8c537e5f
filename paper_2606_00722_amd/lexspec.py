"""Lexer specifications compiled to the trim, minimal lexer DFA both sides consume.

The paper's lexical map (Sec. 3, "Problem Formulation") turns bytes into grammar
terminals; Alg. 1 compiles it once before decoding.  This module is that
compile step, written as plain textbook automata code:

* patterns are small regular-expression trees built with the combinators below;
* Thompson construction gives an NFA, subset construction a DFA;
* an accepting DFA state takes the label of the earliest-listed rule it accepts
  (priority to the earlier rule);
* Moore partition refinement minimises, states that cannot reach acceptance are
  removed (the DFA is trim), and states are renumbered breadth-first from the
  start state, visiting bytes in increasing order.

Output tables (the lexer descriptor of the C ABI):
  ``trans``  int16 [Q, 256], -1 = no transition;
  ``accept`` int16 [Q], -1 = not accepting, -2 = skip (whitespace),
             >= 0 = grammar terminal id.
State 0 is the start state and never accepts.

This is input preparation shared by the oracle and the HIP path; it contains
none of the lexing, validation or selection arithmetic itself.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Sequence, Tuple

import numpy as np

SKIP = -2
NONE = -1


# ----------------------------------------------------------------------------
# regular-expression trees
# ----------------------------------------------------------------------------
class Rx:
    pass


@dataclass(frozen=True)
class Chars(Rx):
    bytes_: frozenset


@dataclass(frozen=True)
class Cat(Rx):
    parts: Tuple[Rx, ...]


@dataclass(frozen=True)
class Alt(Rx):
    parts: Tuple[Rx, ...]


@dataclass(frozen=True)
class Star(Rx):
    inner: Rx


def cls(spec: str) -> Rx:
    """Character class from a spec like 'a-z0-9_' (a '-' at either end is literal)."""
    out = set()
    i = 0
    while i < len(spec):
        if i + 2 < len(spec) and spec[i + 1] == "-":
            for c in range(ord(spec[i]), ord(spec[i + 2]) + 1):
                out.add(c)
            i += 3
        else:
            out.add(ord(spec[i]))
            i += 1
    return Chars(frozenset(out))


def lit(s: str) -> Rx:
    return Cat(tuple(Chars(frozenset([ord(c)])) for c in s))


def seq(*parts: Rx) -> Rx:
    return Cat(tuple(parts))


def alt(*parts: Rx) -> Rx:
    return Alt(tuple(parts))


def star(r: Rx) -> Rx:
    return Star(r)


def plus(r: Rx) -> Rx:
    return Cat((r, Star(r)))


def opt(r: Rx) -> Rx:
    return Alt((r, Cat(())))


def any_of(*words: str) -> Rx:
    return Alt(tuple(lit(w) for w in words))


# ----------------------------------------------------------------------------
# Thompson NFA
# ----------------------------------------------------------------------------
class _NFA:
    def __init__(self):
        self.eps: List[List[int]] = []
        self.edges: List[List[Tuple[frozenset, int]]] = []

    def new(self) -> int:
        self.eps.append([])
        self.edges.append([])
        return len(self.eps) - 1

    def build(self, r: Rx) -> Tuple[int, int]:
        s, t = self.new(), self.new()
        if isinstance(r, Chars):
            self.edges[s].append((r.bytes_, t))
        elif isinstance(r, Cat):
            cur = s
            for p in r.parts:
                a, b = self.build(p)
                self.eps[cur].append(a)
                cur = b
            self.eps[cur].append(t)
        elif isinstance(r, Alt):
            for p in r.parts:
                a, b = self.build(p)
                self.eps[s].append(a)
                self.eps[b].append(t)
        elif isinstance(r, Star):
            a, b = self.build(r.inner)
            self.eps[s].append(a)
            self.eps[s].append(t)
            self.eps[b].append(a)
            self.eps[b].append(t)
        else:
            raise TypeError(r)
        return s, t

    def closure(self, states) -> frozenset:
        seen = set(states)
        stack = list(states)
        while stack:
            u = stack.pop()
            for v in self.eps[u]:
                if v not in seen:
                    seen.add(v)
                    stack.append(v)
        return frozenset(seen)


@dataclass
class LexerRule:
    name: str
    pattern: Rx
    label: int  # grammar terminal id, or SKIP


@dataclass
class LexerTables:
    trans: np.ndarray  # int16 [Q, 256]
    accept: np.ndarray  # int16 [Q]

    @property
    def num_states(self) -> int:
        return int(self.trans.shape[0])


def compile_lexer(rules: Sequence[LexerRule]) -> LexerTables:
    """Compile prioritised rules into the trim, minimal, BFS-numbered DFA."""
    nfa = _NFA()
    start = nfa.new()
    final_label: Dict[int, Tuple[int, int]] = {}  # nfa accept state -> (priority, label)
    for prio, rule in enumerate(rules):
        a, b = nfa.build(rule.pattern)
        nfa.eps[start].append(a)
        final_label[b] = (prio, rule.label)

    # subset construction
    d0 = nfa.closure([start])
    dstates: Dict[frozenset, int] = {d0: 0}
    order = [d0]
    dtrans: List[Dict[int, int]] = []
    i = 0
    while i < len(order):
        S = order[i]
        row: Dict[int, int] = {}
        moves: Dict[int, set] = {}
        for u in S:
            for bset, v in nfa.edges[u]:
                for c in bset:
                    moves.setdefault(c, set()).add(v)
        for c, vs in moves.items():
            T = nfa.closure(vs)
            if T not in dstates:
                dstates[T] = len(order)
                order.append(T)
            row[c] = dstates[T]
        dtrans.append(row)
        i += 1
    nd = len(order)
    dacc = []
    for S in order:
        best = None
        for u in S:
            if u in final_label:
                if best is None or final_label[u][0] < best[0]:
                    best = final_label[u]
        dacc.append(NONE if best is None else best[1])
    if dacc[0] != NONE:
        raise ValueError("a lexer rule accepts the empty string")

    # Moore minimisation (complete the DFA with an implicit dead state = -1)
    block = {s: ("acc", dacc[s]) for s in range(nd)}
    while True:
        keys = {}
        new_block = {}
        for s in range(nd):
            sig = (block[s], tuple(block[dtrans[s][c]] if c in dtrans[s] else None for c in range(256)))
            if sig not in keys:
                keys[sig] = len(keys)
            new_block[s] = keys[sig]
        if len(set(new_block.values())) == len(set(block.values())):
            block = new_block
            break
        block = new_block
    # quotient
    reps: Dict[int, int] = {}
    for s in range(nd):
        reps.setdefault(block[s], s)
    q_trans = {b: {c: block[t] for c, t in dtrans[s].items()} for b, s in reps.items()}
    q_acc = {b: dacc[s] for b, s in reps.items()}
    q_start = block[0]

    # trim: keep blocks that can reach an accepting block
    live = {b for b in q_acc if q_acc[b] != NONE}
    changed = True
    while changed:
        changed = False
        for b, row in q_trans.items():
            if b not in live and any(t in live for t in row.values()):
                live.add(b)
                changed = True
    if q_start not in live:
        raise ValueError("lexer accepts nothing")

    # BFS renumbering, bytes in increasing order
    num = {q_start: 0}
    bfs = [q_start]
    k = 0
    while k < len(bfs):
        b = bfs[k]
        for c in range(256):
            t = q_trans[b].get(c)
            if t is not None and t in live and t not in num:
                num[t] = len(bfs)
                bfs.append(t)
        k += 1
    Q = len(bfs)
    trans = np.full((Q, 256), -1, dtype=np.int16)
    accept = np.full((Q,), NONE, dtype=np.int16)
    for b, i in num.items():
        accept[i] = q_acc[b]
        for c, t in q_trans[b].items():
            if t in num:
                trans[i, c] = num[t]
    if accept[0] != NONE:
        raise ValueError("start state accepts")
    return LexerTables(trans=trans, accept=accept)
