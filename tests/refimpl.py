"""Independent reference procedures used to pin the oracle (tests only).

* ``munch_lex``: maximal-munch lexing with Python's ``re`` engine from regex
  strings written here (not from the DFA tables), earliest rule wins ties.
* ``derives``: CYK-style recognition for a grammar in its given (non-CNF) form,
  by a fixpoint over spans (handles unit and empty productions).
* ``bar_hillel_valid``: the prior pipeline's criterion (App. A.2): the
  character-level completion automaton built here in Python, epsilon-removed,
  intersected with the grammar by computing productive triples (A, p, q).
* ``brute_valid``: enumerate fillings of the masked runs up to a total length.

These share no code with ``oracle.cpp``.
"""
from __future__ import annotations

import itertools
import re
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

SKIP = "SKIP"

REGEX: Dict[str, List[Tuple[str, str]]] = {
    "arith": [("PLUS", r"\+"), ("STAR", r"\*"), ("LP", r"\("), ("RP", r"\)"), ("NUM", r"[0-9]+"),
              ("ID", r"[a-z]+"), (SKIP, r" +")],
    "json": [("LBRACE", r"\{"), ("RBRACE", r"\}"), ("LBRACK", r"\["), ("RBRACK", r"\]"), ("COLON", r":"),
             ("COMMA", r","), ("K_ID", r'"id"'), ("K_NAME", r'"name"'), ("K_TAGS", r'"tags"'),
             ("K_META", r'"meta"'), ("K_ACTIVE", r'"active"'), ("STRING", r'"[a-zA-Z0-9 .+\-]*"'),
             ("NUMBER", r"-?[0-9]+(\.[0-9]+)?"), ("TRUE", r"true"), ("FALSE", r"false"), ("NULL", r"null"),
             (SKIP, r" +")],
    "smiles": [("ATOM_AL", r"B|C|N|O|P|S|F|I|Cl|Br"), ("ATOM_AR", r"[bcnops]"),
               ("ELEM", r"Na|Ca|Fe|Zn|Mg|K|Li|Si|Se|Al"), ("H", r"H"), ("LBRACK", r"\["), ("RBRACK", r"\]"),
               ("LP", r"\("), ("RP", r"\)"), ("DIGIT", r"[0-9]"), ("RING2", r"%[0-9][0-9]"), ("EQ", r"="),
               ("HASH", r"#"), ("MINUS", r"-"), ("PLUS", r"\+"), ("SLASH", r"/"), ("BSLASH", r"\\"),
               ("COLON", r":"), ("AT", r"@"), ("DOT", r"\.")],
    "tiny_paren": [("LP", r"\("), ("RP", r"\)")],
    "tiny_expr": [("PLUS", r"\+"), ("LP", r"\("), ("RP", r"\)"), ("ID", r"a+"), (SKIP, r" +")],
    "tiny_kw": [("IF", r"if"), ("ID", r"[fix]+"), ("LP", r"\("), ("RP", r"\)"), (SKIP, r" +")],
    "tiny_ab": [("AB", r"ab"), ("A", r"a"), ("B", r"b"), ("C", r"c+")],
}


def _clike_regex():
    kws = ["int", "char", "void", "long", "short", "unsigned", "float", "double", "const", "struct", "if",
           "else", "while", "for", "do", "return", "break", "continue", "switch", "case", "default", "sizeof"]
    out = [(k.upper(), re.escape(k)) for k in kws]
    out += [("IDENT", r"[a-zA-Z_][a-zA-Z0-9_]*"), ("NUMBER", r"[0-9]+")]
    ops = [("PLUS", "+"), ("MINUS", "-"), ("STAR", "*"), ("SLASH", "/"), ("PERCENT", "%"), ("ASSIGN", "="),
           ("EQ", "=="), ("NE", "!="), ("LT", "<"), ("GT", ">"), ("LE", "<="), ("GE", ">="), ("ANDAND", "&&"),
           ("OROR", "||"), ("NOT", "!"), ("AMP", "&"), ("PIPE", "|"), ("CARET", "^"), ("TILDE", "~"),
           ("SHL", "<<"), ("SHR", ">>"), ("PLUSEQ", "+="), ("MINUSEQ", "-="), ("STAREQ", "*="),
           ("SLASHEQ", "/="), ("INC", "++"), ("DEC", "--"), ("ARROW", "->"), ("DOT", "."), ("COMMA", ","),
           ("SEMI", ";"), ("COLON", ":"), ("QUEST", "?"), ("LP", "("), ("RP", ")"), ("LBRACE", "{"),
           ("RBRACE", "}"), ("LBRACK", "["), ("RBRACK", "]")]
    out += [(n, re.escape(s)) for n, s in ops]
    out.append((SKIP, r" +"))
    return out


REGEX["clike"] = _clike_regex()


def munch_lex(lang_name: str, text: str) -> Optional[List[str]]:
    """Maximal munch: longest match at each position, earliest rule on ties."""
    rules = [(n, re.compile(p)) for n, p in REGEX[lang_name]]
    out: List[str] = []
    i = 0
    while i < len(text):
        best = None
        for L in range(len(text) - i, 0, -1):
            sub = text[i:i + L]
            for name, rx in rules:
                if rx.fullmatch(sub):
                    best = (L, name)
                    break
            if best:
                break
        if best is None:
            return None
        if best[1] != SKIP:
            out.append(best[1])
        i += best[0]
    return out


# ----------------------------------------------------------------------------
def derives(grammar, terms: Sequence[str]) -> bool:
    """Whether the start symbol derives the terminal-name sequence `terms`."""
    n = len(terms)
    prods = grammar.productions
    nts = set(grammar.nonterminals)
    D: Dict[Tuple[int, int], set] = {}

    def can(sym, i, j):
        if sym in nts:
            return sym in D.get((i, j), ())
        return j == i + 1 and terms[i] == sym

    for L in range(0, n + 1):
        for i in range(0, n - L + 1):
            j = i + L
            cur = D.setdefault((i, j), set())
            changed = True
            while changed:
                changed = False
                for lhs, rhs in prods:
                    if lhs in cur:
                        continue
                    # chain DP over split points
                    reach = {i}
                    for s in rhs:
                        nxt = set()
                        for p in reach:
                            for q in range(p, j + 1):
                                if can(s, p, q):
                                    nxt.add(q)
                        reach = nxt
                        if not reach:
                            break
                    if j in reach:
                        cur.add(lhs)
                        changed = True
    return grammar.start in D[(0, n)]


# ----------------------------------------------------------------------------
def _step(trans, accept, q, c):
    d = int(trans[q, c])
    if d >= 0:
        return d, None
    a = int(accept[q])
    f = int(trans[0, c])
    if a != -1 and f >= 0:
        return f, (None if a == -2 else a)
    return -1, None


def _flush(accept, q):
    if q == 0:
        return True, None
    a = int(accept[q])
    if a >= 0:
        return True, a
    if a == -2:
        return True, None
    return False, None


def bar_hillel_valid(lang, vocab_strings: Sequence[bytes], x: Sequence[int]) -> bool:
    """L(G) cap C_x non-empty, by productive triples over an automaton built here."""
    trans, accept = lang.tables.trans, lang.tables.accept
    Q = trans.shape[0]
    slots: List[int] = []
    for t in x:
        if t < 0:
            if not slots or slots[-1] != -1:
                slots.append(-1)
        else:
            slots.extend(vocab_strings[t])
    S = len(slots)
    FINAL = ("F",)
    eps: Dict = {}
    lab: Dict = {}
    seen = {(0, 0)}
    stack = [(0, 0)]

    def edge(u, o, v):
        (eps if o is None else lab).setdefault(u, set()).add(v if o is None else (o, v))
        if v not in seen:
            seen.add(v)
            stack.append(v)

    while stack:
        u = stack.pop()
        if u == FINAL:
            continue
        s, q = u
        if s == S:
            ok, o = _flush(accept, q)
            if ok:
                edge(u, o, FINAL)
            continue
        if slots[s] >= 0:
            q2, o = _step(trans, accept, q, slots[s])
            if q2 >= 0:
                edge(u, o, (s + 1, q2))
        else:
            edge(u, None, (s + 1, q))
            for c in range(256):
                q2, o = _step(trans, accept, q, c)
                if q2 >= 0:
                    edge(u, o, (s, q2))

    def closure(u):
        out = {u}
        st = [u]
        while st:
            w = st.pop()
            for v in eps.get(w, ()):
                if v not in out:
                    out.add(v)
                    st.append(v)
        return out

    # epsilon-free automaton over the start node and targets of labelled edges
    items = {(0, 0)} | {v for es in lab.values() for (_, v) in es}
    arcs: Dict = {}
    final = set()
    for u in items:
        for w in closure(u):
            if w == FINAL:
                final.add(u)
            for a, v in lab.get(w, ()):
                arcs.setdefault(a, set()).add((u, v))
    g = lang.grammar
    tid = g.tid
    prods = [(l, [tid[s] if s in tid else s for s in r]) for l, r in g.productions]
    prod_triples = set()
    changed = True
    while changed:
        changed = False
        for lhs, rhs in prods:
            pairs = {(p, p) for p in items}
            for s in rhs:
                nxt = set()
                if isinstance(s, int):
                    for (u, v) in arcs.get(s, ()):
                        for (p, r) in pairs:
                            if r == u:
                                nxt.add((p, v))
                else:
                    by_start: Dict = {}
                    for (A, u, v) in prod_triples:
                        if A == s:
                            by_start.setdefault(u, set()).add(v)
                    for (p, r) in pairs:
                        for v in by_start.get(r, ()):
                            nxt.add((p, v))
                pairs = nxt
                if not pairs:
                    break
            for (p, q) in pairs:
                if (lhs, p, q) not in prod_triples:
                    prod_triples.add((lhs, p, q))
                    changed = True
    return any((g.start, (0, 0), f) in prod_triples for f in final)


def brute_valid(lang, vocab_strings: Sequence[bytes], x: Sequence[int], alphabet: str, max_total: int) -> bool:
    """Some filling of the mask runs with strings over `alphabet`, of total
    length <= max_total, lexes (maximal munch) to a sentence of the grammar."""
    parts: List = []
    for t in x:
        if t < 0:
            if not parts or parts[-1] is not None:
                parts.append(None)
        else:
            if parts and isinstance(parts[-1], str):
                parts[-1] += vocab_strings[t].decode()
            else:
                parts.append(vocab_strings[t].decode())
    gaps = sum(1 for p in parts if p is None)
    for total in range(0, max_total + 1):
        for lens in itertools.product(range(total + 1), repeat=gaps):
            if sum(lens) != total:
                continue
            fills = [itertools.product(alphabet, repeat=L) for L in lens]
            for combo in itertools.product(*fills):
                it = iter(combo)
                text = "".join(p if p is not None else "".join(next(it)) for p in parts)
                toks = munch_lex(lang.name, text)
                if toks is not None and derives(lang.grammar, toks):
                    return True
    return False
