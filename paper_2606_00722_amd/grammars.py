"""Synthetic languages standing in for the paper's three tasks (Sec. 5, App. E.2).

The paper evaluates on C++ (HumanEval-X), JSON under instance-specific schemas
and SMILES, with grammars and lexical specifications taken from prior work that
are not available here.  This module defines small, self-written languages of
the same kinds and sizes:

* ``arith``  - the arithmetic-expression grammar E->E+T|T, T->T*F|F, F->(E)|num|id;
* ``json``   - a JSON-like grammar with a few schema keys as their own terminals;
* ``smiles`` - a SMILES-like grammar (atoms, bonds, branches, ring digits,
  bracket atoms; ring closures approximated context-free) whose lexer has no
  whitespace, as the paper notes for SMILES;
* ``clike``  - a C-like statement/expression grammar (about 150 productions,
  63 terminals).

Each language provides the lexer rules (compiled by :mod:`lexspec`), the
grammar as plain productions, the byte alphabet for vocabularies, lexeme
samplers and a separator rule used only to render seeded sentences.  None of
this is the validity arithmetic; it is input data for both sides.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import lexspec as lx


@dataclass
class Grammar:
    """A CFG over named symbols.  Terminals are numbered first (0..T-1),
    nonterminals after them (T..T+N-1); ``start`` is a nonterminal name."""

    terminals: List[str]
    nonterminals: List[str]
    productions: List[Tuple[str, Tuple[str, ...]]]
    start: str

    def __post_init__(self):
        self.tid = {t: i for i, t in enumerate(self.terminals)}
        self.nid = {n: len(self.terminals) + i for i, n in enumerate(self.nonterminals)}
        for lhs, rhs in self.productions:
            if lhs not in self.nid:
                raise ValueError(f"lhs {lhs} is not a nonterminal")
            for s in rhs:
                if s not in self.tid and s not in self.nid:
                    raise ValueError(f"undefined symbol {s}")
        if self.start not in self.nid:
            raise ValueError("start is not a nonterminal")

    def sym(self, name: str) -> int:
        return self.tid[name] if name in self.tid else self.nid[name]

    def arrays(self):
        """(num_terminals, num_nonterminals, start, lhs, rhs_offsets, rhs) as int32 arrays."""
        lhs = np.array([self.nid[l] for l, _ in self.productions], dtype=np.int32)
        offs = [0]
        rhs: List[int] = []
        for _, r in self.productions:
            rhs.extend(self.sym(s) for s in r)
            offs.append(len(rhs))
        return (
            len(self.terminals),
            len(self.nonterminals),
            self.nid[self.start],
            lhs,
            np.array(offs, dtype=np.int32),
            np.array(rhs, dtype=np.int32),
        )

    def num_items(self) -> int:
        """Dotted items including the augmented start production S' -> S."""
        return sum(len(r) + 1 for _, r in self.productions) + 2


@dataclass
class Language:
    name: str
    grammar: Grammar
    rules: List[lx.LexerRule]
    alphabet: str
    lexeme: Dict[str, Callable[[np.random.Generator], str]]
    wordish: frozenset = frozenset()
    opish: frozenset = frozenset()
    # builds a top-level terminal sequence of at least `min_bytes` rendered bytes
    top: Optional[Callable] = None
    _tables: Optional[lx.LexerTables] = None

    @property
    def tables(self) -> lx.LexerTables:
        if self._tables is None:
            self._tables = lx.compile_lexer(self.rules)
        return self._tables

    def needs_space(self, a: str, b: str) -> bool:
        return (a in self.wordish and b in self.wordish) or (a in self.opish and b in self.opish)


def _P(spec: str) -> List[Tuple[str, Tuple[str, ...]]]:
    """Parse 'A -> x y | z ; B -> ...' (one rule per line) into productions.
    The word 'eps' stands for the empty right-hand side."""
    prods = []
    for line in spec.strip().splitlines():
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        lhs, rhs = line.split("->")
        lhs = lhs.strip()
        for alt_ in rhs.split("|"):
            syms = tuple(s for s in alt_.split() if s != "eps")
            prods.append((lhs, syms))
    return prods


def _nonterminals(prods) -> List[str]:
    seen: List[str] = []
    for l, _ in prods:
        if l not in seen:
            seen.append(l)
    return seen


# ----------------------------------------------------------------------------
# random derivation with a depth cap (input generation only)
# ----------------------------------------------------------------------------
class Deriver:
    """Seeded random derivations.  Only productions whose minimal derivation
    height fits the remaining depth are chosen; directly recursive productions
    get a lower weight so that sizes stay moderate."""

    def __init__(self, g: Grammar, weights: Optional[Dict[Tuple[str, Tuple[str, ...]], float]] = None):
        self.g = g
        self.weights = weights or {}
        self.by_lhs: Dict[str, List[Tuple[str, ...]]] = {}
        for l, r in g.productions:
            self.by_lhs.setdefault(l, []).append(r)
        INF = 10**9
        h = {n: INF for n in g.nonterminals}

        def sh(s):
            return 0 if s in g.tid else h[s]

        changed = True
        while changed:
            changed = False
            for l, r in g.productions:
                v = 1 + max([sh(s) for s in r], default=0)
                if v < h[l]:
                    h[l] = v
                    changed = True
        self.h = h
        self.sh = sh

        # per nonterminal: (alternative, its minimal height, its weight); directly
        # recursive alternatives default to a quarter of the weight
        self.table = {}
        for l, alts in self.by_lhs.items():
            self.table[l] = [(r, 1 + max([sh(s) for s in r], default=0),
                              self.weights.get((l, r), 0.25 if l in r else 1.0)) for r in alts]

    def derive(self, rng: np.random.Generator, sym: str, depth: int) -> List[str]:
        if sym in self.g.tid:
            return [sym]
        alts = self.table[sym]
        if depth <= 0:
            best = min(h for _, h, _ in alts)
            alts = [a for a in alts if a[1] == best]
        else:
            alts = [a for a in alts if a[1] <= depth + 1] or alts
        w = np.array([a[2] for a in alts])
        r = alts[int(rng.choice(len(alts), p=w / w.sum()))][0]
        out: List[str] = []
        for s in r:
            out.extend(self.derive(rng, s, depth - 1))
        return out


class TextBuilder:
    """Appends rendered terminal runs while tracking the exact byte length,
    so that top-level generators can stop inside a byte window."""

    def __init__(self, lang: "Language", rng: np.random.Generator, extra_space: float = 0.0):
        self.lang, self.rng, self.extra = lang, rng, extra_space
        self.ws = any(r.label == lx.SKIP for r in lang.rules)
        self.parts: List[str] = []
        self.terms: List[str] = []
        self.n = 0

    def piece(self, terms: Sequence[str]) -> Tuple[str, List[str]]:
        prev = self.terms[-1] if self.terms else None
        out = []
        for t in terms:
            s = self.lang.lexeme[t](self.rng)
            if prev is not None and self.ws:
                if self.lang.needs_space(prev, t) or (self.extra > 0 and self.rng.random() < self.extra):
                    out.append(" ")
            out.append(s)
            prev = t
        return "".join(out), list(terms)

    def add(self, piece: Tuple[str, List[str]]):
        self.parts.append(piece[0])
        self.terms.extend(piece[1])
        self.n += len(piece[0])

    def fits(self, piece, max_bytes: int, reserve: int = 0) -> bool:
        return self.n + len(piece[0]) + reserve <= max_bytes

    @property
    def text(self) -> str:
        return "".join(self.parts)


def grow(b: TextBuilder, make: Callable[[], List[str]], min_bytes: int, max_bytes: int,
         reserve: int = 0, tries: int = 40) -> bool:
    """Append pieces from `make` until at least min_bytes (counting `reserve`
    bytes still to come); pieces that would pass max_bytes are redrawn."""
    while b.n + reserve < min_bytes:
        for _ in range(tries):
            p = b.piece(make())
            if b.fits(p, max_bytes, reserve):
                b.add(p)
                break
        else:
            return False
    return True


def render(lang: Language, rng: np.random.Generator, terms: Sequence[str], extra_space: float = 0.0) -> Tuple[str, List[str]]:
    """Render terminal names to text; spaces only where the language needs them
    to keep lexemes apart (plus optional random spaces for whitespace lexers)."""
    parts: List[str] = []
    lexemes: List[str] = []
    prev = None
    ws = any(r.label == lx.SKIP for r in lang.rules)
    for t in terms:
        s = lang.lexeme[t](rng)
        if prev is not None and ws:
            if lang.needs_space(prev, t) or (extra_space > 0 and rng.random() < extra_space):
                parts.append(" ")
        parts.append(s)
        lexemes.append(s)
        prev = t
    return "".join(parts), lexemes


def _choice(words: Sequence[str]):
    return lambda rng: words[int(rng.integers(len(words)))]


def _const(s: str):
    return lambda rng: s


def _digits(lo: int, hi: int, first_nonzero: bool = False):
    def f(rng):
        n = int(rng.integers(lo, hi + 1))
        d = [str(int(rng.integers(10))) for _ in range(n)]
        if first_nonzero and n > 1 and d[0] == "0":
            d[0] = str(int(rng.integers(1, 10)))
        return "".join(d)

    return f


def _ident(alpha: str, rest: str, lo: int, hi: int, avoid: Sequence[str] = ()):
    avoid_s = set(avoid)

    def f(rng):
        while True:
            n = int(rng.integers(lo, hi + 1))
            s = alpha[int(rng.integers(len(alpha)))] + "".join(rest[int(rng.integers(len(rest)))] for _ in range(n - 1))
            if s not in avoid_s:
                return s

    return f


# ----------------------------------------------------------------------------
# 1. arithmetic
# ----------------------------------------------------------------------------
def _arith() -> Language:
    terms = ["PLUS", "STAR", "LP", "RP", "NUM", "ID"]
    prods = _P(
        """
        E -> E PLUS T | T
        T -> T STAR F | F
        F -> LP E RP | NUM | ID
        """
    )
    g = Grammar(terms, _nonterminals(prods), prods, "E")
    T = g.tid
    rules = [
        lx.LexerRule("PLUS", lx.lit("+"), T["PLUS"]),
        lx.LexerRule("STAR", lx.lit("*"), T["STAR"]),
        lx.LexerRule("LP", lx.lit("("), T["LP"]),
        lx.LexerRule("RP", lx.lit(")"), T["RP"]),
        lx.LexerRule("NUM", lx.plus(lx.cls("0-9")), T["NUM"]),
        lx.LexerRule("ID", lx.plus(lx.cls("a-z")), T["ID"]),
        lx.LexerRule("WS", lx.plus(lx.lit(" ")), lx.SKIP),
    ]
    lexeme = {
        "PLUS": _const("+"),
        "STAR": _const("*"),
        "LP": _const("("),
        "RP": _const(")"),
        "NUM": _digits(1, 3),
        "ID": _ident("abcdefghijklmnopqrstuvwxyz", "abcdefghijklmnopqrstuvwxyz", 1, 3),
    }
    lang = Language("arith", g, rules, "0123456789abcdefghijklmnopqrstuvwxyz+*() ", lexeme,
                    wordish=frozenset({"NUM", "ID"}))
    der = Deriver(g)

    def top(b: TextBuilder, min_bytes: int, max_bytes: int) -> bool:
        return grow(b, lambda: (["PLUS"] if b.terms else []) + der.derive(b.rng, "T", 6), min_bytes, max_bytes)

    lang.top = top
    return lang


# ----------------------------------------------------------------------------
# 2. JSON-like with schema keys
# ----------------------------------------------------------------------------
def _json() -> Language:
    terms = ["LBRACE", "RBRACE", "LBRACK", "RBRACK", "COLON", "COMMA",
             "K_ID", "K_NAME", "K_TAGS", "K_META", "K_ACTIVE",
             "STRING", "NUMBER", "TRUE", "FALSE", "NULL"]
    prods = _P(
        """
        json -> object
        object -> LBRACE RBRACE | LBRACE members RBRACE
        members -> member | member COMMA members
        member -> K_ID COLON NUMBER | K_NAME COLON STRING | K_TAGS COLON strarray | K_META COLON object | K_ACTIVE COLON boolean | STRING COLON value
        value -> object | array | STRING | NUMBER | boolean | NULL
        boolean -> TRUE | FALSE
        array -> LBRACK RBRACK | LBRACK elements RBRACK
        elements -> value | value COMMA elements
        strarray -> LBRACK RBRACK | LBRACK strings RBRACK
        strings -> STRING | STRING COMMA strings
        """
    )
    g = Grammar(terms, _nonterminals(prods), prods, "json")
    T = g.tid
    body = lx.cls("a-zA-Z0-9 .+-")
    rules = [
        lx.LexerRule("LBRACE", lx.lit("{"), T["LBRACE"]),
        lx.LexerRule("RBRACE", lx.lit("}"), T["RBRACE"]),
        lx.LexerRule("LBRACK", lx.lit("["), T["LBRACK"]),
        lx.LexerRule("RBRACK", lx.lit("]"), T["RBRACK"]),
        lx.LexerRule("COLON", lx.lit(":"), T["COLON"]),
        lx.LexerRule("COMMA", lx.lit(","), T["COMMA"]),
        lx.LexerRule("K_ID", lx.lit('"id"'), T["K_ID"]),
        lx.LexerRule("K_NAME", lx.lit('"name"'), T["K_NAME"]),
        lx.LexerRule("K_TAGS", lx.lit('"tags"'), T["K_TAGS"]),
        lx.LexerRule("K_META", lx.lit('"meta"'), T["K_META"]),
        lx.LexerRule("K_ACTIVE", lx.lit('"active"'), T["K_ACTIVE"]),
        lx.LexerRule("STRING", lx.seq(lx.lit('"'), lx.star(body), lx.lit('"')), T["STRING"]),
        lx.LexerRule("NUMBER", lx.seq(lx.opt(lx.lit("-")), lx.plus(lx.cls("0-9")),
                                      lx.opt(lx.seq(lx.lit("."), lx.plus(lx.cls("0-9"))))), T["NUMBER"]),
        lx.LexerRule("TRUE", lx.lit("true"), T["TRUE"]),
        lx.LexerRule("FALSE", lx.lit("false"), T["FALSE"]),
        lx.LexerRule("NULL", lx.lit("null"), T["NULL"]),
        lx.LexerRule("WS", lx.plus(lx.lit(" ")), lx.SKIP),
    ]
    words = ["alpha", "beta", "x", "Item 7", "blue", "k9", "north", "A.B", "zeta-2", "on", "Q"]

    def string(rng):
        return '"' + words[int(rng.integers(len(words)))] + '"'

    def number(rng):
        s = _digits(1, 3, True)(rng)
        if rng.random() < 0.2:
            s = "-" + s
        if rng.random() < 0.2:
            s += "." + _digits(1, 2)(rng)
        return s

    lexeme = {
        "LBRACE": _const("{"), "RBRACE": _const("}"), "LBRACK": _const("["), "RBRACK": _const("]"),
        "COLON": _const(":"), "COMMA": _const(","),
        "K_ID": _const('"id"'), "K_NAME": _const('"name"'), "K_TAGS": _const('"tags"'),
        "K_META": _const('"meta"'), "K_ACTIVE": _const('"active"'),
        "STRING": string, "NUMBER": number,
        "TRUE": _const("true"), "FALSE": _const("false"), "NULL": _const("null"),
    }
    lang = Language("json", g, rules, '{}[]:,"-+.0123456789abcdefghijklmnopqrstuvwxyzABCDEFGHIJKLMNOPQRSTUVWXYZ ',
                    lexeme, wordish=frozenset({"NUMBER", "TRUE", "FALSE", "NULL"}))
    der = Deriver(g)

    def top(b: TextBuilder, min_bytes: int, max_bytes: int) -> bool:
        b.add(b.piece(["LBRACE"]))
        ok = grow(b, lambda: (["COMMA"] if len(b.terms) > 1 else []) + der.derive(b.rng, "member", 6),
                  min_bytes, max_bytes, reserve=1)
        b.add(b.piece(["RBRACE"]))
        return ok

    lang.top = top
    return lang


# ----------------------------------------------------------------------------
# 3. SMILES-like (no whitespace)
# ----------------------------------------------------------------------------
def _smiles() -> Language:
    terms = ["ATOM_AL", "ATOM_AR", "ELEM", "H", "LBRACK", "RBRACK", "LP", "RP",
             "DIGIT", "RING2", "EQ", "HASH", "MINUS", "PLUS", "SLASH", "BSLASH",
             "COLON", "AT", "DOT"]
    prods = _P(
        """
        smiles -> chain | smiles DOT chain
        chain -> branched | chain branched | chain bond branched
        branched -> atom ringbonds branches
        ringbonds -> eps | ringbonds ringbond
        ringbond -> ringnum | bond ringnum
        ringnum -> DIGIT | RING2
        branches -> eps | branches branch
        branch -> LP chain RP | LP bond chain RP | LP DOT chain RP
        atom -> ATOM_AL | ATOM_AR | bracket
        bracket -> LBRACK isotope symbol chiral hcount charge RBRACK
        isotope -> eps | digits
        digits -> DIGIT | digits DIGIT
        symbol -> ATOM_AL | ATOM_AR | ELEM | H
        chiral -> eps | AT | AT AT
        hcount -> eps | H | H DIGIT
        charge -> eps | PLUS | MINUS | PLUS DIGIT | MINUS DIGIT | PLUS PLUS | MINUS MINUS
        bond -> MINUS | EQ | HASH | COLON | SLASH | BSLASH
        """
    )
    g = Grammar(terms, _nonterminals(prods), prods, "smiles")
    T = g.tid
    rules = [
        lx.LexerRule("ATOM_AL", lx.any_of("B", "C", "N", "O", "P", "S", "F", "I", "Cl", "Br"), T["ATOM_AL"]),
        lx.LexerRule("ATOM_AR", lx.any_of("b", "c", "n", "o", "p", "s"), T["ATOM_AR"]),
        lx.LexerRule("ELEM", lx.any_of("Na", "Ca", "Fe", "Zn", "Mg", "K", "Li", "Si", "Se", "Al"), T["ELEM"]),
        lx.LexerRule("H", lx.lit("H"), T["H"]),
        lx.LexerRule("LBRACK", lx.lit("["), T["LBRACK"]),
        lx.LexerRule("RBRACK", lx.lit("]"), T["RBRACK"]),
        lx.LexerRule("LP", lx.lit("("), T["LP"]),
        lx.LexerRule("RP", lx.lit(")"), T["RP"]),
        lx.LexerRule("DIGIT", lx.cls("0-9"), T["DIGIT"]),
        lx.LexerRule("RING2", lx.seq(lx.lit("%"), lx.cls("0-9"), lx.cls("0-9")), T["RING2"]),
        lx.LexerRule("EQ", lx.lit("="), T["EQ"]),
        lx.LexerRule("HASH", lx.lit("#"), T["HASH"]),
        lx.LexerRule("MINUS", lx.lit("-"), T["MINUS"]),
        lx.LexerRule("PLUS", lx.lit("+"), T["PLUS"]),
        lx.LexerRule("SLASH", lx.lit("/"), T["SLASH"]),
        lx.LexerRule("BSLASH", lx.lit("\\"), T["BSLASH"]),
        lx.LexerRule("COLON", lx.lit(":"), T["COLON"]),
        lx.LexerRule("AT", lx.lit("@"), T["AT"]),
        lx.LexerRule("DOT", lx.lit("."), T["DOT"]),
    ]
    lexeme = {
        "ATOM_AL": _choice(["C", "C", "C", "N", "O", "S", "F", "Cl", "Br", "P", "I", "B"]),
        "ATOM_AR": _choice(["c", "c", "n", "o", "s", "p", "b"]),
        "ELEM": _choice(["Na", "Ca", "Fe", "Zn", "Mg", "K", "Li", "Si", "Se", "Al"]),
        "H": _const("H"), "LBRACK": _const("["), "RBRACK": _const("]"),
        "LP": _const("("), "RP": _const(")"),
        "DIGIT": _digits(1, 1), "RING2": lambda rng: "%" + _digits(2, 2)(rng),
        "EQ": _const("="), "HASH": _const("#"), "MINUS": _const("-"), "PLUS": _const("+"),
        "SLASH": _const("/"), "BSLASH": _const("\\"), "COLON": _const(":"), "AT": _const("@"),
        "DOT": _const("."),
    }
    lang = Language("smiles", g, rules, "BCNOPSFIHclbrnopsKLMZAaegi[]()=#-+@%/\\.:0123456789", lexeme)
    der = Deriver(g, {("atom", ("bracket",)): 0.12, ("branch", ("LP", "DOT", "chain", "RP")): 0.1,
                      ("isotope", ("digits",)): 0.3})

    def top(b: TextBuilder, min_bytes: int, max_bytes: int) -> bool:
        def make():
            out = der.derive(b.rng, "bond", 1) if (b.terms and b.rng.random() < 0.3) else []
            return out + der.derive(b.rng, "branched", 8)

        return grow(b, make, min_bytes, max_bytes)

    lang.top = top
    return lang


# ----------------------------------------------------------------------------
# 4. C-like
# ----------------------------------------------------------------------------
_C_KEYWORDS = ["int", "char", "void", "long", "short", "unsigned", "float", "double", "const",
               "struct", "if", "else", "while", "for", "do", "return", "break", "continue",
               "switch", "case", "default", "sizeof"]
_C_OPS = [("PLUS", "+"), ("MINUS", "-"), ("STAR", "*"), ("SLASH", "/"), ("PERCENT", "%"),
          ("ASSIGN", "="), ("EQ", "=="), ("NE", "!="), ("LT", "<"), ("GT", ">"), ("LE", "<="),
          ("GE", ">="), ("ANDAND", "&&"), ("OROR", "||"), ("NOT", "!"), ("AMP", "&"), ("PIPE", "|"),
          ("CARET", "^"), ("TILDE", "~"), ("SHL", "<<"), ("SHR", ">>"), ("PLUSEQ", "+="),
          ("MINUSEQ", "-="), ("STAREQ", "*="), ("SLASHEQ", "/="), ("INC", "++"), ("DEC", "--"),
          ("ARROW", "->"), ("DOT", "."), ("COMMA", ","), ("SEMI", ";"), ("COLON", ":"),
          ("QUEST", "?"), ("LP", "("), ("RP", ")"), ("LBRACE", "{"), ("RBRACE", "}"),
          ("LBRACK", "["), ("RBRACK", "]")]


_C_EXPR_LEVELS = {"expr", "lor", "land", "bor", "bxor", "band", "eqx", "rel", "shift", "add", "mul", "args"}


def _clike() -> Language:
    kw = [k.upper() for k in _C_KEYWORDS]
    terms = kw + ["IDENT", "NUMBER"] + [n for n, _ in _C_OPS]
    prods = _P(
        """
        unit -> ext | unit ext
        ext -> func_def | decl
        func_def -> type_spec declarator compound
        decl -> type_spec SEMI | type_spec init_list SEMI
        init_list -> init_decl | init_list COMMA init_decl
        init_decl -> declarator | declarator ASSIGN initializer
        initializer -> assign_expr | LBRACE init_items RBRACE | LBRACE init_items COMMA RBRACE
        init_items -> initializer | init_items COMMA initializer
        type_spec -> base_type | CONST base_type | UNSIGNED base_type | UNSIGNED | struct_spec
        base_type -> INT | CHAR | VOID | LONG | SHORT | FLOAT | DOUBLE | LONG LONG
        struct_spec -> STRUCT IDENT | STRUCT IDENT LBRACE fields RBRACE | STRUCT LBRACE fields RBRACE
        fields -> field | fields field
        field -> type_spec declarator SEMI
        declarator -> direct_decl | STAR declarator
        direct_decl -> IDENT | LP declarator RP | direct_decl LBRACK RBRACK | direct_decl LBRACK assign_expr RBRACK | direct_decl LP RP | direct_decl LP params RP | direct_decl LP VOID RP
        params -> param | params COMMA param
        param -> type_spec declarator | type_spec | type_spec abs_decl
        abs_decl -> STAR | STAR abs_decl
        compound -> LBRACE RBRACE | LBRACE items RBRACE
        items -> item | items item
        item -> stmt | decl
        stmt -> compound | expr_stmt | if_stmt | while_stmt | for_stmt | do_stmt | jump_stmt | switch_stmt | labeled
        expr_stmt -> SEMI | expr SEMI
        if_stmt -> IF LP expr RP stmt | IF LP expr RP stmt ELSE stmt
        while_stmt -> WHILE LP expr RP stmt
        do_stmt -> DO stmt WHILE LP expr RP SEMI
        for_stmt -> FOR LP for_init opt_expr SEMI opt_expr RP stmt
        for_init -> expr_stmt | decl
        opt_expr -> eps | expr
        jump_stmt -> RETURN SEMI | RETURN expr SEMI | BREAK SEMI | CONTINUE SEMI
        switch_stmt -> SWITCH LP expr RP stmt
        labeled -> CASE cond_expr COLON stmt | DEFAULT COLON stmt
        expr -> assign_expr | expr COMMA assign_expr
        assign_expr -> cond_expr | unary assign_op assign_expr
        assign_op -> ASSIGN | PLUSEQ | MINUSEQ | STAREQ | SLASHEQ
        cond_expr -> lor | lor QUEST expr COLON cond_expr
        lor -> land | lor OROR land
        land -> bor | land ANDAND bor
        bor -> bxor | bor PIPE bxor
        bxor -> band | bxor CARET band
        band -> eqx | band AMP eqx
        eqx -> rel | eqx EQ rel | eqx NE rel
        rel -> shift | rel LT shift | rel GT shift | rel LE shift | rel GE shift
        shift -> add | shift SHL add | shift SHR add
        add -> mul | add PLUS mul | add MINUS mul
        mul -> cast | mul STAR cast | mul SLASH cast | mul PERCENT cast
        cast -> unary | LP type_name RP cast
        type_name -> type_spec | type_spec abs_decl
        unary -> postfix | INC unary | DEC unary | unary_op cast | SIZEOF unary | SIZEOF LP type_name RP
        unary_op -> AMP | STAR | PLUS | MINUS | TILDE | NOT
        postfix -> primary | postfix LBRACK expr RBRACK | postfix LP RP | postfix LP args RP | postfix DOT IDENT | postfix ARROW IDENT | postfix INC | postfix DEC
        args -> assign_expr | args COMMA assign_expr
        primary -> IDENT | NUMBER | LP expr RP
        """
    )
    g = Grammar(terms, _nonterminals(prods), prods, "unit")
    T = g.tid
    ident_first = "abcdefghijklmnopqrstuvwxyzABCDEFGHIJKLMNOPQRSTUVWXYZ_"
    ident_rest = ident_first + "0123456789"
    rules = [lx.LexerRule(k.upper(), lx.lit(k), T[k.upper()]) for k in _C_KEYWORDS]
    rules.append(lx.LexerRule("IDENT", lx.seq(lx.cls("a-zA-Z_"), lx.star(lx.cls("a-zA-Z0-9_"))), T["IDENT"]))
    rules.append(lx.LexerRule("NUMBER", lx.plus(lx.cls("0-9")), T["NUMBER"]))
    for n, s in _C_OPS:
        rules.append(lx.LexerRule(n, lx.lit(s), T[n]))
    rules.append(lx.LexerRule("WS", lx.plus(lx.lit(" ")), lx.SKIP))
    lexeme: Dict[str, Callable] = {k.upper(): _const(k) for k in _C_KEYWORDS}
    lexeme["IDENT"] = _ident(ident_first, ident_rest, 1, 4, avoid=_C_KEYWORDS)
    lexeme["NUMBER"] = _digits(1, 3, True)
    for n, s in _C_OPS:
        lexeme[n] = _const(s)
    noncombining = {"LP", "RP", "LBRACE", "RBRACE", "LBRACK", "RBRACK", "COMMA", "SEMI", "QUEST",
                    "COLON", "TILDE", "DOT"}
    opish = frozenset(n for n, _ in _C_OPS if n not in noncombining)
    lang = Language("clike", g, rules, ident_rest + "+-*/%=!<>&|^~.,;:?(){}[] ", lexeme,
                    wordish=frozenset(kw + ["IDENT", "NUMBER"]), opish=opish)
    der = Deriver(g, {("unary", ("SIZEOF", "LP", "type_name", "RP")): 0.05, ("unary", ("SIZEOF", "unary")): 0.05,
                      ("unary", ("unary_op", "cast")): 0.2, ("unary", ("INC", "unary")): 0.05,
                      ("unary", ("DEC", "unary")): 0.05, ("postfix", ("postfix", "LP", "args", "RP")): 0.2,
                      ("postfix", ("postfix", "LP", "RP")): 0.1, ("postfix", ("postfix", "LBRACK", "expr", "RBRACK")): 0.1,
                      ("postfix", ("postfix", "DOT", "IDENT")): 0.05, ("postfix", ("postfix", "ARROW", "IDENT")): 0.05,
                      ("postfix", ("postfix", "INC")): 0.05, ("postfix", ("postfix", "DEC")): 0.05,
                      ("primary", ("IDENT",)): 2.0, ("stmt", ("expr_stmt",)): 3.0,
                      **{(l, r): 0.07 for l, r in prods if l in _C_EXPR_LEVELS and l in r},
                      ("cast", ("LP", "type_name", "RP", "cast")): 0.08, ("primary", ("LP", "expr", "RP")): 0.3,
                      ("stmt", ("labeled",)): 0.05, ("stmt", ("switch_stmt",)): 0.3, ("stmt", ("do_stmt",)): 0.3,
                      ("stmt", ("compound",)): 0.5, ("type_spec", ("struct_spec",)): 0.15,
                      ("direct_decl", ("LP", "declarator", "RP")): 0.05, ("item", ("decl",)): 0.4,
                      ("expr_stmt", ("SEMI",)): 0.2, ("for_init", ("decl",)): 0.3,
                      ("struct_spec", ("STRUCT", "LBRACE", "fields", "RBRACE")): 0.3,
                      ("struct_spec", ("STRUCT", "IDENT", "LBRACE", "fields", "RBRACE")): 0.3})

    def top(b: TextBuilder, min_bytes: int, max_bytes: int) -> bool:
        # function definitions whose bodies are filled with statements/declarations
        while True:
            b.add(b.piece(der.derive(b.rng, "type_spec", 4) + ["IDENT", "LP", "RP", "LBRACE"]))
            fn_end = min(min_bytes, b.n + 700)
            if not grow(b, lambda: der.derive(b.rng, "item", 30), fn_end, max_bytes, reserve=1):
                return False
            b.add(b.piece(["RBRACE"]))
            if b.n >= min_bytes:
                return True

    lang.top = top
    return lang


_LANGS: Dict[str, Language] = {}


def language(name: str) -> Language:
    if name not in _LANGS:
        table = {"arith": _arith, "json": _json, "smiles": _smiles, "clike": _clike, **_TINY}
        _LANGS[name] = table[name]()
    return _LANGS[name]


# ----------------------------------------------------------------------------
# tiny languages for brute-force pins and edge cases
# ----------------------------------------------------------------------------
def _tiny(name: str, terms: List[str], spec: str, start: str, rules_spec, alphabet: str,
          lexeme: Dict[str, Callable], wordish=()) -> Language:
    prods = _P(spec)
    g = Grammar(terms, _nonterminals(prods), prods, start)
    rules = [lx.LexerRule(n, pat, lx.SKIP if n == "WS" else g.tid[n]) for n, pat in rules_spec]
    return Language(name, g, rules, alphabet, lexeme, wordish=frozenset(wordish))


def _tiny_paren() -> Language:
    # balanced parentheses with an empty production (nullable start)
    return _tiny("tiny_paren", ["LP", "RP"], "S -> LP S RP S | eps", "S",
                 [("LP", lx.lit("(")), ("RP", lx.lit(")"))], "()",
                 {"LP": _const("("), "RP": _const(")")})


def _tiny_expr() -> Language:
    return _tiny("tiny_expr", ["PLUS", "LP", "RP", "ID"],
                 """
                 E -> E PLUS T | T
                 T -> ID | LP E RP
                 """, "E",
                 [("PLUS", lx.lit("+")), ("LP", lx.lit("(")), ("RP", lx.lit(")")),
                  ("ID", lx.plus(lx.cls("a"))), ("WS", lx.plus(lx.lit(" ")))], "a+() ",
                 {"PLUS": _const("+"), "LP": _const("("), "RP": _const(")"), "ID": _const("a")},
                 wordish=("ID",))


def _tiny_kw() -> Language:
    # keyword versus identifier: 'if' is a keyword, other letter runs are identifiers
    return _tiny("tiny_kw", ["IF", "ID", "LP", "RP"],
                 """
                 S -> IF LP ID RP S | ID
                 """, "S",
                 [("IF", lx.lit("if")), ("ID", lx.plus(lx.cls("fix"))), ("LP", lx.lit("(")),
                  ("RP", lx.lit(")")), ("WS", lx.plus(lx.lit(" ")))], "fix() ",
                 {"IF": _const("if"), "ID": _const("x"), "LP": _const("("), "RP": _const(")")},
                 wordish=("IF", "ID"))


def _tiny_ab() -> Language:
    # no whitespace; 'a' immediately followed by 'b' always lexes as AB, so the
    # terminal sequence A B can never be produced (adjacency constraints in gaps)
    return _tiny("tiny_ab", ["A", "AB", "B", "C"],
                 """
                 S -> A B | AB S | C S | C | A C B
                 """, "S",
                 [("AB", lx.lit("ab")), ("A", lx.lit("a")), ("B", lx.lit("b")), ("C", lx.plus(lx.lit("c")))],
                 "abc", {"A": _const("a"), "AB": _const("ab"), "B": _const("b"), "C": _const("c")})


_TINY = {"tiny_paren": _tiny_paren, "tiny_expr": _tiny_expr, "tiny_kw": _tiny_kw, "tiny_ab": _tiny_ab}
