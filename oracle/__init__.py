"""ctypes loader for the CPU oracle (``oracle.cpp``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only users.  The product path never imports this
package.  Functions take the seeded generator's plain arrays; see
``oracle.cpp`` for what each one computes and which passage of the paper it
follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.cpp")
LIB = os.path.join(HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile the oracle with the host compiler (plain g++, -O2)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-o", tmp, SRC, "-lpthread"])
        os.replace(tmp, LIB)
    return LIB


class _Lexer(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("trans", ctypes.c_void_p), ("accept", ctypes.c_void_p)]


class _Grammar(ctypes.Structure):
    _fields_ = [("num_terminals", ctypes.c_int32), ("num_nonterminals", ctypes.c_int32),
                ("start", ctypes.c_int32), ("num_productions", ctypes.c_int32),
                ("lhs", ctypes.c_void_p), ("rhs_offsets", ctypes.c_void_p), ("rhs", ctypes.c_void_p)]


class _Vocab(ctypes.Structure):
    _fields_ = [("vocab_size", ctypes.c_int32), ("bytes", ctypes.c_void_p), ("offsets", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build(force=True)
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32 = ctypes.c_int
        L.oracle_lex_step.argtypes = [P, i32, i32, P]
        L.oracle_lex_bytes.argtypes = [P, i32, P, i32, i32, P, i32, P]
        L.oracle_memo.argtypes = [P, P, P]
        L.oracle_valid.argtypes = [P, P, P, P, i32]
        L.oracle_cover.argtypes = [P, P, P, P, i32]
        L.oracle_dfa_states.argtypes = [P, P, P, P, i32]
        L.oracle_validate_batch.argtypes = [P, P, P, P, i32, i32, P, P, P, i32, P, i32]
        L.oracle_select.argtypes = [P, P, P, P, i32, i32, P, P, P, P, P, i32, P, P, i32]
        L.oracle_witness.argtypes = [P, P, P, P, i32, P, i32, P, i32, P]
        L.oracle_valid_text.argtypes = [P, P, P, i32]
        L.oracle_con_validate_batch.argtypes = [P, P, P, P, i32, i32, P, P, P, i32, P, P, i32]
        L.oracle_con_dfa_states.argtypes = [P, P, P, P, i32]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


@dataclass
class Problem:
    """Lexer DFA, grammar and vocabulary as contiguous arrays plus C structs."""

    trans: np.ndarray
    accept: np.ndarray
    T: int
    N: int
    start: int
    lhs: np.ndarray
    roff: np.ndarray
    rhs: np.ndarray
    vbytes: np.ndarray
    voffs: np.ndarray

    def __post_init__(self):
        self.trans = np.ascontiguousarray(self.trans, dtype=np.int16)
        self.accept = np.ascontiguousarray(self.accept, dtype=np.int16)
        self.lhs = np.ascontiguousarray(self.lhs, dtype=np.int32)
        self.roff = np.ascontiguousarray(self.roff, dtype=np.int32)
        self.rhs = np.ascontiguousarray(self.rhs, dtype=np.int32)
        self.vbytes = np.ascontiguousarray(self.vbytes, dtype=np.uint8)
        if self.vbytes.size == 0:
            self.vbytes = np.zeros(1, dtype=np.uint8)
        self.voffs = np.ascontiguousarray(self.voffs, dtype=np.int32)
        self._lx = _Lexer(self.trans.shape[0], _ptr(self.trans), _ptr(self.accept))
        self._gr = _Grammar(self.T, self.N, self.start, len(self.lhs), _ptr(self.lhs), _ptr(self.roff),
                            _ptr(self.rhs) if self.rhs.size else _ptr(np.zeros(1, np.int32)))
        self._vc = _Vocab(len(self.voffs) - 1, _ptr(self.vbytes), _ptr(self.voffs))

    @property
    def Q(self) -> int:
        return int(self.trans.shape[0])

    @property
    def V(self) -> int:
        return len(self.voffs) - 1

    @property
    def refs(self):
        return ctypes.byref(self._lx), ctypes.byref(self._gr), ctypes.byref(self._vc)


def problem_from(lang, vocab) -> Problem:
    """Build a Problem from a grammars.Language and a workloads.Vocab."""
    tb = lang.tables
    T, N, start, lhs, roff, rhs = lang.grammar.arrays()
    vb, vo = vocab.csr()
    return Problem(tb.trans, tb.accept, T, N, start, lhs, roff, rhs, vb, vo)


def lex_step(p: Problem, q: int, c: int) -> Tuple[int, int]:
    e = ctypes.c_int(0)
    r = lib().oracle_lex_step(ctypes.byref(p._lx), q, c, ctypes.byref(e))
    return r, e.value


def lex_bytes(p: Problem, q: int, data: bytes, flush: bool):
    """(terminals, final_state) or None if the greedy lexer dies."""
    buf = np.frombuffer(data, dtype=np.uint8).copy() if data else np.zeros(1, np.uint8)
    out = np.zeros(len(data) + 2, dtype=np.int32)
    fs = ctypes.c_int(-1)
    n = lib().oracle_lex_bytes(ctypes.byref(p._lx), q, _ptr(buf), len(data), int(flush), _ptr(out), len(out),
                               ctypes.byref(fs))
    if n < 0:
        return None
    return out[:n].tolist(), fs.value


def memo(p: Problem) -> np.ndarray:
    out = np.zeros((p.V, p.Q, 16), dtype=np.uint8)
    r = lib().oracle_memo(ctypes.byref(p._lx), ctypes.byref(p._vc), _ptr(out))
    if r != 0:
        raise ValueError("token longer than 8 bytes or empty")
    return out


def _seq(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def valid(p: Problem, x) -> int:
    xs = _seq(x)
    lx, gr, vc = p.refs
    return lib().oracle_valid(lx, gr, vc, _ptr(xs) if xs.size else _ptr(np.zeros(1, np.int32)), int(xs.size))


def cover(p: Problem, x) -> int:
    xs = _seq(x)
    lx, gr, vc = p.refs
    return lib().oracle_cover(lx, gr, vc, _ptr(xs) if xs.size else _ptr(np.zeros(1, np.int32)), int(xs.size))


def dfa_states(p: Problem, x) -> int:
    xs = _seq(x)
    lx, gr, vc = p.refs
    return lib().oracle_dfa_states(lx, gr, vc, _ptr(xs) if xs.size else _ptr(np.zeros(1, np.int32)), int(xs.size))


def witness(p: Problem, x):
    """A completion of x (failure recovery, Sec. 4): (1, [bytes of each
    maximal masked run, in order]) when x is valid, (0, None) when it is not,
    (-3, None) on a construction limit of the oracle."""
    xs = _seq(x)
    lx, gr, vc = p.refs
    cap, max_gaps = 1 << 16, max(1, int(xs.size))
    out = np.zeros(cap, dtype=np.uint8)
    lens = np.zeros(max_gaps, dtype=np.int32)
    ng = ctypes.c_int32(0)
    r = lib().oracle_witness(lx, gr, vc, _ptr(xs) if xs.size else _ptr(np.zeros(1, np.int32)), int(xs.size),
                             _ptr(out), cap, _ptr(lens), max_gaps, ctypes.byref(ng))
    if r != 1:
        return r, None
    gaps, k = [], 0
    for j in range(ng.value):
        gaps.append(bytes(out[k:k + lens[j]]))
        k += int(lens[j])
    return 1, gaps


def con_validate_batch(p: Problem, seqs: np.ndarray, seq, pos, tok, nthreads: int = 1):
    """The prior pipeline ("Con.": lexing automaton, subset construction,
    Hopcroft minimisation, intersection emptiness) on every candidate: returns
    (verdict uint8[C], summed ms per phase [lex, dfa, val])."""
    s = np.ascontiguousarray(seqs, dtype=np.int32)
    cs, cp, ct = _cands(seq, pos, tok)
    C = int(cs.size)
    out = np.zeros(max(C, 1), dtype=np.uint8)
    ms = np.zeros(3, dtype=np.float64)
    lx, gr, vc = p.refs
    r = lib().oracle_con_validate_batch(lx, gr, vc, _ptr(s), s.shape[0], s.shape[1], _ptr(cs) if C else 0,
                                        _ptr(cp) if C else 0, _ptr(ct) if C else 0, C, _ptr(out), _ptr(ms), nthreads)
    if r != 0:
        raise RuntimeError(f"oracle_con_validate_batch failed ({r})")
    return out[:C], ms


def con_dfa_states(p: Problem, x) -> int:
    xs = _seq(x)
    lx, gr, vc = p.refs
    return lib().oracle_con_dfa_states(lx, gr, vc, _ptr(xs) if xs.size else _ptr(np.zeros(1, np.int32)), int(xs.size))


def valid_text(p: Problem, text: bytes) -> int:
    """Valid of a byte string with no masks (greedy lexing, then membership in
    L(G)): 1, 0, or -3 on a construction limit."""
    buf = np.frombuffer(text, dtype=np.uint8).copy() if text else np.zeros(1, np.uint8)
    lx, gr, _ = p.refs
    return lib().oracle_valid_text(lx, gr, _ptr(buf), len(text))


def _cands(seq, pos, tok):
    return _seq(seq), _seq(pos), _seq(tok)


def validate_batch(p: Problem, seqs: np.ndarray, seq, pos, tok, nthreads: int = 1) -> np.ndarray:
    s = np.ascontiguousarray(seqs, dtype=np.int32)
    cs, cp, ct = _cands(seq, pos, tok)
    C = int(cs.size)
    out = np.zeros(max(C, 1), dtype=np.uint8)
    lx, gr, vc = p.refs
    r = lib().oracle_validate_batch(lx, gr, vc, _ptr(s), s.shape[0], s.shape[1], _ptr(cs) if C else 0,
                                    _ptr(cp) if C else 0, _ptr(ct) if C else 0, C, _ptr(out), nthreads)
    if r != 0:
        raise RuntimeError(f"oracle_validate_batch failed ({r})")
    return out[:C]


def select(p: Problem, seqs: np.ndarray, seq, pos, tok, conf, verdict, nthreads: int = 1):
    """Returns (selected uint8[C], (cover_calls, exact_calls), status)."""
    s = np.ascontiguousarray(seqs, dtype=np.int32)
    cs, cp, ct = _cands(seq, pos, tok)
    cf = np.ascontiguousarray(conf, dtype=np.float32)
    vd = np.ascontiguousarray(verdict, dtype=np.uint8)
    C = int(cs.size)
    out = np.zeros(max(C, 1), dtype=np.uint8)
    stats = np.zeros(2, dtype=np.int64)
    lx, gr, vc = p.refs
    if C == 0:
        return out[:0], (0, 0), 0
    r = lib().oracle_select(lx, gr, vc, _ptr(s), s.shape[0], s.shape[1], _ptr(cs), _ptr(cp), _ptr(ct), _ptr(cf),
                            _ptr(vd), C, _ptr(out), _ptr(stats), nthreads)
    return out[:C], (int(stats[0]), int(stats[1])), int(r)


def fallback(p: Problem, seqs: np.ndarray, seq, pos, tok, conf, verdict, selected, num_commit, nthreads: int = 1):
    """The sequential fallback after the relaxed batch in EPIC decoding (App. C.1,
    Alg. 1 and the paragraph after it), taken step by step:
    per sequence b, commit the selected set B to x_b, then walk the remaining
    candidates of b by descending confidence (ties to the lower index) and
    commit each whose exact check Valid(x_b + c) holds on the current x_b, until
    num_commit[b] - |B| more are committed or the candidates run out.  Every
    candidate is checked whatever its verdict; one whose position is no longer
    masked cannot be applied and is passed over.  Input rule as in `select`: a
    sequence whose verdict-1 candidates repeat a position or carry a NaN
    confidence commits nothing (status -4).  There is no limit on the number
    of candidates (Alg. 1 has none).  `nthreads` runs sequences concurrently.
    Returns (accepted uint8[C], status)."""
    s = np.ascontiguousarray(seqs, dtype=np.int32)
    cs, cp, ct = _cands(seq, pos, tok)
    cf = np.asarray(conf, dtype=np.float32)
    vd = np.asarray(verdict, dtype=np.uint8)
    sl = np.asarray(selected, dtype=np.uint8)
    nc = np.asarray(num_commit, dtype=np.int64)
    C = int(cs.size)
    acc = np.zeros(C, dtype=np.uint8)

    def one(b: int) -> int:  # sequences are independent: one loop each
        mine = [c for c in range(C) if cs[c] == b]
        v1 = [c for c in mine if vd[c] == 1]
        if any(np.isnan(cf[c]) for c in v1) or len({int(cp[c]) for c in v1}) < len(v1):
            return -4
        x = s[b].copy()
        committed = [c for c in mine if sl[c]]
        for c in committed:
            x[cp[c]] = ct[c]
        need = int(nc[b]) - len(committed)
        order = sorted((c for c in mine if not np.isnan(cf[c])), key=lambda c: (-float(cf[c]), c))
        order += [c for c in mine if np.isnan(cf[c])]
        for c in order:
            if need <= 0:
                break
            if sl[c] or not (0 <= cp[c] < s.shape[1]) or x[cp[c]] != -1 or not (0 <= ct[c] < len(p.voffs) - 1):
                continue
            y = x.copy()
            y[cp[c]] = ct[c]
            if valid(p, y) == 1:
                x = y
                acc[c] = 1
                need -= 1
        return 0

    if nthreads > 1 and s.shape[0] > 1:
        from concurrent.futures import ThreadPoolExecutor

        with ThreadPoolExecutor(nthreads) as ex:  # the oracle's C calls release the GIL
            sts = list(ex.map(one, range(s.shape[0])))
    else:
        sts = [one(b) for b in range(s.shape[0])]
    return acc, min(sts, default=0)
