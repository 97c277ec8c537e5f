"""Seeded synthetic workloads shaped like the paper's decoding runs.

The paper decodes with diffusion LMs on HumanEval-X C++, a JSON-schema
benchmark and a SMILES benchmark (App. E.2).  Neither models nor datasets are
used here: these generators stand in for them with seeded inputs of the same
kind and shape (vocabularies, partially masked answers, proposals and
confidences).  Five named presets:

=====  ========  ======  ====  ========  ==================  ==========  =====
preset language  vocab   Lmax  B x n     masking             props/seq   steps
=====  ========  ======  ====  ========  ==================  ==========  =====
1      arith     512     4     4 x 32    50 %                16          1
2      json      4096    6     8 x 128   U[0.25, 0.75]/seq   8           8
3      smiles    8192    4     16 x 256  60 %                8           16
4      clike     32768   8     16 x 256  70 %                16          4
5      clike     32768   8     64 x 1024 32-token blocks     16          32
=====  ========  ======  ====  ========  ==================  ==========  =====

Recipe (all draws from numpy PCG64 sub-streams of the seed):

* vocabulary: ids 0..|A|-1 are the single bytes of the language alphabet A in
  byte order (so every sentence can be tokenised); the remaining ids are
  strings of uniform length 1..Lmax with uniform bytes of A (duplicates kept);
* hidden answer: a random derivation of the grammar rendered to text (a
  generator device only), split into exactly n vocabulary tokens by sampling
  uniformly among all such splits;
* masks: uniform positions (preset 5: the answer is decoded in 32-token blocks;
  each sequence starts with its active block k ~ U{0..31}, earlier blocks
  unmasked, 80 % of block k masked, later blocks fully masked; when a block
  fills the next one becomes active with 20 % of it revealed);
* proposals per step and sequence: min(props, #masked) distinct masked
  positions (within the active block for preset 5); the token is the hidden
  token with probability 1/2, else uniform over the vocabulary; confidence is
  uniform float32 in [0, 1).

This module holds no lexing, validation or selection arithmetic; the commit
policy below only consumes verdicts and selections computed elsewhere.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np

from . import grammars as G

MASK = -1

PRESETS: Dict[int, dict] = {
    1: dict(lang="arith", vocab=512, lmax=4, B=4, n=32, mask=("ratio", 0.5), props=16, steps=1),
    2: dict(lang="json", vocab=4096, lmax=6, B=8, n=128, mask=("uniform", 0.25, 0.75), props=8, steps=8),
    3: dict(lang="smiles", vocab=8192, lmax=4, B=16, n=256, mask=("ratio", 0.6), props=8, steps=16),
    4: dict(lang="clike", vocab=32768, lmax=8, B=16, n=256, mask=("ratio", 0.7), props=16, steps=4),
    5: dict(lang="clike", vocab=32768, lmax=8, B=64, n=1024, mask=("block", 32, 0.8, 0.2), props=16, steps=32),
}

PRESET_NAMES = {
    1: "arith-E+T|T*F: vocab 512, 4x32 tokens, 50% masked, 16 proposals/seq, 1 step",
    2: "json-like: vocab 4096, 8x128 tokens, mask U[0.25,0.75], 64 proposals/step, 8 steps",
    3: "smiles-like: vocab 8192, 16x256 tokens, 60% masked, 128 proposals/step, 16 steps",
    4: "c-like: vocab 32768, 16x256 tokens, 70% masked, 256 proposals/step, 4 steps",
    5: "c-like: vocab 32768, 64x1024 tokens in 32-token blocks, up to 16 proposals/seq (1024/step) in the active block, 32 steps",
}


@dataclass
class Vocab:
    strings: List[bytes]

    @property
    def size(self) -> int:
        return len(self.strings)

    def csr(self) -> Tuple[np.ndarray, np.ndarray]:
        offs = np.zeros(self.size + 1, dtype=np.int32)
        offs[1:] = np.cumsum([len(s) for s in self.strings])
        return np.frombuffer(b"".join(self.strings), dtype=np.uint8).copy(), offs


def make_vocab(rng: np.random.Generator, alphabet: str, size: int, lmax: int) -> Vocab:
    singles = sorted(set(alphabet.encode()))
    if size < len(singles):
        raise ValueError("vocabulary smaller than the alphabet")
    A = np.array(singles, dtype=np.uint8)
    out = [bytes([c]) for c in singles]
    for _ in range(size - len(singles)):
        L = int(rng.integers(1, lmax + 1))
        out.append(bytes(A[rng.integers(0, len(A), size=L)].tolist()))
    return Vocab(out)


def _segment(rng: np.random.Generator, text: bytes, vocab_index: Dict[bytes, List[int]], lmax: int,
             n: int) -> Optional[List[int]]:
    """Split `text` into exactly n vocabulary tokens, uniformly over all splits
    (duplicate strings count as distinct tokens).  None if impossible."""
    L = len(text)
    if L < n:
        return None
    NEG = -np.inf
    lw = np.full((L + 1, n + 1), NEG)
    lw[L, 0] = 0.0
    opts: List[List[Tuple[int, List[int]]]] = [[] for _ in range(L)]
    for i in range(L - 1, -1, -1):
        acc = np.full(n + 1, NEG)
        for ln in range(1, min(lmax, L - i) + 1):
            ids = vocab_index.get(text[i:i + ln])
            if not ids:
                continue
            opts[i].append((ln, ids))
            shifted = np.full(n + 1, NEG)
            shifted[1:] = lw[i + ln, :-1] + np.log(len(ids))
            acc = np.logaddexp(acc, shifted)
        lw[i] = acc
    if not np.isfinite(lw[0, n]):
        return None
    out: List[int] = []
    i, k = 0, n
    while i < L:
        ws = np.array([np.log(len(ids)) + lw[i + ln, k - 1] for ln, ids in opts[i]])
        p = np.exp(ws - lw[i, k])
        p = p / p.sum()
        j = int(rng.choice(len(opts[i]), p=p))
        ln, ids = opts[i][j]
        out.append(ids[int(rng.integers(len(ids)))])
        i += ln
        k -= 1
    assert k == 0 and len(out) == n
    return out


@dataclass
class Instance:
    preset: int
    seed: int
    lang: G.Language
    vocab: Vocab
    hidden: np.ndarray  # int32 [B, n]
    seqs: np.ndarray  # int32 [B, n], MASK = -1
    texts: List[str]
    active_block: Optional[np.ndarray] = None  # preset 5 only
    prop_rng: np.random.Generator = field(default=None, repr=False)
    cfg: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return int(self.seqs.shape[0])

    @property
    def n(self) -> int:
        return int(self.seqs.shape[1])


def make_instance(preset: int, seed: int = 42, B: Optional[int] = None, n: Optional[int] = None) -> Instance:
    cfg = dict(PRESETS[preset])
    if B is not None:
        cfg["B"] = B
    if n is not None:
        cfg["n"] = n
    lang = G.language(cfg["lang"])
    ss = np.random.SeedSequence([seed, preset])
    r_vocab, r_sent, r_mask, r_prop = [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4)]
    vocab = make_vocab(r_vocab, lang.alphabet, cfg["vocab"], cfg["lmax"])
    index: Dict[bytes, List[int]] = {}
    for i, s in enumerate(vocab.strings):
        index.setdefault(s, []).append(i)
    Bn, n_ = cfg["B"], cfg["n"]
    hidden = np.zeros((Bn, n_), dtype=np.int32)
    texts = []
    for b in range(Bn):
        slack = max(2, n_ // 16)
        for _attempt in range(2000):
            tb = G.TextBuilder(lang, r_sent, extra_space=0.15)
            if not lang.top(tb, n_, n_ + slack):
                continue
            text = tb.text
            seg = _segment(r_sent, text.encode(), index, cfg["lmax"], n_)
            if seg is not None:
                break
        else:
            raise RuntimeError("could not generate a sentence of the requested token length")
        hidden[b] = seg
        texts.append(text)
    seqs = hidden.copy()
    active = None
    kind = cfg["mask"][0]
    if kind == "ratio":
        m = int(round(cfg["mask"][1] * n_))
        for b in range(Bn):
            seqs[b, r_mask.choice(n_, m, replace=False)] = MASK
    elif kind == "uniform":
        for b in range(Bn):
            r = r_mask.uniform(cfg["mask"][1], cfg["mask"][2])
            m = int(round(r * n_))
            seqs[b, r_mask.choice(n_, m, replace=False)] = MASK
    elif kind == "block":
        bs, ratio = cfg["mask"][1], cfg["mask"][2]
        nblk = n_ // bs
        active = r_mask.integers(0, nblk, size=Bn).astype(np.int32)
        for b in range(Bn):
            k = int(active[b])
            seqs[b, (k + 1) * bs:] = MASK
            m = int(round(ratio * bs))
            seqs[b, k * bs + r_mask.choice(bs, m, replace=False)] = MASK
    else:
        raise ValueError(kind)
    return Instance(preset, seed, lang, vocab, hidden, seqs, texts, active, r_prop, cfg)


@dataclass
class Proposals:
    seq: np.ndarray  # int32 [C]
    pos: np.ndarray  # int32 [C]
    tok: np.ndarray  # int32 [C]
    conf: np.ndarray  # float32 [C]

    @property
    def C(self) -> int:
        return int(self.seq.shape[0])


def propose(inst: Instance) -> Proposals:
    """Draw this step's proposals from the instance's proposal stream."""
    rng = inst.prop_rng
    props = inst.cfg["props"]
    V = inst.vocab.size
    S, P, T, F = [], [], [], []
    for b in range(inst.B):
        masked = np.flatnonzero(inst.seqs[b] == MASK)
        if inst.active_block is not None:
            bs = inst.cfg["mask"][1]
            k = int(inst.active_block[b])
            masked = masked[(masked >= k * bs) & (masked < (k + 1) * bs)]
        m = min(props, len(masked))
        if m == 0:
            continue
        pos = rng.choice(masked, m, replace=False).astype(np.int32)
        keep = rng.random(m) < 0.5
        tok = np.where(keep, inst.hidden[b, pos], rng.integers(0, V, size=m)).astype(np.int32)
        conf = rng.random(m, dtype=np.float32)
        S.append(np.full(m, b, dtype=np.int32))
        P.append(pos)
        T.append(tok)
        F.append(conf)
    if not S:
        z = np.zeros(0, dtype=np.int32)
        return Proposals(z, z.copy(), z.copy(), np.zeros(0, dtype=np.float32))
    return Proposals(np.concatenate(S), np.concatenate(P), np.concatenate(T), np.concatenate(F))


def commit(inst: Instance, props: Proposals, verdict: np.ndarray, selected: np.ndarray) -> np.ndarray:
    """Harness commit policy: commit the selected subset; if a sequence's
    subset is empty but it has a valid candidate, commit its single
    highest-confidence valid candidate (ties to the lower index).  Returns the
    per-candidate commit mask.  Preset 5 then advances filled blocks."""
    committed = np.zeros(props.C, dtype=np.uint8)
    for b in range(inst.B):
        idx = np.flatnonzero(props.seq == b)
        if idx.size == 0:
            continue
        sel = idx[selected[idx] == 1]
        if sel.size:
            committed[sel] = 1
        else:
            val = idx[verdict[idx] == 1]
            if val.size:
                best = val[0]
                for c in val[1:]:
                    if props.conf[c] > props.conf[best]:
                        best = c
                committed[best] = 1
    for c in np.flatnonzero(committed):
        inst.seqs[props.seq[c], props.pos[c]] = props.tok[c]
    if inst.active_block is not None:
        bs, reveal = inst.cfg["mask"][1], inst.cfg["mask"][3]
        nblk = inst.n // bs
        for b in range(inst.B):
            k = int(inst.active_block[b])
            if k + 1 < nblk and not np.any(inst.seqs[b, k * bs:(k + 1) * bs] == MASK):
                k += 1
                inst.active_block[b] = k
                r = int(round(reveal * bs))
                pos = k * bs + inst.prop_rng.choice(bs, r, replace=False)
                inst.seqs[b, pos] = inst.hidden[b, pos]
    return committed


@dataclass
class StepRecord:
    seqs: np.ndarray
    props: Proposals
    verdict: np.ndarray
    selected: np.ndarray
    committed: np.ndarray


def run_steps(inst: Instance, validate: Callable, select: Callable, steps: Optional[int] = None) -> List[StepRecord]:
    """Drive `steps` denoising steps: propose -> validate -> select -> commit.
    ``validate(seqs, props) -> uint8[C]`` and ``select(seqs, props, verdict) -> uint8[C]``."""
    steps = inst.cfg["steps"] if steps is None else steps
    out = []
    for _ in range(steps):
        props = propose(inst)
        x = inst.seqs.copy()
        v = np.asarray(validate(x, props), dtype=np.uint8)
        s = np.asarray(select(x, props, v), dtype=np.uint8)
        c = commit(inst, props, v, s)
        out.append(StepRecord(x, props, v, s, c))
    return out


@dataclass
class Arrays:
    """Lexer DFA, grammar and vocabulary as the plain arrays both sides consume."""

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


def arrays(lang: G.Language, vocab: Vocab) -> Arrays:
    tb = lang.tables
    T, N, start, lhs, roff, rhs = lang.grammar.arrays()
    vb, vo = vocab.csr()
    return Arrays(tb.trans, tb.accept, T, N, start, lhs, roff, rhs, vb, vo)
