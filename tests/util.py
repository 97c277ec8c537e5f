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
