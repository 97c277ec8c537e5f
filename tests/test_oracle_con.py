"""Pins for the prior pipeline ("Con.", Sec. 2 and App. A.1-A.2), the CPU
comparator that the benchmark times beside the oracle: lexing automaton,
subset construction, Hopcroft minimisation, intersection emptiness.  It decides
the same completable criterion by another route, so its verdicts must equal
Valid; Hopcroft's minimal DFA must have as many states as Moore's (both are
the minimal automaton of the same language)."""
import numpy as np
import pytest

from paper_2606_00722_amd import grammars as G
from paper_2606_00722_amd import workloads as W
from tests import refimpl
from tests.util import custom_vocab


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
def test_con_equals_valid_and_bar_hillel(oracle_lib, name):
    """Random short sequences over tiny languages, each with a candidate at a
    masked position: the prior pipeline's verdict equals Valid and the Python
    intersection-grammar check; Hopcroft and Moore give DFAs of equal size."""
    lang, vocab, xs = _tiny(name, 60, 6, 91)
    p = oracle_lib.problem_from(lang, vocab)
    rng = np.random.default_rng(3)
    seen = set()
    for x in xs:
        masked = np.flatnonzero(x < 0)
        if masked.size == 0:
            continue
        i, t = int(masked[0]), int(rng.integers(0, vocab.size))
        got, ms = oracle_lib.con_validate_batch(p, x[None, :], [0], [i], [t])
        z = x.copy()
        z[i] = t
        assert got[0] == oracle_lib.valid(p, z)
        assert got[0] == int(refimpl.bar_hillel_valid(lang, vocab.strings, z))
        seen.add(int(got[0]))
        assert oracle_lib.con_dfa_states(p, x) == oracle_lib.dfa_states(p, x)
        assert (ms >= 0).all()
    assert seen == {0, 1}


@pytest.mark.parametrize("preset,B,n", [(1, 4, 32), (2, 3, 48), (3, 2, 40)])
def test_con_equals_oracle_on_workload_candidates(oracle_lib, preset, B, n):
    """Step-1 candidates of shortened workloads: the prior pipeline and the
    oracle agree on every verdict, and the minimal DFAs have equal sizes."""
    inst = W.make_instance(preset, 5, B=B, n=n)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    pr = W.propose(inst)
    got, ms = oracle_lib.con_validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, 4)
    want = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, 4)
    assert np.array_equal(got, want)
    assert 0 < int(want.sum()) < len(want)
    assert ms.sum() > 0
    for b in range(inst.B):
        assert oracle_lib.con_dfa_states(p, inst.seqs[b]) == oracle_lib.dfa_states(p, inst.seqs[b])
