"""The grammar padding used to reach 2- and 8-word item sets keeps the
language: the oracle's verdicts on a workload step are the same with and
without it (CPU only)."""
import numpy as np

from paper_2606_00722_amd import workloads as W
from tests.util import pad_language, packed_words


def test_padding_keeps_verdicts_and_widens_items(oracle_lib):
    inst = W.make_instance(1, 42)
    pr = W.propose(inst)
    padded = pad_language(inst.lang)
    assert packed_words(inst.lang.grammar) == 1 and packed_words(padded.grammar) == 2
    p0 = oracle_lib.problem_from(inst.lang, inst.vocab)
    p1 = oracle_lib.problem_from(padded, inst.vocab)
    v0 = oracle_lib.validate_batch(p0, inst.seqs, pr.seq, pr.pos, pr.tok, 4)
    v1 = oracle_lib.validate_batch(p1, inst.seqs, pr.seq, pr.pos, pr.tok, 4)
    assert v0.sum() > 0 and (v0 == 0).sum() > 0
    assert np.array_equal(v0, v1)
