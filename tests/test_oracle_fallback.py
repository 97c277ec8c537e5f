"""Pins of the oracle's sequential fallback (the loop after the relaxed batch
in EPIC decoding): it commits only what the exact check justifies, in
confidence order, and no more than the step's budget."""
import numpy as np

from paper_2606_00722_amd import workloads as W


def _step(oracle_lib, preset, seed=42):
    inst = W.make_instance(preset, seed)
    pr = W.propose(inst)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    v = oracle_lib.validate_batch(p, inst.seqs, pr.seq, pr.pos, pr.tok, 4)
    return inst, pr, p, v


def test_budget_met_by_the_batch_commits_nothing(oracle_lib):
    inst, pr, p, v = _step(oracle_lib, 1)
    sel, _, st = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v)
    assert st == 0
    nb = np.array([int(sel[pr.seq == b].sum()) for b in range(inst.B)])
    acc, st = oracle_lib.fallback(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, sel, nb)
    assert st == 0 and acc.sum() == 0


def test_first_commit_is_the_most_confident_valid_candidate(oracle_lib):
    inst, pr, p, v = _step(oracle_lib, 1)
    none = np.zeros(len(pr.seq), np.uint8)
    acc, st = oracle_lib.fallback(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, none, np.ones(inst.B, np.int64))
    assert st == 0
    for b in range(inst.B):
        mine = np.flatnonzero(pr.seq == b)
        ok = [c for c in mine if v[c] == 1]
        want = min(ok, key=lambda c: (-float(pr.conf[c]), c)) if ok else None
        got = np.flatnonzero(acc[mine])
        assert (len(got) == 0) if want is None else (list(mine[got]) == [want])


def test_commits_are_valid_within_budget_and_never_invalid_candidates(oracle_lib):
    for preset in (1, 2):
        inst, pr, p, v = _step(oracle_lib, preset)
        sel, _, st = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v)
        assert st == 0
        rng = np.random.default_rng(preset)
        nc = rng.integers(0, inst.cfg["props"] + 2, size=inst.B)
        acc, st = oracle_lib.fallback(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v, sel, nc)
        assert st == 0
        assert not np.any(acc & (v != 1)) and not np.any(acc & sel)
        for b in range(inst.B):
            mine = pr.seq == b
            assert acc[mine].sum() <= max(0, nc[b] - sel[mine].sum())
            x = inst.seqs[b].copy()
            for c in np.flatnonzero(mine & ((sel == 1) | (acc == 1))):
                x[pr.pos[c]] = pr.tok[c]
            if sel[mine].sum() + acc[mine].sum():  # whatever was committed keeps x_b completable
                assert oracle_lib.valid(p, x) == 1


def test_invalid_candidates_stay_invalid_after_commits(oracle_lib):
    """The reading the device's fallback relies on: filling masked positions
    only shrinks the character language of x, so a candidate invalid on x is
    invalid on x with Alg. 4's batch committed (checked for every verdict-0
    candidate of two workloads)."""
    checked = 0
    for preset in (1, 2):
        inst, pr, p, v = _step(oracle_lib, preset)
        sel, _, st = oracle_lib.select(p, inst.seqs, pr.seq, pr.pos, pr.tok, pr.conf, v)
        assert st == 0
        for b in range(inst.B):
            mine = pr.seq == b
            x = inst.seqs[b].copy()
            for c in np.flatnonzero(mine & (sel == 1)):
                x[pr.pos[c]] = pr.tok[c]
            for c in np.flatnonzero(mine & (v == 0)):
                if x[pr.pos[c]] != -1:
                    continue
                y = x.copy()
                y[pr.pos[c]] = pr.tok[c]
                assert oracle_lib.valid(p, y) == 0
                checked += 1
    assert checked > 10


def test_no_limit_on_the_number_of_candidates(oracle_lib):
    """Alg. 1's loop has no cap on the candidates it walks: one sequence with
    every masked position proposed with its hidden token (about a hundred
    candidates, each valid, and jointly valid since the hidden answer fills
    them) commits exactly the budget, in confidence order."""
    inst = W.make_instance(1, 42, B=1, n=200)
    masked = np.flatnonzero(inst.seqs[0] == W.MASK).astype(np.int32)
    assert len(masked) > 64
    C = len(masked)
    seq = np.zeros(C, np.int32)
    tok = inst.hidden[0, masked].astype(np.int32)
    conf = np.random.default_rng(7).random(C, dtype=np.float32)
    p = oracle_lib.problem_from(inst.lang, inst.vocab)
    v = np.ones(C, np.uint8)
    budget = 70
    acc, st = oracle_lib.fallback(p, inst.seqs, seq, masked, tok, conf, v, np.zeros(C, np.uint8), [budget])
    assert st == 0 and int(acc.sum()) == budget
    order = sorted(range(C), key=lambda c: (-float(conf[c]), c))
    assert set(np.flatnonzero(acc).tolist()) == set(order[:budget])
