"""The paper's execution histories (Fig. 1, Fig. 3) and its theorems as
properties of the history predicates, then the link to conflict levels:
a level-by-level execution keeps every feature's accesses serial."""
import itertools
import os

import numpy as np
import pytest

import datagen
import oracle
from oracle import history as H

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "histories.txt")


def golden():
    out = []
    for line in open(GOLDEN):
        if not line.strip() or line.startswith("#"):
            continue
        name, s, b, r, text = [x.strip() for x in line.split("|")]
        out.append((name, bool(int(s)), bool(int(b)), bool(int(r)), H.parse(text)))
    return out


def test_golden_verdicts():
    rows = golden()
    assert [r[0] for r in rows] == ["SEQ1", "SEQ2", "H1", "H2", "H3"]
    for name, seq, bsp, rcwc, h in rows:
        assert H.sequential(h) == seq, name
        assert H.bsp(h) == bsp, name
        assert H.rcwc(h) == rcwc, name
        # with every partition touched in every iteration, the per-partition
        # conditions of the proof of Theorem 2 coincide with RC + WC
        assert H.partition_serial(h) == rcwc, name


def all_two_worker_histories():
    """Every interleaving of 2 workers x 2 iterations over {pi_1, pi_2} in
    which each worker issues, per iteration, its two reads then its write."""
    progs = {}
    for wk in (1, 2):
        ops = []
        for it in (1, 2):
            ops += [("r", wk, 1, it), ("r", wk, 2, it), ("w", wk, wk, it)]
        progs[wk] = ops
    n1, n2 = len(progs[1]), len(progs[2])
    for pos in itertools.combinations(range(n1 + n2), n1):
        h, a, b = [], 0, 0
        pos = set(pos)
        for t in range(n1 + n2):
            if t in pos:
                h.append(progs[1][a]); a += 1
            else:
                h.append(progs[2][b]); b += 1
        yield h


def test_theorems_as_properties():
    n = n_bsp = n_rcwc = 0
    for h in all_two_worker_histories():
        n += 1
        if H.bsp(h):
            n_bsp += 1
            assert H.sequential(h)         # Theorem 1
            assert H.rcwc(h)               # Theorem 3
        if H.rcwc(h):
            n_rcwc += 1
            assert H.partition_serial(h)   # Theorem 2 (per-partition serial)
    assert n == 924 and 0 < n_bsp < n_rcwc < n    # RC/WC admits strictly more


@pytest.mark.parametrize("seed", range(5))
def test_level_execution_is_partition_serial(seed):
    g = datagen.generate(1, n=400, d=60, seed=seed)
    level, L = oracle.levels_seq(g["row_ptr"], g["col"], g["d"])
    h = H.level_history(g["row_ptr"], g["col"], level)
    assert H.partition_serial(h)
    assert H.partition_serial(H.level_history(g["row_ptr"], g["col"], level,
                                              within=lambda m: m[::-1]))
    # one level lower for an example breaks its feature order
    i = int(np.nonzero(level > 1)[0][0])
    bad = level.copy()
    bad[i] -= 1
    assert not H.partition_serial(H.level_history(g["row_ptr"], g["col"], bad))
