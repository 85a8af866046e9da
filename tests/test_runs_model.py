"""A CPU model of how the walk settles a chain-like input that forms few runs
(a run: rows each of which shares a feature with the row before it), checked
against the oracle's sequential levels (Theorem 2's conflict levels).

Within a run starting at row a, levels rise by one at least from row to row,
so only writers before a can decide a level:
    level(j) = j + 1 + max over a <= t <= j of (M_t - t),
M_t the largest level among row t's writers before a (0 if none).  The grid
settles one run at a time: G blocks each own a stretch of the run's rows and
stage the stretch's prefix maxima of M_t - t; a block's levels add the maxima
of the stretches before it, and are written while the next run gathers its
M -- where a writer in the run just settled has its level formed from those
staged values.  Planted mistakes (writers in the run just settled ignored, a
stretch ignoring the stretches before it, the settled run read from the level
array before it is written) must be caught.  Plain Python: no kernel code is run and
none is shared."""
import random

import numpy as np
import pytest

import oracle

NONE = -(1 << 40)


def prev_rows(rows):
    last, prev = {}, []
    for i, r in enumerate(rows):
        prev.append([last.get(f, -1) for f in sorted(r)])
        for f in r:
            last[f] = i
    return prev


def runs_levels(rows, G, plant=None):
    n = len(rows)
    prev = prev_rows(rows)
    starts = [i for i in range(n) if i == 0 or (i - 1) not in prev[i]] + [n]
    level = [0] * n          # final levels (written one run late)
    stg = [NONE] * n         # staged prefix maxima
    pre, pa, ps, stretch = None, 0, 1, (0, 0)
    def settle_previous():   # the run just settled: every block's stretch
        for j in range(G):
            lo, hi = stretch[j]
            for t in range(lo, hi):
                level[t] = t + 1 + max(pre[j], stg[t])

    for k in range(len(starts) - 1):
        a, b = starts[k], starts[k + 1]
        # M of this run's rows; the run just settled is written in the same
        # step, so the model gathers first (the order that can go wrong)
        M = {t: 0 for t in range(a, b)}
        for t in range(a, b):
            for w in prev[t]:
                if w < 0 or w >= a:
                    continue
                if k > 0 and w >= pa:
                    if plant == "skip_settled":
                        continue
                    lw = level[w] if plant == "read_early" else \
                        w + 1 + max(pre[(w - pa) // ps], stg[w])
                else:
                    lw = level[w]
                M[t] = max(M[t], lw)
        if k > 0:
            settle_previous()
        span = (b - a + G - 1) // G
        bmax, stretch = [], []
        for j in range(G):
            lo = min(b, a + j * span)
            hi = min(b, lo + span)
            carry = NONE
            for t in range(lo, hi):
                carry = max(carry, M[t] - t)
                stg[t] = carry
            bmax.append(carry)
            stretch.append((lo, hi))
        pre = [NONE if plant == "no_before" else max(bmax[:j], default=NONE) for j in range(G)]
        pa, ps = a, span
    if len(starts) > 1:
        settle_previous()
    return level, len(starts) - 1


def chain_like(rng, n, d, hot_p=0.85):
    rows = []
    for _ in range(n):
        r = set(rng.sample(range(2, d), rng.randint(0, 4)))
        if rng.random() < hot_p:
            r.add(0 if rng.random() < 0.6 else 1)
        rows.append(r)
    return rows


def oracle_levels(rows, d):
    row_ptr = np.zeros(len(rows) + 1, np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in sorted(r)], np.int32)
    return list(oracle.levels_seq(row_ptr, col, d, len(rows))[0])


@pytest.mark.parametrize("seed", range(12))
def test_runs_model_equals_sequential_levels(seed):
    rng = random.Random(seed)
    n, d = rng.randint(1, 300), rng.randint(4, 80)
    rows = chain_like(rng, n, d)
    want = oracle_levels(rows, d)
    for G in (1, 2, 3, 7, 16):
        got, _ = runs_levels(rows, G)
        assert got == want, (seed, G)


@pytest.mark.parametrize("plant", ["skip_settled", "no_before", "read_early"])
def test_runs_model_planted_mistakes_caught(plant):
    caught = 0
    for seed in range(30):
        rng = random.Random(100 + seed)
        rows = chain_like(rng, 200, 40, hot_p=0.7)
        if runs_levels(rows, 5, plant)[0] != oracle_levels(rows, 40):
            caught += 1
    assert caught > 0, "a planted mistake in the run decomposition went unnoticed"
