"""Pins for the oracle's conflict levels, grouping, transpose and previous writer.

Pins, not re-derivations:
  * the invariants I1-I3 below characterise the earliest layering uniquely
    (induction on the example index), checked here by direct enumeration;
  * closed forms for structured inputs (fully conflicting, disjoint, chains);
  * the grouping is checked against numpy's lexicographic sort, the
    transpose against scipy's CSR->CSC conversion.
"""
import itertools

import numpy as np
import pytest
import scipy.sparse as sp

import datagen
import oracle


def csr_from_rows(rows):
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in sorted(r)], dtype=np.int32)
    return row_ptr, col


def rows_of(row_ptr, col):
    return [set(col[row_ptr[i]:row_ptr[i + 1]].tolist()) for i in range(len(row_ptr) - 1)]


def check_invariants(rows, level):
    """I1: examples of one level share no feature.  I2: an earlier example
    sharing a feature has a strictly lower level.  I3: an example of level
    l > 1 has an earlier conflicting example at level l - 1.  Levels >= 1."""
    n = len(rows)
    for i in range(n):
        assert level[i] >= 1
        conflicting = [j for j in range(i) if rows[i] & rows[j]]
        for j in conflicting:
            assert level[j] < level[i]                       # I2
        if level[i] > 1:
            assert any(level[j] == level[i] - 1 for j in conflicting)   # I3
        for j in range(n):
            if j != i and level[j] == level[i]:
                assert not (rows[i] & rows[j])               # I1


def random_rows(rng, n, d, max_m):
    return [set(rng.choice(d, size=rng.integers(0, max_m + 1), replace=False).tolist())
            for _ in range(n)]


@pytest.mark.parametrize("seed", range(40))
def test_seq_equals_brute_and_invariants(seed):
    rng = np.random.default_rng(seed)
    n, d = int(rng.integers(1, 60)), int(rng.integers(1, 14))
    rows = random_rows(rng, n, d, min(d, 4))
    row_ptr, col = csr_from_rows(rows)
    lv_s, L_s = oracle.levels_seq(row_ptr, col, d)
    lv_b, L_b = oracle.levels_brute(row_ptr, col)
    assert np.array_equal(lv_s, lv_b) and L_s == L_b == lv_s.max()
    check_invariants(rows, lv_s)


def test_exhaustive_small_patterns():
    # every sparsity pattern with n <= 4 examples over d = 3 features, plus
    # every pattern of 5 examples drawn from a subset family
    subsets = [set(s) for k in range(4) for s in itertools.combinations(range(3), k)]
    count = 0
    for n in range(1, 5):
        for rows in itertools.product(subsets, repeat=n):
            row_ptr, col = csr_from_rows(list(rows))
            lv, L = oracle.levels_seq(row_ptr, col, 3)
            check_invariants(list(rows), lv)
            lb, _ = oracle.levels_brute(row_ptr, col)
            assert np.array_equal(lv, lb)
            count += 1
    assert count == sum(8 ** n for n in range(1, 5))
    for rows in itertools.product(subsets[1:5], repeat=5):
        row_ptr, col = csr_from_rows(list(rows))
        lv, _ = oracle.levels_seq(row_ptr, col, 3)
        check_invariants(list(rows), lv)


def test_closed_forms():
    n = 37
    # fully conflicting: every example holds feature 0 -> levels 1..n
    lv, L = oracle.levels_seq(*csr_from_rows([{0, 1 + i % 5} for i in range(n)]), 6)
    assert lv.tolist() == list(range(1, n + 1)) and L == n
    # pairwise disjoint -> one level
    lv, L = oracle.levels_seq(*csr_from_rows([{2 * i, 2 * i + 1} for i in range(n)]), 2 * n)
    assert lv.tolist() == [1] * n and L == 1
    # a chain i -> i+1 through feature i+1 -> levels 1..n
    lv, _ = oracle.levels_seq(*csr_from_rows([{i, i + 1} for i in range(n)]), n + 1)
    assert lv.tolist() == list(range(1, n + 1))
    # two interleaved chains -> ceil((i+1)/2)
    lv, _ = oracle.levels_seq(*csr_from_rows([{i % 2} for i in range(n)]), 2)
    assert lv.tolist() == [(i + 2) // 2 for i in range(n)]
    # empty examples conflict with nothing -> level 1
    lv, _ = oracle.levels_seq(*csr_from_rows([{0}, set(), {0}, set()]), 1)
    assert lv.tolist() == [1, 1, 2, 1]
    # no examples
    lv, L = oracle.levels_seq(np.zeros(1, np.int64), np.zeros(0, np.int32), 4)
    assert len(lv) == 0 and L == 0


@pytest.mark.parametrize("seed", range(10))
def test_bucket_against_lexsort(seed):
    rng = np.random.default_rng(100 + seed)
    rows = random_rows(rng, 300, 25, 4)
    row_ptr, col = csr_from_rows(rows)
    level, L = oracle.levels_seq(row_ptr, col, 25)
    perm, level_ptr = oracle.bucket(level, L)
    ref = np.lexsort((np.arange(len(level)), level))
    assert np.array_equal(perm, ref)
    assert level_ptr[0] == 0 and level_ptr[-1] == len(level)
    assert np.array_equal(np.diff(level_ptr), np.bincount(level, minlength=L + 1)[1:])


@pytest.mark.parametrize("seed", range(10))
def test_transpose_and_prev_writer(seed):
    rng = np.random.default_rng(200 + seed)
    n, d = 200, 30
    rows = random_rows(rng, n, d, 6)
    row_ptr, col = csr_from_rows(rows)
    col_ptr, csc_row = oracle.transpose(row_ptr, col, d)
    A = sp.csr_matrix((np.ones(len(col)), col, row_ptr), shape=(n, d)).tocsc()
    A.sort_indices()
    assert np.array_equal(col_ptr, A.indptr) and np.array_equal(csc_row, A.indices)
    prev = oracle.prev_writer(row_ptr, col, d)
    for i in range(n):
        for p in range(row_ptr[i], row_ptr[i + 1]):
            earlier = [j for j in range(i) if col[p] in rows[j]]
            assert prev[p] == (max(earlier) if earlier else -1)


def test_config1_level_statistics():
    # the structure of the 10k x 1k Zipf(1.0) workload: about 9.0e3 levels of
    # mean width about 1.1 (independent estimate with a different generator)
    g = datagen.generate(1)
    level, L = oracle.levels_seq(g["row_ptr"], g["col"], g["d"])
    assert 8500 <= L <= 9500
    widths = np.bincount(level)[1:]
    assert widths.max() <= 8 and abs(g["n"] / L - 1.11) < 0.06


@pytest.mark.slow
def test_config2_level_statistics():
    g = datagen.generate(2)
    level, L = oracle.levels_seq(g["row_ptr"], g["col"], g["d"])
    assert abs(L - 999_785) < 2000
