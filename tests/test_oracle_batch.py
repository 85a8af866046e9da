"""Pins for the oracle's mini-batch gradient descent (Sec. 6.3: a batch of B
examples per iteration), independent of its own arithmetic:

  * batch size 1 is the SGD oracle bit for bit (levels, union, epoch);
  * batch levels: brute force from the definition equals the one-pass sweep,
    and the invariants that characterise the layering (no two batches of a
    level share a feature; every conflicting earlier batch is lower; every
    batch above level 1 has a conflicting batch one level down) hold;
    closed forms (one shared feature: 1..nb; disjoint batches: all 1);
  * the union and its occurrence lists against numpy (unique, lexsort);
  * reads before writes (Definition 3): a dyadic least-squares closed form
    in which all examples of a batch see the batch-start weights
    (w_k = 1 - 2^-k with lr = 1/4 and two examples per batch, unlike
    sequential SGD), and the logistic first-touch form;
  * the step against an fp64 central-difference gradient of the batch loss;
  * Theorem 2 over batches: any order that runs batch levels in increasing
    order is bitwise the sequential result; breaking one conflict is not.
"""
import math

import numpy as np
import pytest

import datagen
import oracle
from oracle import LOGISTIC, MATCHED, NATURAL, SQUARED


def random_csr(rng, n, d, max_m):
    rows = [sorted(rng.choice(d, rng.integers(0, min(max_m, d) + 1), replace=False)) for _ in range(n)]
    row_ptr = np.zeros(n + 1, np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in r], np.int32)
    return row_ptr, col


def batch_features(row_ptr, col, B, b):
    n = len(row_ptr) - 1
    return set(col[row_ptr[b * B]:row_ptr[min((b + 1) * B, n)]].tolist())


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_batch_of_one_is_sgd(cfg, mode):
    g = datagen.generate(cfg, n=3000, d=2000 if cfg == 4 else 300, seed=11)
    lv1, L1 = oracle.batch_levels_seq(g["row_ptr"], g["col"], g["d"], 1)
    lv, L = oracle.levels_seq(g["row_ptr"], g["col"], g["d"])
    assert L1 == L and np.array_equal(lv1, lv)
    bptr, ucol, uptr, occ = oracle.batch_union(g["row_ptr"], g["col"], g["d"], 1)
    assert np.array_equal(bptr, g["row_ptr"]) and np.array_equal(ucol, g["col"])
    assert np.array_equal(occ, np.arange(len(g["col"])))
    w0 = np.zeros(g["d"], np.float32)
    a = oracle.batch_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], mode, 1)
    b = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], mode)
    assert np.array_equal(a.view(np.int32), b.view(np.int32))


@pytest.mark.parametrize("seed", range(30))
def test_batch_levels_brute_equals_sweep_and_invariants(seed):
    rng = np.random.default_rng(seed)
    n, d = int(rng.integers(1, 60)), int(rng.integers(1, 25))
    row_ptr, col = random_csr(rng, n, d, 4)
    for B in (1, 2, 3, 7, n, n + 5):
        brute, Lb = oracle.batch_levels_brute(row_ptr, col, B)
        seq, Ls = oracle.batch_levels_seq(row_ptr, col, d, B)
        assert Lb == Ls and np.array_equal(brute, seq)
        nb = oracle.n_batches(n, B)
        feats = [batch_features(row_ptr, col, B, b) for b in range(nb)]
        for b in range(nb):
            earlier = [a for a in range(b) if feats[a] & feats[b]]
            for a in earlier:
                assert seq[a] < seq[b]                       # conflicting earlier batch is lower
            if seq[b] > 1:                                   # tightness
                assert any(seq[a] == seq[b] - 1 for a in earlier)
            else:
                assert not earlier
        for l in range(1, Ls + 1):                           # a level is feature-disjoint
            members = [b for b in range(nb) if seq[b] == l]
            for i, a in enumerate(members):
                for c in members[i + 1:]:
                    assert not (feats[a] & feats[c])


def test_batch_levels_closed_forms():
    n = 50
    shared = [{0, 1 + i % 9} for i in range(n)]
    disjoint = [{2 * i, 2 * i + 1} for i in range(n)]
    for rows, expect in ((shared, lambda nb: np.arange(1, nb + 1)), (disjoint, lambda nb: np.ones(nb))):
        row_ptr = np.zeros(n + 1, np.int64)
        row_ptr[1:] = np.cumsum([len(r) for r in rows])
        col = np.array([c for r in rows for c in sorted(r)], np.int32)
        for B in (1, 4, 7, 50):
            lv, L = oracle.batch_levels_seq(row_ptr, col, int(col.max()) + 1, B)
            assert np.array_equal(lv, expect(oracle.n_batches(n, B)))
    # batches of two alternating single-feature examples {0}, {1}: every batch
    # touches both features, so the batches form one chain
    row_ptr = np.arange(n + 1, dtype=np.int64)
    col = (np.arange(n) % 2).astype(np.int32)
    lv, L = oracle.batch_levels_seq(row_ptr, col, 2, 2)
    assert np.array_equal(lv, np.arange(1, 26))
    lv, L = oracle.batch_levels_seq(row_ptr, col, 2, 1)      # as SGD: two interleaved chains
    assert np.array_equal(lv, (np.arange(n) // 2) + 1)


@pytest.mark.parametrize("seed", range(10))
def test_batch_union_against_numpy(seed):
    rng = np.random.default_rng(100 + seed)
    n, d = int(rng.integers(1, 200)), int(rng.integers(1, 60))
    row_ptr, col = random_csr(rng, n, d, 6)
    for B in (1, 3, 10, n + 1):
        bptr, ucol, uptr, occ = oracle.batch_union(row_ptr, col, d, B)
        row_of = np.repeat(np.arange(n), np.diff(row_ptr))
        bat = row_of // B
        order = np.lexsort((np.arange(len(col)), col, bat))   # by batch, feature, entry
        assert np.array_equal(occ, order)
        key = bat[order].astype(np.int64) * (d + 1) + col[order]
        first = np.ones(len(key), bool)
        first[1:] = key[1:] != key[:-1]
        assert np.array_equal(ucol, col[order][first])
        assert np.array_equal(uptr[:-1], np.nonzero(first)[0]) and uptr[-1] == len(col)
        nb = oracle.n_batches(n, B)
        assert np.array_equal(bptr, np.searchsorted(bat[order][first], np.arange(nb + 1)))


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_least_squares_batch_reads_before_writes(mode):
    # one feature, x = 1, y = 1, lr = 1/4, two examples per batch: both see the
    # batch-start w, so w <- w + 2 * (1 - w)/4 = (w + 1)/2 and w_k = 1 - 2^-k
    # after k batches; sequential SGD with the same lr gives 1 - (3/4)^m instead
    for k in range(1, 20):
        m = 2 * k
        row_ptr, col = np.arange(m + 1, dtype=np.int64), np.zeros(m, np.int32)
        one = np.ones(m, np.float32)
        w = oracle.batch_epoch(row_ptr, col, one, one, np.zeros(1, np.float32), 0.25, SQUARED, mode, 2)
        assert w[0] == np.float32(1.0 - 2.0 ** -k)
        w_sgd = oracle.sgd_epoch(row_ptr, col, one, one, np.zeros(1, np.float32), 0.25, SQUARED, mode)
        assert w_sgd[0] != w[0]
        if m <= 12:   # 0.75^m = 3^m / 4^m fits in binary32 exactly
            assert w_sgd[0] == np.float32(1.0 - 0.75 ** m)


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_logistic_batch_first_touch(mode):
    # w0 = 0: every example of the first batch has z = 0 and sigma = 1/2, so
    # w_f = -sum_i lr (1/2 - t_i) x_if, exact with dyadic values
    row_ptr = np.array([0, 2, 4, 5], np.int64)
    col = np.array([0, 1, 1, 2, 0], np.int32)
    val = np.array([1.0, 2.0, 4.0, -0.5, 8.0], np.float32)
    y = np.array([1.0, -1.0, -1.0], np.float32)
    w = oracle.batch_epoch(row_ptr, col, val, y, np.zeros(3, np.float32), 0.5, LOGISTIC, mode, 3)
    # s = 0.5 * (0.5 - t): example 0 -> -0.25, examples 1, 2 -> +0.25
    assert w.tolist() == [0.25 - 2.0, 0.5 - 1.0, 0.125]


def fd_grad(f, x, h=1e-6):
    g = np.zeros_like(x)
    for i in range(len(x)):
        e = np.zeros_like(x)
        e[i] = h
        g[i] = (f(x + e) - f(x - e)) / (2 * h)
    return g


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_batch_step_against_fp64_gradient(seed, mode):
    rng = np.random.default_rng(seed)
    n, d = 5, 40
    row_ptr, col = random_csr(rng, n, d, 20)
    val = rng.normal(size=len(col)).astype(np.float32)
    w0 = (0.3 * rng.normal(size=d)).astype(np.float32)
    lr = np.float32(0.02)
    for loss in (LOGISTIC, SQUARED):
        y = (np.where(rng.random(n) < 0.5, -1.0, 1.0) if loss == LOGISTIC
             else rng.normal(size=n)).astype(np.float32)
        w1 = oracle.batch_epoch(row_ptr, col, val, y, w0, lr, loss, mode, n)
        X = np.zeros((n, d))
        for i in range(n):
            X[i, col[row_ptr[i]:row_ptr[i + 1]]] = val[row_ptr[i]:row_ptr[i + 1]]
        yd = y.astype(np.float64)
        if loss == LOGISTIC:
            f = lambda v: sum(math.log1p(math.exp(-yd[i] * float(X[i] @ v))) for i in range(n))
        else:
            f = lambda v: sum(0.5 * (float(X[i] @ v) - yd[i]) ** 2 for i in range(n))
        ref = w0.astype(np.float64) - float(lr) * fd_grad(f, w0.astype(np.float64))
        assert np.max(np.abs(w1 - ref)) < 2e-6


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("B", [3, 100])
def test_theorem2_over_batches(cfg, B):
    g = datagen.generate(cfg, n=4000, d=4000 if cfg == 4 else 600, seed=21)
    w0 = np.zeros(g["d"], np.float32)
    args = (g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], MATCHED, B)
    seq = oracle.batch_epoch(*args)
    level, perm, level_ptr, L = oracle.batch_schedule(g["row_ptr"], g["col"], g["d"], B)
    rev = np.concatenate([perm[level_ptr[l]:level_ptr[l + 1]][::-1] for l in range(L)])
    got = oracle.batch_epoch(*args, order=rev)
    assert np.array_equal(got.view(np.int32), seq.view(np.int32))
    # a batch of level 2 moved in front of the batch of level 1 it conflicts with
    if L >= 2:
        b = perm[level_ptr[1]]
        order = np.concatenate([[b], perm[perm != b]]).astype(np.int32)
        assert not np.array_equal(oracle.batch_epoch(*args, order=order), seq)


def test_ragged_last_batch_and_empty_rows():
    row_ptr = np.array([0, 1, 1, 2, 2, 3], np.int64)       # rows 1 and 3 empty
    col = np.array([0, 0, 1], np.int32)
    val = np.array([1.0, 1.0, 1.0], np.float32)
    y = np.array([1.0, 1.0, 1.0, 1.0, 1.0], np.float32)
    # B = 2: batches {0,1}, {2,3}, {4}; least squares lr = 1/2
    w = oracle.batch_epoch(row_ptr, col, val, y, np.zeros(2, np.float32), 0.5, SQUARED, MATCHED, 2)
    assert w.tolist() == [0.75, 0.5]
    lv, L = oracle.batch_levels_seq(row_ptr, col, 2, 2)
    assert lv.tolist() == [1, 2, 1] and L == 2
