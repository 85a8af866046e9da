"""Pins for the oracle's bounded-delay SGD (Sec. 7), in the execution that
reads as early as the Asynchronous Read Constraint allows: example alpha
reads the weights after examples 0 .. alpha - delay - 1, and updates are
applied in example order per feature.

  * delay 0 is the sequential SGD oracle, bit for bit;
  * a delay of n - 1 or more reads the initial weights everywhere: one
    mini-batch of all n examples, bit for bit;
  * the per-entry form equals the literal form built from whole weight
    snapshots after every example;
  * a one-feature least-squares recurrence against exact rational
    arithmetic (every value is dyadic, so binary32 holds it exactly);
  * the constraint itself: each read sees exactly the writes of the
    examples before alpha - delay (checked by replaying the snapshots).
"""
from fractions import Fraction

import numpy as np
import pytest

import datagen
import oracle
from oracle import LOGISTIC, MATCHED, NATURAL, SQUARED


def random_csr(rng, n, d, max_m):
    rows = [sorted(rng.choice(d, rng.integers(0, min(max_m, d) + 1), replace=False))
            for _ in range(n)]
    row_ptr = np.zeros(n + 1, np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in r], np.int32)
    return row_ptr, col


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_delay_zero_is_sgd(cfg, mode):
    g = datagen.generate(cfg, n=3000, d=2000 if cfg == 4 else 300, seed=12)
    w0 = (0.1 * np.random.default_rng(1).normal(size=g["d"])).astype(np.float32)
    a = oracle.stale_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], mode, 0)
    b = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], mode)
    assert np.array_equal(a.view(np.int32), b.view(np.int32))


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_full_delay_is_one_batch(cfg, mode):
    g = datagen.generate(cfg, n=2000, d=2000 if cfg == 4 else 300, seed=13)
    n = g["n"]
    lr = np.float32(g["lr"] / 50)
    w0 = np.zeros(g["d"], np.float32)
    args = (g["row_ptr"], g["col"], g["val"], g["y"], w0, lr, g["loss"], mode)
    ref = oracle.batch_epoch(*args, n)
    for delay in (n - 1, n, 10 * n):
        got = oracle.stale_epoch(*args, delay)
        assert np.array_equal(got.view(np.int32), ref.view(np.int32))


@pytest.mark.parametrize("seed", range(12))
def test_per_entry_form_equals_snapshots(seed):
    rng = np.random.default_rng(200 + seed)
    n, d = int(rng.integers(1, 80)), int(rng.integers(1, 20))
    row_ptr, col = random_csr(rng, n, d, 6)
    val = rng.normal(size=len(col)).astype(np.float32)
    w0 = (0.2 * rng.normal(size=d)).astype(np.float32)
    for loss in (LOGISTIC, SQUARED):
        y = (np.where(rng.random(n) < 0.5, -1.0, 1.0) if loss == LOGISTIC
             else rng.normal(size=n)).astype(np.float32)
        for mode in (NATURAL, MATCHED):
            for delay in (0, 1, 2, 3, 7, n):
                a = oracle.stale_epoch(row_ptr, col, val, y, w0, 0.05, loss, mode, delay)
                b = oracle.stale_snapshot(row_ptr, col, val, y, w0, 0.05, loss, mode, delay)
                assert np.array_equal(a.view(np.int32), b.view(np.int32)), (loss, mode, delay)


@pytest.mark.parametrize("delay", [0, 1, 2, 5])
@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_one_feature_recurrence_exact(delay, mode):
    # least squares, x = 1, y = 1, lr = 1/4 on one feature:
    #   w_{a+1} = w_a - (w_{max(0, a - delay)} - 1) / 4
    # (continued while every value stays exact in binary32)
    def exact(v):
        return Fraction(float(np.float32(float(v)))) == v

    W = [Fraction(0)]
    while len(W) < 60:
        a = len(W) - 1
        nxt = W[a] - (W[max(0, a - delay)] - 1) / 4
        if not exact(nxt):
            break
        W.append(nxt)
    m = len(W) - 1
    assert m >= 8
    row_ptr, col = np.arange(m + 1, dtype=np.int64), np.zeros(m, np.int32)
    one = np.ones(m, np.float32)
    got = oracle.stale_epoch(row_ptr, col, one, one, np.zeros(1, np.float32), 0.25, SQUARED, mode,
                             delay)
    assert all(v.denominator & (v.denominator - 1) == 0 for v in W)   # dyadic
    assert got[0] == np.float32(float(W[m]))
    assert float(W[m]) == float(np.float32(float(W[m])))                # exact in binary32


def test_reads_see_exactly_the_writes_before_the_window():
    # replay: with delay 3, example a's read of a feature must equal that
    # feature's value in the snapshot after examples 0 .. a - 4
    rng = np.random.default_rng(7)
    n, d = 40, 4
    row_ptr, col = random_csr(rng, n, d, 3)
    val = np.ones(len(col), np.float32)
    y = np.ones(n, np.float32)
    delay = 3
    snaps = [np.zeros(d, np.float32)]
    for a in range(n):
        sub_rp = row_ptr[:a + 2]
        w = oracle.stale_epoch(sub_rp, col[:sub_rp[-1]], val[:sub_rp[-1]], y[:a + 1],
                               np.zeros(d, np.float32), 0.25, SQUARED, MATCHED, delay)
        snaps.append(w)
    # the weight change example a makes is -s_a x with s_a = 0.25 (z_a - 1),
    # z_a the sum over its features of the snapshot after a - delay examples
    for a in range(n):
        feats = col[row_ptr[a]:row_ptr[a + 1]]
        if len(feats) == 0:
            continue
        R = snaps[max(0, a - delay)]
        zs = [R[f] for f in feats]
        f0 = feats[0]
        # the first feature's new value is its value after a examples minus s_a
        got_step = snaps[a][f0] - snaps[a + 1][f0]
        exp_z = sum(float(v) for v in zs)
        assert abs(float(got_step) - 0.25 * (exp_z - 1.0)) < 1e-5
