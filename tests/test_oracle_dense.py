"""Pins of the oracle's dense full-batch gradient descent (Sec. 2's update
with every example in every iteration, the dense workloads of Sec. 6.1-6.2)
against what the mathematics fixes: exact rational arithmetic on small
integer data, the closed form of gradient descent on least squares, its limit
(the least-squares solution), the logistic step from its definition in
binary64, the mini-batch oracle with one batch of all examples, and the
degenerate cases."""
from fractions import Fraction

import numpy as np
import pytest

import oracle

BLOCKINGS = [(None, None, None), (1, 4, None), (2, 8, None), (3, 1, 1), (5, 64, 2), (1000, 3, None),
             (1000, 3, 32), (11, 8, 4)]


def exact_gd(X, y, w, lr, iters):
    """Least-squares gradient descent in rational arithmetic."""
    n, d = X.shape
    W = [Fraction(float(v)) for v in w]
    L = Fraction(float(lr))
    for _ in range(iters):
        s = []
        for i in range(n):
            z = sum((Fraction(float(X[i, j])) * W[j] for j in range(d)), Fraction(0))
            s.append(L * (z - Fraction(float(y[i]))))
        G = [sum((s[i] * Fraction(float(X[i, j])) for i in range(n)), Fraction(0)) for j in range(d)]
        W = [W[j] - G[j] for j in range(d)]
    return W


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("iters", [1, 2])
def test_exact_integer_iterations(seed, iters):
    # small integers and a power-of-two step: every intermediate of every
    # summation order is exact in binary32, so all orders equal the rationals
    rng = np.random.default_rng(seed)
    n, d = 7 + seed, 9 + 2 * seed
    X = rng.integers(-2, 3, size=(n, d)).astype(np.float32)
    y = rng.integers(-4, 5, size=n).astype(np.float32)
    w = rng.integers(-2, 3, size=d).astype(np.float32)
    lr = np.float32(2.0 ** -7)
    want = exact_gd(X, y, w, lr, iters)
    assert all(Fraction(float(np.float32(float(v)))) == v for v in want), "premise: exact in binary32"
    want = np.array([float(v) for v in want], np.float32)
    got = oracle.dense_gd(X, y, w, lr, oracle.SQUARED, oracle.NATURAL, iters)
    assert np.array_equal(got, want)
    for rb, cb, rc in BLOCKINGS:
        got = oracle.dense_gd(X, y, w, lr, oracle.SQUARED, oracle.MATCHED, iters, rb, cb, rc)
        assert np.array_equal(got, want), (rb, cb, rc)


def closed_form_lsq(X, y, w0, lr, T):
    """w_T for w <- w - lr X^T (X w - y) in binary64 by the eigenvectors of
    X^T X: along eigenvalue lam the error to the fixed point shrinks by
    (1 - lr lam) per step; along lam = 0 the component stays."""
    X = X.astype(np.float64)
    A = X.T @ X
    b = X.T @ y.astype(np.float64)
    lam, V = np.linalg.eigh(A)
    u0, bt = V.T @ w0.astype(np.float64), V.T @ b
    q = 1.0 - lr * lam
    uT = np.empty_like(u0)
    for k in range(len(lam)):
        if abs(lam[k]) > 1e-9 * max(lam.max(), 1.0):
            uT[k] = q[k] ** T * u0[k] + (1.0 - q[k] ** T) * bt[k] / lam[k]
        else:
            uT[k] = u0[k] + T * lr * bt[k]
    return V @ uT


@pytest.mark.parametrize("n,d", [(40, 12), (12, 40), (64, 64)])
@pytest.mark.parametrize("mode", [oracle.NATURAL, oracle.MATCHED])
def test_closed_form_least_squares(n, d, mode):
    rng = np.random.default_rng(n * 100 + d)
    X = rng.normal(size=(n, d)).astype(np.float32)
    y = rng.normal(size=n).astype(np.float32)
    w0 = rng.normal(size=d).astype(np.float32)
    lam_max = np.linalg.eigvalsh(X.astype(np.float64).T @ X).max()
    lr = np.float32(0.9 / lam_max)
    T = 30
    want = closed_form_lsq(X, y, w0, float(lr), T)
    got = oracle.dense_gd(X, y, w0, lr, oracle.SQUARED, mode, T, 7, 8)
    assert np.max(np.abs(got - want)) <= 2e-5 * max(1.0, np.abs(want).max())


def test_limit_is_least_squares_solution():
    rng = np.random.default_rng(5)
    n, d = 200, 16
    X = rng.normal(size=(n, d)).astype(np.float32)
    y = (X.astype(np.float64) @ rng.normal(size=d) + 0.1 * rng.normal(size=n)).astype(np.float32)
    ev = np.linalg.eigvalsh(X.astype(np.float64).T @ X)
    lr = np.float32(1.0 / ev.max())
    T = int(np.ceil(np.log(1e-9) / np.log(1.0 - ev.min() / ev.max())))
    sol = np.linalg.lstsq(X.astype(np.float64), y.astype(np.float64), rcond=None)[0]
    for mode in (oracle.NATURAL, oracle.MATCHED):
        got = oracle.dense_gd(X, y, np.zeros(d), lr, oracle.SQUARED, mode, T, 32, 4)
        assert np.max(np.abs(got - sol)) <= 1e-5 * max(1.0, np.abs(sol).max())


@pytest.mark.parametrize("mode", [oracle.NATURAL, oracle.MATCHED])
def test_logistic_step_from_definition(mode):
    import math

    rng = np.random.default_rng(11)
    n, d = 50, 30
    X = rng.normal(size=(n, d)).astype(np.float32)
    y = np.where(rng.random(n) < 0.5, -1.0, 1.0).astype(np.float32)
    w0 = (0.3 * rng.normal(size=d)).astype(np.float32)
    lr = np.float32(0.01)
    Xd, w = X.astype(np.float64), w0.astype(np.float64)
    z = Xd @ w
    g = np.array([1.0 / (1.0 + math.exp(-v)) for v in z]) - (y > 0)
    want = w - float(lr) * (Xd.T @ g)
    got = oracle.dense_gd(X, y, w0, lr, oracle.LOGISTIC, mode, 1, 9, 12)
    assert np.max(np.abs(got - want)) <= 1e-6 * max(1.0, np.abs(want).max())


def test_logistic_loss_decreases():
    rng = np.random.default_rng(12)
    n, d = 300, 20
    X = rng.normal(size=(n, d)).astype(np.float32)
    y = np.where(X[:, 0] + 0.5 * rng.normal(size=n) > 0, 1.0, -1.0).astype(np.float32)

    def loss(w):
        m = (2.0 * (y > 0) - 1.0) * (X.astype(np.float64) @ w.astype(np.float64))
        return np.sum(np.logaddexp(0.0, -m))

    w = np.zeros(d, np.float32)
    prev = loss(w)
    for _ in range(15):
        w = oracle.dense_gd(X, y, w, np.float32(0.002), oracle.LOGISTIC, oracle.MATCHED, 1, 64, 8)
        cur = loss(w)
        assert cur < prev
        prev = cur


@pytest.mark.parametrize("loss", [oracle.LOGISTIC, oracle.SQUARED])
def test_blockings_agree_with_natural(loss):
    rng = np.random.default_rng(13)
    n, d = 37, 301
    X = rng.normal(size=(n, d)).astype(np.float32)
    y = (np.where(rng.random(n) < 0.5, -1.0, 1.0) if loss == oracle.LOGISTIC
         else rng.normal(size=n)).astype(np.float32)
    lr = np.float32(0.5 / (n + d))
    nat = oracle.dense_gd(X, y, np.zeros(d), lr, loss, oracle.NATURAL, 5)
    for rb, cb, rc in BLOCKINGS + [(37, 512, None), (36, 300, 32), (37, 300, 5)]:
        got = oracle.dense_gd(X, y, np.zeros(d), lr, loss, oracle.MATCHED, 5, rb, cb, rc)
        assert np.max(np.abs(got - nat)) <= 1e-6, (rb, cb, rc)


def test_equals_one_batch_of_all_examples():
    # the mini-batch oracle with B = n is the same step; it accumulates the
    # updates into w one example at a time, so the two agree up to rounding
    rng = np.random.default_rng(14)
    n, d = 60, 25
    X = rng.normal(size=(n, d)).astype(np.float32)
    y = rng.normal(size=n).astype(np.float32)
    w0 = rng.normal(size=d).astype(np.float32)
    row_ptr = np.arange(0, n * d + 1, d, dtype=np.int64)
    col = np.tile(np.arange(d, dtype=np.int32), n)
    lr = np.float32(0.002)
    b = oracle.batch_epoch(row_ptr, col, X.ravel(), y, w0, lr, oracle.SQUARED, oracle.NATURAL, B=n)
    g = oracle.dense_gd(X, y, w0, lr, oracle.SQUARED, oracle.NATURAL, 1)
    assert np.max(np.abs(b - g)) <= 1e-5
    assert not np.array_equal(b, w0)


def test_strided_rows():
    rng = np.random.default_rng(15)
    big = rng.normal(size=(20, 33)).astype(np.float32)
    X = big[:, :30]  # row stride 33
    y = rng.normal(size=20).astype(np.float32)
    a = oracle.dense_gd(X, y, np.zeros(30), np.float32(0.01), oracle.SQUARED, oracle.MATCHED, 3, 4, 8)
    b = oracle.dense_gd(np.ascontiguousarray(X), y, np.zeros(30), np.float32(0.01), oracle.SQUARED,
                        oracle.MATCHED, 3, 4, 8)
    assert np.array_equal(a, b)


def test_degenerate_cases():
    rng = np.random.default_rng(16)
    X = rng.normal(size=(5, 4)).astype(np.float32)
    y = rng.normal(size=5).astype(np.float32)
    w0 = rng.normal(size=4).astype(np.float32)
    for mode in (oracle.NATURAL, oracle.MATCHED):
        # no iterations, no examples: w unchanged
        assert np.array_equal(oracle.dense_gd(X, y, w0, 0.1, oracle.SQUARED, mode, 0), w0)
        assert np.array_equal(oracle.dense_gd(np.zeros((0, 4), np.float32), np.zeros(0), w0, 0.1,
                                              oracle.SQUARED, mode, 3), w0)
        # zero rows contribute nothing; zero step leaves w
        Xz = np.vstack([X, np.zeros((3, 4), np.float32)])
        yz = np.concatenate([y, np.zeros(3, np.float32)])
        assert np.array_equal(oracle.dense_gd(Xz, yz, w0, 0.01, oracle.SQUARED, mode, 2, 3, 4),
                              oracle.dense_gd(X, y, w0, 0.01, oracle.SQUARED, mode, 2, 3, 4))
        assert np.array_equal(oracle.dense_gd(X, y, w0, 0.0, oracle.SQUARED, mode, 2), w0)
    with pytest.raises(ValueError):
        oracle.dense_gd(X, y, w0, 0.1, oracle.SQUARED, oracle.MATCHED, 1, 0, 4)
    with pytest.raises(ValueError):
        oracle.dense_gd(X, y, w0, 0.1, oracle.SQUARED, oracle.MATCHED, 1, 2, 4, 0)


def test_row_chunks_split_the_gradient_chain():
    # a chunk as long as the row block is the single chain; shorter chunks
    # regroup the same sum (equal here up to rounding, and bitwise when the
    # data make every partial exact)
    rng = np.random.default_rng(17)
    X = rng.normal(size=(64, 10)).astype(np.float32)
    y = rng.normal(size=64).astype(np.float32)
    w0 = rng.normal(size=10).astype(np.float32)
    a = oracle.dense_gd(X, y, w0, 0.01, oracle.SQUARED, oracle.MATCHED, 2, 64, 12)
    b = oracle.dense_gd(X, y, w0, 0.01, oracle.SQUARED, oracle.MATCHED, 2, 64, 12, 64)
    c = oracle.dense_gd(X, y, w0, 0.01, oracle.SQUARED, oracle.MATCHED, 2, 64, 12, 7)
    assert np.array_equal(a, b)
    assert np.max(np.abs(a - c)) <= 1e-5 and not np.array_equal(a, c)
