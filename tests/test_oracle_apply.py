"""Pins for the oracle's sequential SGD and its exponential.

  * exp against the correctly rounded fp64 library exp, within 2 ulp;
  * closed forms with dyadic inputs that are exact in binary32
    (least squares: w_k = 1 - 2^-k; logistic first touch: z = 0 gives
    sigma = 1/2 exactly; matrix completion with simultaneous updates);
  * the update direction and scale against an fp64 central-difference
    gradient of each loss (the gradient step of Sec. 2), within fp32 error;
  * Theorem 2 as a property: any order that runs levels in increasing order,
    with any order inside a level, gives bitwise the sequential result; and a
    negative case that breaks a per-feature order and changes it.
"""
import math

import numpy as np
import pytest

import datagen
import oracle
from oracle import LOGISTIC, MATCHED, NATURAL, SQUARED


def ulp_distance(a, b):
    ia = np.float32(a).view(np.int32).astype(np.int64)
    ib = np.float32(b).view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, np.int64(-(2 ** 31)) - ia, ia)
    ib = np.where(ib < 0, np.int64(-(2 ** 31)) - ib, ib)
    return abs(int(ia) - int(ib))


def test_exp_against_library_exp():
    xs = np.concatenate([np.linspace(-103.9, 88.7, 60001), np.linspace(-1, 1, 20001),
                         np.float32([0.34657359, -0.34657359, 1e-8, -1e-8])]).astype(np.float32)
    worst = 0
    for x in xs:
        ref = np.float32(math.exp(float(x)))
        got = oracle.exp(float(x))
        if ref < np.float32(1.1754944e-38):     # subnormal results: absolute bound
            assert abs(float(got) - float(ref)) <= 2 * 1.4e-45
            continue
        worst = max(worst, ulp_distance(got, ref))
    assert worst <= 2


def test_exp_special_values():
    assert oracle.exp(0.0) == np.float32(1.0)
    assert oracle.exp(-0.0) == np.float32(1.0)
    assert np.isnan(oracle.exp(float("nan")))
    assert oracle.exp(float("inf")) == np.inf and oracle.exp(float("-inf")) == 0.0
    assert oracle.exp(89.0) == np.inf and oracle.exp(-104.0) == 0.0
    assert oracle.exp(88.72283172607421875) < np.inf       # largest finite result
    assert oracle.exp(88.72283935546875) == np.inf
    assert oracle.exp(-103.0) > 0.0                          # subnormal, not flushed


def test_sigmoid_against_fp64_logistic():
    # matched-mode logistic: within 4 ulp of the fp64 value 1/(1+e^-z) (exp
    # within 2 ulp, then one rounding for 1 + e and one for the division)
    # wherever -z <= 87; the cap keeps the value at 1/(1 + e^87) below
    zs = np.concatenate([np.linspace(-87.0, 104.0, 40001), np.linspace(-2, 2, 4001)]).astype(np.float32)
    for z in zs:
        ref = np.float32(1.0 / (1.0 + math.exp(-float(z))))
        assert ulp_distance(oracle.sigmoid(float(z)), ref) <= 4, z
    floor = oracle.sigmoid(-87.0)
    assert floor == np.float32(1.0) / (np.float32(1.0) + oracle.exp(87.0))
    assert np.float32(1.1754944e-38) < floor < np.float32(1.7e-38)  # normal, tiny
    for z in (-87.5, -100.0, -1e30, -np.inf):
        assert oracle.sigmoid(z) == floor
    assert oracle.sigmoid(np.inf) == np.float32(1.0) and oracle.sigmoid(200.0) == np.float32(1.0)
    assert oracle.sigmoid(0.0) == np.float32(0.5)
    assert np.isnan(oracle.sigmoid(float("nan")))


def test_sigmoid_monotone():
    zs = np.linspace(-90.0, 20.0, 200001).astype(np.float32)
    v = np.array([oracle.sigmoid(float(z)) for z in zs], dtype=np.float32)
    assert np.all(np.diff(v) >= 0)


def one_feature_rows(k):
    return np.arange(k + 1, dtype=np.int64), np.zeros(k, dtype=np.int32)


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_least_squares_dyadic_closed_form(mode):
    # x = 1, y = 1, lr = 1/2 on one feature: w <- (w + 1)/2, so w_k = 1 - 2^-k
    for k in range(1, 25):
        row_ptr, col = one_feature_rows(k)
        w = oracle.sgd_epoch(row_ptr, col, np.ones(k, np.float32), np.ones(k, np.float32),
                             np.zeros(1, np.float32), 0.5, SQUARED, mode)
        assert w[0] == np.float32(1.0 - 2.0 ** -k)


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_logistic_first_touch_closed_form(mode):
    # w0 = 0 -> z = 0 -> sigma = 1/2 exactly; w_f = lr (t - 1/2) x_f with t = [y > 0]
    row_ptr = np.array([0, 2, 4], np.int64)
    col = np.array([0, 1, 2, 3], np.int32)
    val = np.array([1.0, 2.0, 4.0, -0.5], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    w = oracle.sgd_epoch(row_ptr, col, val, y, np.zeros(4, np.float32), 0.5, LOGISTIC, mode)
    assert w.tolist() == [0.25, 0.5, -1.0, 0.125]


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_mf_dyadic_simultaneous_update(mode):
    U = np.zeros((1, 32), np.float32); U[0, 0] = 1.0
    V = np.zeros((1, 32), np.float32); V[0, 0] = 1.0
    # <U,V> = 1, e = 3 - 1 = 2; U0 <- 1 + 1/2 (2*1 - 1/2*1) = 1.75, V0 uses the old U0
    U1, V1 = oracle.mf_epoch([0], [0], [3.0], U, V, 0.5, 0.5, mode)
    assert U1[0, 0] == 1.75 and V1[0, 0] == 1.75
    assert np.all(U1[0, 1:] == 0) and np.all(V1[0, 1:] == 0)
    U1, V1 = oracle.mf_epoch([0], [0], [3.0], U, V, 0.5, 0.0, mode)
    assert U1[0, 0] == 2.0 and V1[0, 0] == 2.0


def fd_grad(f, x, h=1e-6):
    g = np.zeros_like(x)
    for i in range(len(x)):
        e = np.zeros_like(x); e[i] = h
        g[i] = (f(x + e) - f(x - e)) / (2 * h)
    return g


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_single_step_against_fp64_gradient(seed, mode):
    rng = np.random.default_rng(seed)
    m, d = 70, 90
    cols = np.sort(rng.choice(d, m, replace=False)).astype(np.int32)
    x = rng.normal(size=m).astype(np.float32)
    w0 = (0.3 * rng.normal(size=d)).astype(np.float32)
    row_ptr = np.array([0, m], np.int64)
    lr = np.float32(0.05)
    for loss, yv in ((LOGISTIC, 1.0), (LOGISTIC, -1.0), (SQUARED, 0.7)):
        y = np.array([yv], np.float32)
        w1 = oracle.sgd_epoch(row_ptr, cols, x, y, w0, lr, loss, mode)
        xs, wd = x.astype(np.float64), w0.astype(np.float64)[cols]
        if loss == LOGISTIC:
            f = lambda v: math.log1p(math.exp(-yv * float(np.dot(v, xs))))
        else:
            f = lambda v: 0.5 * (float(np.dot(v, xs)) - yv) ** 2
        ref = wd - float(lr) * fd_grad(f, wd)
        assert np.max(np.abs(w1[cols] - ref)) < 2e-6
        untouched = np.setdiff1d(np.arange(d), cols)
        assert np.array_equal(w1[untouched], w0[untouched])


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
def test_mf_step_against_fp64_gradient(mode):
    rng = np.random.default_rng(5)
    U = (rng.normal(size=(3, 32)) / np.sqrt(32)).astype(np.float32)
    V = (rng.normal(size=(2, 32)) / np.sqrt(32)).astype(np.float32)
    lr, reg, r = np.float32(0.05), np.float32(0.02), 0.8
    U1, V1 = oracle.mf_epoch([2], [1], [r], U, V, lr, reg, mode)
    u, v = U[2].astype(np.float64), V[1].astype(np.float64)
    f = lambda z: 0.5 * (r - np.dot(z[:32], z[32:])) ** 2 + 0.5 * float(reg) * np.dot(z, z)
    ref = np.concatenate([u, v]) - float(lr) * fd_grad(f, np.concatenate([u, v]))
    assert np.max(np.abs(np.concatenate([U1[2], V1[1]]) - ref)) < 1e-6
    assert np.array_equal(U1[:2], U[:2]) and np.array_equal(V1[0], V[0])


def small_problem(seed, cfg=1, n=3000, d=300):
    return datagen.generate(cfg, n=n, d=d, seed=seed)


@pytest.mark.parametrize("mode", [NATURAL, MATCHED])
@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_theorem2_level_order_is_bitwise_sequential(cfg, mode):
    g = small_problem(77, cfg=cfg, n=4000, d=2000 if cfg == 4 else 400)
    w0 = np.zeros(g["d"], np.float32)
    seq = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], mode)
    level, perm, level_ptr, L = oracle.schedule(g["row_ptr"], g["col"], g["d"])
    rng = np.random.default_rng(1)
    orders = [perm]
    rev = np.concatenate([perm[level_ptr[l]:level_ptr[l + 1]][::-1] for l in range(L)])
    shuf = np.concatenate([rng.permutation(perm[level_ptr[l]:level_ptr[l + 1]]) for l in range(L)])
    orders += [rev, shuf]
    for order in orders:
        got = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"],
                               mode, order=order)
        assert np.array_equal(got.view(np.int32), seq.view(np.int32))


def test_breaking_a_feature_order_changes_the_result():
    g = small_problem(78)
    w0 = np.zeros(g["d"], np.float32)
    seq = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"])
    level, perm, level_ptr, L = oracle.schedule(g["row_ptr"], g["col"], g["d"])
    # move the first example of level 2 in front of level 1: it then runs
    # before the earlier example it conflicts with
    i = perm[level_ptr[1]]
    order = np.concatenate([[i], perm[perm != i]]).astype(np.int32)
    got = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"],
                           order=order)
    assert not np.array_equal(got, seq)


@pytest.mark.parametrize("seed", range(3))
def test_mf_theorem2_level_order(seed):
    g = datagen.generate_mf(5, n=20000, n_users=3000, n_items=600, seed=seed)
    seq = oracle.mf_epoch(g["user"], g["item"], g["rating"], g["U0"], g["V0"], g["lr"], g["reg"])
    level, perm, level_ptr, L = oracle.schedule(g["row_ptr"], g["col"], g["d"])
    rev = np.concatenate([perm[level_ptr[l]:level_ptr[l + 1]][::-1] for l in range(L)])
    got = oracle.mf_epoch(g["user"], g["item"], g["rating"], g["U0"], g["V0"], g["lr"], g["reg"],
                          order=rev)
    assert np.array_equal(got[0], seq[0]) and np.array_equal(got[1], seq[1])


def test_empty_examples_leave_weights_unchanged():
    row_ptr = np.array([0, 0, 1, 1], np.int64)
    col = np.array([1], np.int32)
    w = oracle.sgd_epoch(row_ptr, col, np.array([2.0], np.float32),
                         np.array([1.0, 1.0, -1.0], np.float32), np.zeros(3, np.float32), 0.5)
    assert w.tolist() == [0.0, 0.5, 0.0]


def test_natural_and_matched_orders_agree_closely():
    g = datagen.generate(1)
    w0 = np.zeros(g["d"], np.float32)
    a = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], NATURAL)
    b = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"], MATCHED)
    assert np.max(np.abs(a - b)) < 1e-4


ADVERSARIAL_LANES = {"pairs_1_before_32": (0, 1, 32, 33), "pairs_16_before_32": (0, 16, 32, 48)}


def adversarial_order_row(lanes=(0, 1, 32, 33)):
    """64 entries with w = 1: x_a = 2^24, x_b = 1, x_c = -2^24, x_d = 1 for
    lanes (a, b, c, d), the rest 0, plus entry 64 (partial 0) on a feature
    with w = 0 and x = 1 that reads out the step.  With (0, 1, 32, 33),
    pairing partials l, l^1 first (ascending offsets) rounds 2^24 + 1 to 2^24
    and gives z = 1, while pairing l, l^32 first gives the exact sum 2.  With
    (0, 16, 32, 48), pairing rows 0-1 and 2-3 of 16 lanes before the halves
    gives 1, pairing 0-2 and 1-3 first gives 2."""
    a, b, c, d = lanes
    x = np.zeros(65, np.float32)
    x[a], x[b], x[c], x[d], x[64] = 2.0 ** 24, 1.0, -(2.0 ** 24), 1.0, 1.0
    w0 = np.ones(65, np.float32)
    w0[64] = 0.0
    return np.array([0, 65], np.int64), np.arange(65, dtype=np.int32), x, w0


@pytest.mark.parametrize("name", sorted(ADVERSARIAL_LANES))
def test_matched_order_is_ascending_butterfly(name):
    row_ptr, col, x, w0 = adversarial_order_row(ADVERSARIAL_LANES[name])
    y = np.zeros(1, np.float32)
    # least squares, lr = 1, y = 0: s = z, and the read-out feature ends at -z
    wm = oracle.sgd_epoch(row_ptr, col, x, y, w0, 1.0, SQUARED, MATCHED)
    wn = oracle.sgd_epoch(row_ptr, col, x, y, w0, 1.0, SQUARED, NATURAL)
    assert wm[64] == -1.0
    # natural order accumulates in CSR order: 2^24, 2^24 (the +1 is lost), 0
    # after -2^24, then 1
    assert wn[64] == -1.0
