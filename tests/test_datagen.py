"""Synthetic input generator: determinism and distributions (CPU)."""
import numpy as np
import pytest
from scipy import stats

import datagen


def test_philox_known_answers():
    # Known-answer vectors published with the Random123 library (Salmon et al., SC'11)
    assert [hex(x) for x in datagen.philox_block([0, 0, 0, 0], [0, 0])] == \
        ["0x6627e8d5", "0xe169c58d", "0xbc57ac4c", "0x9b00dbd8"]
    assert [hex(x) for x in datagen.philox_block([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2)] == \
        ["0x408f276d", "0x41c83b0e", "0xa20bc7c6", "0x6d5451fd"]
    assert [hex(x) for x in datagen.philox_block(
        [0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0])] == \
        ["0xd16cfe09", "0x94fdcceb", "0x5001e420", "0x24126ea1"]


def _same(a, b):
    for k in ("row_ptr", "col", "val", "y"):
        if a[k] is None or b[k] is None:
            assert a[k] is None and b[k] is None
        else:
            assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_deterministic_any_thread_count(cfg):
    n = 5000 if cfg != 1 else None
    a = datagen.generate(cfg, n=n, nthreads=1)
    b = datagen.generate(cfg, n=n, nthreads=7)
    _same(a, b)
    c = datagen.generate(cfg, n=n, seed=a["seed"] + 1)
    assert not np.array_equal(a["col"], c["col"])


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_rows_sorted_unique_in_range(cfg):
    g = datagen.generate(cfg, n=20000)
    rp, col, d = g["row_ptr"], g["col"], g["d"]
    assert rp[0] == 0 and np.all(np.diff(rp) >= 0)
    assert col.min() >= 0 and col.max() < d
    rows = np.repeat(np.arange(g["n"]), np.diff(rp))
    same_row = rows[1:] == rows[:-1]
    assert np.all(col[1:][same_row] > col[:-1][same_row])


def test_nnz_per_row_distributions():
    m1 = np.diff(datagen.generate(1)["row_ptr"])
    assert np.all(m1 == 10)
    m2 = np.diff(datagen.generate(2, n=50000)["row_ptr"])
    assert m2.min() == 20 and m2.max() == 40
    counts = np.bincount(m2 - 20, minlength=21)
    assert stats.chisquare(counts).pvalue > 1e-4
    assert np.all(np.diff(datagen.generate(3, n=2000)["row_ptr"]) == 50)
    m4 = np.diff(datagen.generate(4, n=50000)["row_ptr"])
    assert m4.min() >= 1 and m4.max() <= 400
    assert abs(m4.mean() - 80) < 0.3 and abs(m4.var() - 80) < 4


def test_poisson_ptrs_matches_pmf():
    x = datagen.poisson_sample(7, 80.0, 200000)
    lo, hi = 55, 106
    obs = np.array([np.sum(x < lo)] + [np.sum(x == k) for k in range(lo, hi)] + [np.sum(x >= hi)])
    pmf = stats.poisson(80.0)
    exp = np.array([pmf.cdf(lo - 1)] + [pmf.pmf(k) for k in range(lo, hi)] + [pmf.sf(hi - 1)])
    exp = exp / exp.sum() * len(x)
    assert stats.chisquare(obs, exp).pvalue > 1e-4


def test_uniform_open_interval():
    u = datagen.uniform_sample(3, 400000)
    assert u.min() > 0.0 and u.max() < 1.0
    assert stats.kstest(u, "uniform").pvalue > 1e-4


@pytest.mark.parametrize("alpha,d", [(1.0, 1000), (1.2, 1_000_000), (1.1, 100_000)])
def test_zipf_head_frequencies(alpha, d):
    x = datagen.zipf_sample(11, d, alpha, 400000)
    H = np.sum(np.arange(1, d + 1, dtype=np.float64) ** -alpha)
    for k in range(1, 6):
        p = k ** -alpha / H
        f = np.mean(x == k - 1)
        assert abs(f - p) < 5 * np.sqrt(p * (1 - p) / len(x)), (k, f, p)


def test_labels_planted_sign_with_flips():
    g = datagen.generate(1)
    wstar = np.empty(g["d"], dtype=np.float64)
    datagen._load().gen_wstar(g["seed"], g["d"], wstar.ctypes.data, 1)
    rows = np.repeat(np.arange(g["n"]), np.diff(g["row_ptr"]))
    dot = np.bincount(rows, weights=g["val"].astype(np.float64) * wstar[g["col"]], minlength=g["n"])
    clean = np.where(dot >= 0, 1.0, -1.0)
    assert set(np.unique(g["y"]).tolist()) == {-1.0, 1.0}
    flip = np.mean(clean != g["y"])
    assert abs(flip - 0.05) < 0.01


def test_least_squares_targets():
    g = datagen.generate(4, n=20000)
    wstar = np.empty(g["d"], dtype=np.float64)
    datagen._load().gen_wstar(g["seed"], g["d"], wstar.ctypes.data, 4)
    rows = np.repeat(np.arange(g["n"]), np.diff(g["row_ptr"]))
    dot = np.bincount(rows, weights=g["val"].astype(np.float64) * wstar[g["col"]], minlength=g["n"])
    resid = g["y"] - dot
    assert abs(resid.std() - 0.1) < 0.01 and abs(resid.mean()) < 0.01


def test_matrix_completion_shapes_and_scale():
    g = datagen.generate_mf(5, n=200000, n_users=20000, n_items=4000)
    assert g["user"].min() >= 0 and g["user"].max() < 20000
    assert g["item"].min() >= 0 and g["item"].max() < 4000
    assert g["U0"].shape == (20000, 32) and g["V0"].shape == (4000, 32)
    assert abs(g["U0"].std() - 1 / np.sqrt(32)) < 0.005
    # rating = <u*, v*> + N(0, 0.5): variance 32 * (1/32)^2 + 0.25
    assert abs(g["rating"].var() - (1 / 32 + 0.25)) < 0.02
    assert np.array_equal(g["col"][0::2], g["user"])
    assert np.array_equal(g["col"][1::2], g["item"] + 20000)


def test_dense_examples():
    a = datagen.generate_dense(1, n=300, d=200, nthreads=1)
    b = datagen.generate_dense(1, n=300, d=200, nthreads=7, ldx=203)
    assert a["X"].shape == (300, 200) and b["X"].strides == (203 * 4, 4)
    assert np.array_equal(a["X"], b["X"]) and np.array_equal(a["y"], b["y"])
    assert abs(a["X"].mean()) < 0.02 and abs(a["X"].std() - 1.0) < 0.02
    # least squares: y = <x, w*> / sqrt(d) + 0.1 N(0,1), so var(y) ~ |w*|^2 / d + 0.01
    assert 0.7 < a["y"].var() < 1.3
    c = datagen.generate_dense(1, n=300, d=200, loss=datagen.LOGISTIC)
    assert set(np.unique(c["y"])) <= {-1.0, 1.0}
    full = datagen.DENSE[1]
    assert (full.n, full.d) == (5000, 960)
