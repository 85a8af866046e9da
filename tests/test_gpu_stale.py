"""GPU parity of bounded-delay SGD (pdb_stale_epoch, Sec. 7) against the CPU
oracle on the same seeded inputs: weights bitwise equal to the oracle's
matched order and within 1e-5 of its natural order, for delays from 0
(sequential SGD) to beyond n (every read at the initial weights)."""
import numpy as np
import pytest

import datagen
import oracle
from pdbtest import csr_from_rows, gpu_schedule, gpu_sgd
from test_gpu_parity import structured_cases

pytestmark = pytest.mark.gpu


def native_mod():
    from paper_1508_00703_amd import native
    return native


def gpu_stale(native, dev, g, lv, delay, w0=None, opt=None):
    import torch

    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], dev)
    y = torch.from_numpy(g["y"]).to(dev)
    w = torch.from_numpy(np.zeros(g["d"], np.float32) if w0 is None else w0.copy()).to(dev)
    ws = native.pdb_stale_epoch(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], delay, lv,
                                opt=opt)
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    return w.cpu().numpy()


def check_stale(native, dev, g, lv, delay, w0=None, tol=1e-5, opt=None):
    got = gpu_stale(native, dev, g, lv, delay, w0, opt=opt)
    w_init = np.zeros(g["d"], np.float32) if w0 is None else w0
    args = (g["row_ptr"], g["col"], g["val"], g["y"], w_init, g["lr"], g["loss"])
    ref_m = oracle.stale_epoch(*args, oracle.MATCHED, delay)
    bad = np.nonzero(got.view(np.int32) != ref_m.view(np.int32))[0]
    assert len(bad) == 0, "delay %d, first mismatches %s: gpu %s oracle %s" % (
        delay, bad[:5], got[bad[:5]], ref_m[bad[:5]])
    ref_n = oracle.stale_epoch(*args, oracle.NATURAL, delay)
    assert np.max(np.abs(got - ref_n), initial=0.0) <= tol
    return got


def structured_problem(rows, loss, with_val, seed):
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1 if len(col) else 1
    n = len(rows)
    rng = np.random.default_rng(seed)
    val = rng.normal(size=len(col)).astype(np.float32) if with_val else None
    y = (np.where(rng.random(n) < 0.5, -1.0, 1.0) if loss == oracle.LOGISTIC
         else rng.normal(size=n)).astype(np.float32)
    # a contractive step: stale reads need a smaller step than sequential ones
    sq = np.bincount(np.repeat(np.arange(n), np.diff(row_ptr)),
                     weights=(val.astype(np.float64) ** 2 if with_val else np.ones(len(col))),
                     minlength=n)
    lr = np.float32(min(0.01, 0.1 / max(sq.max(), 1.0)))
    return dict(row_ptr=row_ptr, col=col, val=val, y=y, n=n, d=d, lr=lr, loss=loss)


STALE_MODES = [2, 1]  # windowed where the windows fit, sync-free


@pytest.mark.parametrize("name", sorted(structured_cases()))
@pytest.mark.parametrize("loss", [0, 1])
@pytest.mark.parametrize("with_val", [True, False])
@pytest.mark.parametrize("delay", [0, 1, 3, 17, 1000])
@pytest.mark.parametrize("mode", STALE_MODES)
def test_structured_stale_epochs(gpu, name, loss, with_val, delay, mode):
    native = native_mod()
    g = structured_problem(structured_cases()[name], loss, with_val, delay + 7 * loss)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_stale(native, gpu, g, lv, delay, opt=dict(stale_mode=mode))


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("delay", [0, 2, 8, 64])
@pytest.mark.parametrize("mode", STALE_MODES)
def test_random_stale_epochs(gpu, cfg, delay, mode):
    native = native_mod()
    g = datagen.generate(cfg, n=8000, d=4000 if cfg == 4 else 500, seed=40 + delay)
    g["lr"] = np.float32(g["lr"] / 4)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    w0 = (0.05 * np.random.default_rng(delay).normal(size=g["d"])).astype(np.float32)
    check_stale(native, gpu, g, lv, delay, w0, opt=dict(stale_mode=mode))


def test_delay_zero_equals_gpu_sgd(gpu):
    native = native_mod()
    g = datagen.generate(2, n=5000, d=400, seed=46)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    got = check_stale(native, gpu, g, lv, 0)
    sgd = gpu_sgd(native, gpu, g, lv)
    assert np.array_equal(got.view(np.int32), sgd.view(np.int32))


def test_stale_errors(gpu):
    import torch

    native = native_mod()
    row_ptr, col = csr_from_rows([{0, 1}, {1, 2}])
    g = dict(row_ptr=row_ptr, col=col, val=None, y=np.ones(2, np.float32), n=2, d=3,
             lr=np.float32(0.1), loss=0)
    lv, _ = gpu_schedule(native, gpu, row_ptr, col, 3, 0)
    csr = native.Csr.from_numpy(row_ptr, col, None, gpu)
    y = torch.ones(2, dtype=torch.float32, device=gpu)
    w = torch.zeros(3, dtype=torch.float32, device=gpu)
    with pytest.raises(native.PdbError) as e:
        native.pdb_stale_epoch(csr, y, 2, 3, w, 0.1, 0, -1, lv)
    assert e.value.code == native.PDB_ERR_INVALID_ARG
    small = native.workspace(16, gpu)
    with pytest.raises(native.PdbError) as e:
        native.pdb_stale_epoch(csr, y, 2, 3, w, 0.1, 0, 1, lv, ws=small)
    assert e.value.code == native.PDB_ERR_WORKSPACE
    check_stale(native, gpu, g, lv, 1)


def test_windows_too_large_fall_back(gpu):
    # 60 entries per example: windows of 40 examples hold 2400 entries, over
    # the block's 2048, so the sync-free execution runs; 30 fit
    native = native_mod()
    rows = [set(range(i % 7, i % 7 + 60)) for i in range(500)]
    g = structured_problem(rows, 1, True, 3)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    for delay in (29, 39):
        check_stale(native, gpu, g, lv, delay, opt=dict(stale_mode=2))


@pytest.mark.parametrize("mode", [0, 2])
def test_empty_rows_and_window_edges(gpu, mode):
    opt = dict(stale_mode=mode)
    # empty examples, a last window shorter than delay + 1, one example
    native = native_mod()
    rows = [set(), {0, 1}, set(), {1, 2}, {2}, set(), {0, 2, 3}, {3}, set(), {1}, {0}]
    for delay in (0, 1, 2, 3, 4, 10, 11, 50):
        g = structured_problem(rows, 0, True, delay)
        lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
        check_stale(native, gpu, g, lv, delay, opt=opt)
    g = structured_problem([{5}], 1, False, 2)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_stale(native, gpu, g, lv, 3, opt=opt)
    # the largest delay: every read at the initial weights
    g = structured_problem(rows, 0, True, 9)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_stale(native, gpu, g, lv, 2 ** 63 - 1, opt=opt)


@pytest.mark.parametrize("cfg,delay", [(2, 8), (4, 8)])
def test_full_size_stale(gpu, cfg, delay):
    # the executions bench.py --delay 8 times (windowed on config 2, sync-free
    # on config 4)
    native = native_mod()
    g = datagen.generate(cfg)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_stale(native, gpu, g, lv, delay)
