"""GPU parity of mini-batch gradient descent (pdb_batch_schedule,
pdb_batch_epoch) against the CPU oracle on the same seeded inputs: the batch
unions, occurrence lists, batch levels and grouping bit-exact; weights bitwise
equal to the oracle's matched order and within 1e-5 of its natural order."""
import numpy as np
import pytest

import datagen
import oracle
from pdbtest import csr_from_rows
from test_gpu_parity import structured_cases

pytestmark = pytest.mark.gpu


def native_mod():
    from paper_1508_00703_amd import native
    return native


def gpu_batch_schedule(native, dev, row_ptr, col, d, B, method=0):
    import torch

    n, nnz = len(row_ptr) - 1, len(col)
    csr = native.Csr.from_numpy(row_ptr, col, None, dev)
    bt = native.Batches(n, nnz, B, dev)
    lv = native.Levels(bt.nb, nnz, dev)
    info = native.pdb_batch_schedule(csr, n, d, bt, lv, method)
    torch.cuda.synchronize()
    return bt, lv, info


def check_batch_schedule(native, dev, row_ptr, col, d, B, method=0):
    bt, lv, info = gpu_batch_schedule(native, dev, row_ptr, col, d, B, method)
    bptr, ucol, uptr, occ = oracle.batch_union(row_ptr, col, d, B)
    U = len(ucol)
    assert bt.U_host == U
    assert np.array_equal(bt.bptr.cpu().numpy(), bptr)
    assert np.array_equal(bt.ucol.cpu().numpy()[:U], ucol)
    assert np.array_equal(bt.uptr.cpu().numpy()[:U + 1], uptr)
    nnz = len(col)
    assert np.array_equal(bt.occ.cpu().numpy()[:nnz], occ)
    row_of = np.repeat(np.arange(len(row_ptr) - 1), np.diff(row_ptr)).astype(np.int32)
    assert np.array_equal(bt.occ_row.cpu().numpy()[:nnz], row_of[occ])
    assert np.array_equal(bt.occ_u.cpu().numpy()[:nnz], np.repeat(np.arange(U), np.diff(uptr)))
    level, perm, level_ptr, L = oracle.batch_schedule(row_ptr, col, d, B)
    assert lv.L_host == L
    assert np.array_equal(lv.level.cpu().numpy(), level)
    assert np.array_equal(lv.perm.cpu().numpy(), perm)
    assert np.array_equal(lv.level_ptr.cpu().numpy()[:L + 1], level_ptr)
    # previous writer over the union CSR: the union entry of the latest earlier
    # batch on the same feature
    pn = lv.prev_nz.cpu().numpy()[:U]
    nxt = np.full(U, -1, np.int64)
    nxt[pn[pn >= 0]] = np.nonzero(pn >= 0)[0]
    assert np.array_equal(bt.unext.cpu().numpy()[:U], nxt)
    prev_batch = oracle.prev_writer(bptr, ucol, d)
    has = prev_batch >= 0
    assert np.array_equal(pn >= 0, has)
    assert np.array_equal(ucol[pn[has]], ucol[has])
    assert np.array_equal(np.searchsorted(bptr, pn[has], side="right") - 1, prev_batch[has])
    return bt, lv


def check_batch_epoch(native, dev, g, B, bt, lv, tol=1e-5, opt=None):
    import torch

    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], dev)
    y = torch.from_numpy(g["y"]).to(dev)
    w = torch.zeros(g["d"], dtype=torch.float32, device=dev)
    ws = native.pdb_batch_epoch(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], bt, lv,
                                opt=opt)
    # (the default workspace holds a word per feature: sync-free unless the
    # options ask for batch levels)
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    got = w.cpu().numpy()
    w0 = np.zeros(g["d"], np.float32)
    args = (g["row_ptr"], g["col"], g["val"], g["y"], w0, g["lr"], g["loss"])
    ref_m = oracle.batch_epoch(*args, oracle.MATCHED, B)
    bad = np.nonzero(got.view(np.int32) != ref_m.view(np.int32))[0]
    assert len(bad) == 0, "first mismatches %s: gpu %s oracle %s" % (bad[:5], got[bad[:5]],
                                                                     ref_m[bad[:5]])
    ref_n = oracle.batch_epoch(*args, oracle.NATURAL, B)
    assert np.max(np.abs(got - ref_n), initial=0.0) <= tol
    return got


BATCHES = [1, 2, 3, 7, 64, 4096]


@pytest.mark.parametrize("name", sorted(structured_cases()))
@pytest.mark.parametrize("B", BATCHES)
def test_structured_batch_schedules(gpu, name, B):
    rows = structured_cases()[name]
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1 if len(col) else 1
    check_batch_schedule(native_mod(), gpu, row_ptr, col, d, B)


def structured_problem(rows, loss, with_val, seed, B=1):
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1 if len(col) else 1
    n = len(rows)
    rng = np.random.default_rng(seed)
    val = rng.normal(size=len(col)).astype(np.float32) if with_val else None
    y = (np.where(rng.random(n) < 0.5, -1.0, 1.0) if loss == oracle.LOGISTIC
         else rng.normal(size=n)).astype(np.float32)
    # a step size that keeps each batch step contractive (lr times the sum of
    # the batch's |x_i|^2 below 1/2): diverging weights would make every
    # summation order disagree
    sq = np.bincount(np.repeat(np.arange(n), np.diff(row_ptr)),
                     weights=(val.astype(np.float64) ** 2 if with_val else np.ones(len(col))),
                     minlength=n)
    per_batch = np.add.reduceat(sq, np.arange(0, n, B)) if n else np.zeros(1)
    lr = np.float32(min(0.01, 0.5 / max(per_batch.max(), 1.0)))
    return dict(row_ptr=row_ptr, col=col, val=val, y=y, n=n, d=d, lr=lr, loss=loss)


EPOCH_MODES = [1, 2]  # batch levels, sync-free


@pytest.mark.parametrize("name", sorted(structured_cases()))
@pytest.mark.parametrize("loss", [0, 1])
@pytest.mark.parametrize("with_val", [True, False])
@pytest.mark.parametrize("B", [1, 3, 64])
@pytest.mark.parametrize("mode", EPOCH_MODES)
def test_structured_batch_epochs(gpu, name, loss, with_val, B, mode):
    native = native_mod()
    g = structured_problem(structured_cases()[name], loss, with_val, B + loss, B)
    bt, lv = check_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], B)
    check_batch_epoch(native, gpu, g, B, bt, lv, opt=dict(epoch_mode=mode))


def batch_workload(g, B):
    """A workload's mini-batch form: its learning rate divided by B, so that the
    summed gradient of a batch takes the step of its mean."""
    g = dict(g)
    g["lr"] = np.float32(g["lr"] / B)
    return g


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("B", [1, 5, 100, 1000, 4096])
@pytest.mark.parametrize("mode", EPOCH_MODES)
def test_random_batch_epochs(gpu, cfg, B, mode):
    native = native_mod()
    g = batch_workload(datagen.generate(cfg, n=6000, d=3000 if cfg == 4 else 500, seed=31 + B), B)
    bt, lv = check_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], B)
    check_batch_epoch(native, gpu, g, B, bt, lv, opt=dict(epoch_mode=mode))


@pytest.mark.parametrize("thin", [1, 1000000])
def test_wide_and_narrow_batch_levels(gpu, thin):
    # disjoint pairs of rows then a shared feature: wide levels (the grid and
    # device barriers) and a chain of narrow ones (block 0), or everything in
    # one block
    opt = dict(batch_thin_max=thin, epoch_mode=1)
    native = native_mod()
    rows = [{2 * i, 2 * i + 1} for i in range(3000)] + [{0, 7 + i % 50} for i in range(500)]
    rows += [{10000 + i} for i in range(2000)]
    for B in (2, 7):
        g = structured_problem(rows, oracle.LOGISTIC, True, 5, B)
        bt, lv = check_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], B)
        assert lv.max_width_host > 100
        check_batch_epoch(native, gpu, g, B, bt, lv, opt=opt)


def test_batch_of_one_equals_gpu_sgd(gpu):
    import torch

    from pdbtest import gpu_schedule, gpu_sgd

    native = native_mod()
    g = datagen.generate(2, n=5000, d=400, seed=44)
    bt, lv = check_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 1)
    got = check_batch_epoch(native, gpu, g, 1, bt, lv)
    lv1, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    sgd = gpu_sgd(native, gpu, g, lv1)
    assert np.array_equal(got.view(np.int32), sgd.view(np.int32))
    torch.cuda.synchronize()


def test_batch_errors(gpu):
    native = native_mod()
    row_ptr, col = csr_from_rows([{0, 1}, {1, 2}])
    csr = native.Csr.from_numpy(row_ptr, col, None, gpu)
    for B in (0, 4097):
        bt = native.Batches(2, 4, max(B, 1), gpu)
        bt.batch = B
        lv = native.Levels(2, 4, gpu)
        with pytest.raises(native.PdbError) as e:
            native.pdb_batch_schedule(csr, 2, 3, bt, lv)
        assert e.value.code == native.PDB_ERR_INVALID_ARG


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_full_size_batch(gpu, cfg):
    # the launch configuration bench.py --batch 100 times (sync-free)
    native = native_mod()
    g = batch_workload(datagen.generate(cfg), 100)
    bt, lv = check_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 100)
    print("config %d, batches of 100: L=%d max width=%d U=%d" % (cfg, lv.L_host, lv.max_width_host,
                                                                 bt.U_host), flush=True)
    check_batch_epoch(native, gpu, g, 100, bt, lv)


@pytest.mark.parametrize("cfg", [2, 4])
def test_full_size_batch_levels(gpu, cfg):
    # the batch-level execution at full size
    native = native_mod()
    g = batch_workload(datagen.generate(cfg), 100)
    bt, lv = check_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 100)
    check_batch_epoch(native, gpu, g, 100, bt, lv, opt=dict(epoch_mode=1))
