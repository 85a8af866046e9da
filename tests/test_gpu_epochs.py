"""Several epochs on one cached schedule (the schedule depends only on the
sparsity pattern, so it is computed once per data set): E epochs on the GPU,
each starting from the previous epoch's weights, against E epochs of the
oracle -- bitwise in matched order, within 1e-5 of natural order."""
import numpy as np
import pytest

import datagen
import oracle
from pdbtest import gpu_schedule
from test_gpu_batch import batch_workload, gpu_batch_schedule

pytestmark = pytest.mark.gpu

EPOCHS = 3


def native_mod():
    from paper_1508_00703_amd import native
    return native


def oracle_epochs(g, mode, B=0):
    w = np.zeros(g["d"], np.float32)
    for _ in range(EPOCHS):
        args = (g["row_ptr"], g["col"], g["val"], g["y"], w, g["lr"], g["loss"], mode)
        w = oracle.batch_epoch(*args, B) if B else oracle.sgd_epoch(*args)
    return w


def compare(got, g, B=0):
    ref_m = oracle_epochs(g, oracle.MATCHED, B)
    assert np.array_equal(got.view(np.int32), ref_m.view(np.int32))
    ref_n = oracle_epochs(g, oracle.NATURAL, B)
    assert np.max(np.abs(got - ref_n)) <= 1e-5


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("mode", [1, 2])
def test_sgd_epochs_on_a_cached_schedule(gpu, cfg, mode):
    import torch

    native = native_mod()
    g = datagen.generate(cfg, n=20000, d=6000 if cfg == 4 else 1000, seed=9)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], gpu)
    y = torch.from_numpy(g["y"]).to(gpu)
    w = torch.zeros(g["d"], dtype=torch.float32, device=gpu)
    ws = native.workspace(native.pdb_epoch_workspace_bytes(g["d"]), gpu)
    for _ in range(EPOCHS):
        native.pdb_sgd_epoch(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], lv, ws=ws,
                             opt=dict(epoch_mode=mode))
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    compare(w.cpu().numpy(), g)


@pytest.mark.parametrize("cfg", [1, 2, 4])
@pytest.mark.parametrize("mode", [1, 2])
def test_batch_epochs_on_a_cached_schedule(gpu, cfg, mode):
    import torch

    native = native_mod()
    B = 100
    g = batch_workload(datagen.generate(cfg, n=20000, d=6000 if cfg == 4 else 1000, seed=10), B)
    bt, lv, _ = gpu_batch_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], B)
    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], gpu)
    y = torch.from_numpy(g["y"]).to(gpu)
    w = torch.zeros(g["d"], dtype=torch.float32, device=gpu)
    ws = native.workspace(native.pdb_epoch_workspace_bytes(g["d"]), gpu)
    for _ in range(EPOCHS):
        native.pdb_batch_epoch(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], bt, lv, ws=ws,
                               opt=dict(epoch_mode=mode))
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    compare(w.cpu().numpy(), g, B)
