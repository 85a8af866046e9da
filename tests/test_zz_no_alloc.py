"""The entry point that allocates nothing (pdb_sgd_epoch_noalloc), through
the C ABI, against pdb_sgd_epoch on the same inputs: bitwise equal weights,
on two calls in a row (the second with a smaller input, so the scratch holds
the first call's contents), in both executions; the status word reports no
device error; sizes beyond the scratch are refused."""
import numpy as np
import pytest

import datagen
from pdbtest import gpu_schedule

pytestmark = pytest.mark.gpu


def run_pair(native, gpu, g, mode):
    import torch

    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], gpu)
    y = torch.from_numpy(g["y"]).to(gpu)
    opt = dict(epoch_mode=mode)
    w_ref = torch.zeros(g["d"], dtype=torch.float32, device=gpu)
    ws = native.pdb_sgd_epoch(csr, y, g["n"], g["d"], w_ref, float(g["lr"]), g["loss"], lv,
                              opt=opt)
    w = torch.zeros(g["d"], dtype=torch.float32, device=gpu)
    status = torch.full((1,), -7, dtype=torch.int32, device=gpu)
    native.pdb_sgd_epoch_noalloc(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], lv,
                                 status=status, opt=opt)
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    assert int(status.item()) == 0
    a, b = w_ref.cpu().numpy(), w.cpu().numpy()
    assert np.array_equal(a.view(np.int32), b.view(np.int32))
    return b


@pytest.mark.parametrize("mode", [1, 2])  # level by level, sync-free
def test_noalloc_equals_workspace_entry_point(gpu, mode):
    from paper_1508_00703_amd import native

    # a large call, then a smaller one on the scratch the first left behind
    big = datagen.generate(4, n=40_000, d=1_500_000)
    small = datagen.generate(2, n=20_000, d=2_000)
    run_pair(native, gpu, big, mode)
    run_pair(native, gpu, small, mode)


def test_noalloc_limits(gpu):
    import torch

    from paper_1508_00703_amd import native

    g = datagen.generate(1, n=200, d=50)
    lv, _ = gpu_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], gpu)
    y = torch.from_numpy(g["y"]).to(gpu)
    d_big = (1 << 21) + 1
    w = torch.zeros(d_big, dtype=torch.float32, device=gpu)
    with pytest.raises(native.PdbError) as e:
        native.pdb_sgd_epoch_noalloc(csr, y, g["n"], d_big, w, 0.1, 0, lv)
    assert e.value.code == native.PDB_ERR_UNSUPPORTED
    # the largest d the scratch holds, sync-free (a word per feature)
    d_max = 1 << 21
    w = torch.zeros(d_max, dtype=torch.float32, device=gpu)
    status = torch.full((1,), -7, dtype=torch.int32, device=gpu)
    native.pdb_sgd_epoch_noalloc(csr, y, g["n"], d_max, w, float(g["lr"]), g["loss"], lv,
                                 status=status, opt=dict(epoch_mode=2))
    w2 = torch.zeros(d_max, dtype=torch.float32, device=gpu)
    native.pdb_sgd_epoch(csr, y, g["n"], d_max, w2, float(g["lr"]), g["loss"], lv,
                         opt=dict(epoch_mode=2))
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert np.array_equal(w.cpu().numpy().view(np.int32), w2.cpu().numpy().view(np.int32))
    # no examples: nothing runs, the status still reads 0
    status.fill_(-7)
    native.pdb_sgd_epoch_noalloc(native.Csr.from_numpy(np.zeros(1, np.int64),
                                                       np.zeros(0, np.int32), None, gpu),
                                 y, 0, 10, w, 0.1, 0, native.Levels(0, 0, gpu), status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
