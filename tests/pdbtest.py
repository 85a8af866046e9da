"""Shared helpers for the tests: run the HIP path through the C ABI and the
oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import numpy as np

import oracle


def csr_from_rows(rows):
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in sorted(r)], dtype=np.int32)
    return row_ptr, col


def gpu_schedule(native, dev, row_ptr, col, d, method, with_prev=True, opt=None):
    import torch

    csr = native.Csr.from_numpy(row_ptr, col, None, dev)
    n = len(row_ptr) - 1
    lv = native.Levels(n, len(col), dev, with_prev_nz=with_prev)
    info = native.pdb_schedule(csr, None, n, d, lv, method, opt=opt)
    torch.cuda.synchronize()
    return lv, info


def check_schedule(native, dev, row_ptr, col, d, method, opt=None):
    """GPU levels, perm, level_ptr, L equal the oracle's exactly."""
    lv, info = gpu_schedule(native, dev, row_ptr, col, d, method, opt=opt)
    level, perm, level_ptr, L = oracle.schedule(row_ptr, col, d)
    assert lv.L_host == L and int(lv.n_levels.item()) == L
    assert np.array_equal(lv.level.cpu().numpy(), level)
    assert np.array_equal(lv.perm.cpu().numpy(), perm)
    assert np.array_equal(lv.level_ptr.cpu().numpy()[:L + 1], level_ptr)
    widths = np.diff(level_ptr)
    assert lv.max_width_host == (widths.max() if L else 0)
    if lv.prev_nz is not None:
        check_prev_nz(row_ptr, col, d, lv.prev_nz.cpu().numpy())
    return lv, info


def check_prev_nz(row_ptr, col, d, pn):
    """pn[p] is the entry, on the same feature, of the latest earlier example
    touching it (columns are unique in a row, so feature + row fix it)."""
    prev = oracle.prev_writer(row_ptr, col, d)
    has = prev >= 0
    assert np.array_equal(pn >= 0, has)
    assert np.array_equal(col[pn[has]], col[has])
    rows = np.searchsorted(row_ptr, pn[has], side="right") - 1
    assert np.array_equal(rows, prev[has])


def gpu_sgd(native, dev, g, lv, w0=None, opt=None):
    import torch

    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], dev)
    y = torch.from_numpy(g["y"]).to(dev)
    w = torch.from_numpy(np.zeros(g["d"], np.float32) if w0 is None else w0.copy()).to(dev)
    ws = native.pdb_sgd_epoch(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], lv, opt=opt)
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    return w.cpu().numpy()


def check_sgd(native, dev, g, lv, w0=None, tol=1e-5, opt=None):
    """Bitwise equal to the oracle in matched summation order; within tol of
    the natural-order oracle."""
    got = gpu_sgd(native, dev, g, lv, w0, opt=opt)
    w_init = np.zeros(g["d"], np.float32) if w0 is None else w0
    ref_m = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w_init, g["lr"], g["loss"],
                             oracle.MATCHED)
    bad = np.nonzero(got.view(np.int32) != ref_m.view(np.int32))[0]
    assert len(bad) == 0, "first mismatches %s: gpu %s oracle %s" % (
        bad[:5], got[bad[:5]], ref_m[bad[:5]])
    ref_n = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], w_init, g["lr"], g["loss"],
                             oracle.NATURAL)
    assert np.max(np.abs(got - ref_n), initial=0.0) <= tol
    return got


def gpu_mf(native, dev, g, lv, opt=None):
    import torch

    U = torch.from_numpy(g["U0"].copy()).to(dev)
    V = torch.from_numpy(g["V0"].copy()).to(dev)
    t = lambda a: torch.from_numpy(a).to(dev)
    ws = native.pdb_mf_epoch(t(g["user"]), t(g["item"]), t(g["rating"]), g["n"], U, g["n_users"],
                             V, g["n_items"], g["rank"], float(g["lr"]), float(g["reg"]), lv,
                             opt=opt)
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    return U.cpu().numpy(), V.cpu().numpy()


def check_mf(native, dev, g, lv, tol=1e-5, opt=None):
    U, V = gpu_mf(native, dev, g, lv, opt=opt)
    Um, Vm = oracle.mf_epoch(g["user"], g["item"], g["rating"], g["U0"], g["V0"], g["lr"], g["reg"],
                             oracle.MATCHED)
    assert np.array_equal(U.view(np.int32), Um.view(np.int32))
    assert np.array_equal(V.view(np.int32), Vm.view(np.int32))
    Un, Vn = oracle.mf_epoch(g["user"], g["item"], g["rating"], g["U0"], g["V0"], g["lr"], g["reg"],
                             oracle.NATURAL)
    assert max(np.abs(U - Un).max(), np.abs(V - Vn).max()) <= tol
