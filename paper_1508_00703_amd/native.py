"""ctypes binding of libpdb.so (argument marshalling only).

Every entry point has the C name.  Arrays are torch tensors on the GPU (torch
is used for device memory and streams only); all computation happens in the
HIP kernels of libpdb.so.  If the library is missing, ``load()`` raises:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpdb.so")

PDB_OK = 0
PDB_ERR_INVALID_ARG = -1
PDB_ERR_BAD_CSR = -2
PDB_ERR_WORKSPACE = -3
PDB_ERR_HIP = -4
PDB_ERR_DEVICE = -5
PDB_ERR_UNSUPPORTED = -6
PDB_LOGISTIC, PDB_SQUARED = 0, 1
PDB_SCHED_AUTO, PDB_SCHED_CHAINSCAN, PDB_SCHED_DATAFLOW, PDB_SCHED_SPINE = 0, 1, 2, 3
PDB_SCHED_CHAIN = 4
PDB_SCHED_WALK = 5
PDB_SCHED_SHORT = 6
PDB_EPOCH_AUTO, PDB_EPOCH_LEVELS, PDB_EPOCH_SYNCFREE = 0, 1, 2
PDB_STALE_AUTO, PDB_STALE_SYNCFREE, PDB_STALE_WINDOWED = 0, 1, 2

# every symbol declared in include/pdb.h
EXPORTS = (
    "pdb_strerror", "pdb_last_hip_error", "pdb_schedule_workspace_bytes",
    "pdb_epoch_workspace_bytes", "pdb_schedule", "pdb_sgd_epoch", "pdb_mf_epoch",
    "pdb_validate_csr", "pdb_workspace_status", "pdb_transpose", "pdb_prev_writer",
    "pdb_check_reciprocal", "pdb_batch_schedule", "pdb_batch_epoch",
    "pdb_stale_workspace_bytes", "pdb_stale_epoch", "pdb_dense_plan",
    "pdb_dense_workspace_bytes", "pdb_dense_gd", "pdb_options_init", "pdb_validate_schedule",
    "pdb_sgd_epoch_noalloc",
    # include/pdb_mb.h
    "pdb_mb_workspace_bytes", "pdb_mb_copy", "pdb_mb_hop", "pdb_mb_barrier",
)


class PdbCsr(ctypes.Structure):
    _fields_ = [("row_ptr", ctypes.c_void_p), ("col", ctypes.c_void_p), ("val", ctypes.c_void_p),
                ("nnz", ctypes.c_int64)]


class PdbLevels(ctypes.Structure):
    _fields_ = [("level", ctypes.c_void_p), ("perm", ctypes.c_void_p),
                ("level_ptr", ctypes.c_void_p), ("n_levels", ctypes.c_void_p),
                ("prev_nz", ctypes.c_void_p), ("L_host", ctypes.c_int64),
                ("max_width_host", ctypes.c_int64)]


class PdbBatches(ctypes.Structure):
    _fields_ = [("bptr", ctypes.c_void_p), ("ucol", ctypes.c_void_p), ("uptr", ctypes.c_void_p),
                ("occ", ctypes.c_void_p), ("occ_row", ctypes.c_void_p), ("occ_u", ctypes.c_void_p),
                ("unext", ctypes.c_void_p), ("U_host", ctypes.c_int64)]


class PdbScheduleInfo(ctypes.Structure):
    _fields_ = [("method_used", ctypes.c_int32), ("rounds", ctypes.c_int32),
                ("n_levels", ctypes.c_int64), ("max_width", ctypes.c_int64)]


class PdbOptions(ctypes.Structure):
    _fields_ = [("epoch_mode", ctypes.c_int32), ("pipeline", ctypes.c_int32),
                ("pipeline_width", ctypes.c_int32), ("thin_max", ctypes.c_int32),
                ("hot_features", ctypes.c_int64), ("spin_timeout_us", ctypes.c_int64),
                ("batch_thin_max", ctypes.c_int32), ("batch_syncfree_blocks", ctypes.c_int32),
                ("stale_mode", ctypes.c_int32), ("dense_stream", ctypes.c_int32),
                ("mf_one_cu", ctypes.c_int32)]


class PdbError(RuntimeError):
    def __init__(self, code: int, where: str):
        lib = load()
        msg = lib.pdb_strerror(code).decode()
        hip = lib.pdb_last_hip_error() if code == PDB_ERR_HIP else 0
        super().__init__("%s: %s (status %d%s)" % (where, msg, code,
                                                     ", hipError %d" % hip if hip else ""))
        self.code = code


_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libpdb.so not built: run paper_1508_00703_amd/build.py "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, i64, i32, f32, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                            ctypes.c_size_t)
    lib.pdb_strerror.argtypes = [ctypes.c_int]
    lib.pdb_strerror.restype = ctypes.c_char_p
    lib.pdb_last_hip_error.argtypes = []
    lib.pdb_schedule_workspace_bytes.argtypes = [i64, i64, i64, ctypes.POINTER(sz)]
    lib.pdb_epoch_workspace_bytes.argtypes = [i64, ctypes.POINTER(sz)]
    O = ctypes.POINTER(PdbOptions)
    lib.pdb_options_init.argtypes = [O]
    lib.pdb_schedule.argtypes = [ctypes.POINTER(PdbCsr), P, i64, i64, ctypes.POINTER(PdbLevels),
                                 ctypes.c_int, ctypes.POINTER(PdbScheduleInfo), P, sz, O, P]
    lib.pdb_sgd_epoch.argtypes = [ctypes.POINTER(PdbCsr), P, i64, i64, P, f32, ctypes.c_int,
                                  ctypes.POINTER(PdbLevels), P, sz, O, P]
    lib.pdb_sgd_epoch_noalloc.argtypes = [ctypes.POINTER(PdbCsr), P, i64, i64, P, f32,
                                          ctypes.c_int, ctypes.POINTER(PdbLevels), P, O, P]
    lib.pdb_mf_epoch.argtypes = [P, P, P, i64, P, i64, P, i64, i32, f32, f32,
                                 ctypes.POINTER(PdbLevels), P, sz, O, P]
    lib.pdb_validate_csr.argtypes = [ctypes.POINTER(PdbCsr), i64, i64, P, sz, P]
    lib.pdb_validate_schedule.argtypes = [ctypes.POINTER(PdbCsr), i64, i64,
                                          ctypes.POINTER(PdbLevels), P, sz, P]
    lib.pdb_workspace_status.argtypes = [P, P]
    lib.pdb_transpose.argtypes = [ctypes.POINTER(PdbCsr), i64, i64, P, P, P, sz, P]
    lib.pdb_prev_writer.argtypes = [ctypes.POINTER(PdbCsr), i64, i64, P, P, P, sz, P]
    lib.pdb_check_reciprocal.argtypes = [ctypes.c_uint32, ctypes.c_uint32,
                                         ctypes.POINTER(ctypes.c_uint64),
                                         ctypes.POINTER(ctypes.c_uint32), P, sz, P]
    lib.pdb_batch_schedule.argtypes = [ctypes.POINTER(PdbCsr), i64, i64, i64,
                                       ctypes.POINTER(PdbBatches), ctypes.POINTER(PdbLevels),
                                       ctypes.c_int, ctypes.POINTER(PdbScheduleInfo), P, sz, O, P]
    lib.pdb_batch_epoch.argtypes = [ctypes.POINTER(PdbCsr), P, i64, i64, i64, P, f32, ctypes.c_int,
                                    ctypes.POINTER(PdbBatches), ctypes.POINTER(PdbLevels), P, sz,
                                    O, P]
    lib.pdb_stale_workspace_bytes.argtypes = [i64, ctypes.POINTER(sz)]
    lib.pdb_stale_epoch.argtypes = [ctypes.POINTER(PdbCsr), P, i64, i64, P, f32, ctypes.c_int, i64,
                                    P, P, sz, O, P]
    lib.pdb_dense_plan.argtypes = [i64, i64, ctypes.c_int, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.pdb_dense_workspace_bytes.argtypes = [i64, i64, i64, i64, ctypes.POINTER(sz)]
    lib.pdb_dense_gd.argtypes = [P, i64, P, i64, i64, P, f32, ctypes.c_int, i64, i64, i64, P, sz,
                                 O, P]
    lib.pdb_mb_workspace_bytes.argtypes = [ctypes.POINTER(sz)]
    lib.pdb_mb_copy.argtypes = [P, P, sz, P]
    lib.pdb_mb_hop.argtypes = [i64, i32, P, sz, ctypes.POINTER(ctypes.c_double),
                               ctypes.POINTER(i32), ctypes.POINTER(i32), O, P]
    lib.pdb_mb_barrier.argtypes = [i64, i32, P, sz, ctypes.POINTER(ctypes.c_double), O, P]
    for name in EXPORTS:
        if name not in ("pdb_strerror",):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(code: int, where: str):
    if code != PDB_OK:
        raise PdbError(code, where)


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def options(**fields) -> PdbOptions:
    """pdb_options with the library's defaults, then the given fields
    (e.g. options(epoch_mode=PDB_EPOCH_LEVELS, hot_features=0))."""
    o = PdbOptions()
    _check(load().pdb_options_init(ctypes.byref(o)), "pdb_options_init")
    for k, v in fields.items():
        if k not in dict(PdbOptions._fields_):
            raise TypeError("unknown option %r" % k)
        setattr(o, k, int(v))
    return o


def _opt(opt):
    """None (defaults), a PdbOptions, or a dict of fields."""
    if opt is None:
        return None
    if isinstance(opt, dict):
        opt = options(**opt)
    return ctypes.byref(opt)


def _stream(stream, device):
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


class Csr:
    """Device CSR: row_ptr int64[n+1], col int32[nnz], val float32[nnz] or None."""

    def __init__(self, row_ptr: torch.Tensor, col: torch.Tensor, val: torch.Tensor | None):
        if row_ptr.dtype != torch.int64 or col.dtype != torch.int32:
            raise TypeError("row_ptr must be int64 and col int32")
        if val is not None and val.dtype != torch.float32:
            raise TypeError("val must be float32")
        self.row_ptr, self.col, self.val = row_ptr, col, val
        self.n = row_ptr.numel() - 1
        self.nnz = col.numel()
        self.device = row_ptr.device

    @classmethod
    def from_numpy(cls, row_ptr, col, val=None, device="cuda"):
        rp = torch.from_numpy(row_ptr).to(device)
        c = torch.from_numpy(col).to(device)
        v = None if val is None else torch.from_numpy(val).to(device)
        return cls(rp, c, v)

    def c(self) -> PdbCsr:
        return PdbCsr(_ptr(self.row_ptr), _ptr(self.col), _ptr(self.val), self.nnz)


class Levels:
    """Device output of pdb_schedule."""

    def __init__(self, n: int, nnz: int, device, with_prev_nz: bool = True):
        self.level = torch.empty(max(n, 0), dtype=torch.int32, device=device)
        self.perm = torch.empty(max(n, 0), dtype=torch.int32, device=device)
        self.level_ptr = torch.empty(n + 1, dtype=torch.int64, device=device)
        self.n_levels = torch.empty(1, dtype=torch.int32, device=device)
        self.prev_nz = (torch.empty(max(nnz, 0), dtype=torch.int32, device=device)
                        if with_prev_nz else None)
        self.L_host = 0
        self.max_width_host = 0

    @classmethod
    def from_host(cls, level, perm, level_ptr, device, max_width=None):
        """Schedule given as host arrays (e.g. from another implementation)."""
        import numpy as np

        n = len(level)
        lv = cls(n, 0, device, with_prev_nz=False)
        lv.level.copy_(torch.from_numpy(np.asarray(level, np.int32)))
        lv.perm.copy_(torch.from_numpy(np.asarray(perm, np.int32)))
        lv.level_ptr = torch.from_numpy(np.asarray(level_ptr, np.int64)).to(device)
        L = len(level_ptr) - 1
        lv.n_levels.fill_(L)
        lv.L_host = L
        lv.max_width_host = int(max_width if max_width is not None else
                                (np.diff(level_ptr).max() if L > 0 else 0))
        return lv

    def c(self) -> PdbLevels:
        return PdbLevels(_ptr(self.level), _ptr(self.perm), _ptr(self.level_ptr),
                         _ptr(self.n_levels), _ptr(self.prev_nz), self.L_host,
                         self.max_width_host)


class Batches:
    """Device output of pdb_batch_schedule: each batch's union of features and the
    occurrence lists (sized for the worst case U = nnz)."""

    def __init__(self, n: int, nnz: int, batch: int, device):
        nb = (n + batch - 1) // batch
        self.batch = batch
        self.nb = nb
        self.bptr = torch.empty(nb + 1, dtype=torch.int64, device=device)
        self.ucol = torch.empty(max(nnz, 1), dtype=torch.int32, device=device)
        self.uptr = torch.empty(nnz + 1, dtype=torch.int64, device=device)
        self.occ = torch.empty(max(nnz, 1), dtype=torch.int32, device=device)
        self.occ_row = torch.empty(max(nnz, 1), dtype=torch.int32, device=device)
        self.occ_u = torch.empty(max(nnz, 1), dtype=torch.int32, device=device)
        self.unext = torch.empty(max(nnz, 1), dtype=torch.int32, device=device)
        self.U_host = 0

    def c(self) -> PdbBatches:
        return PdbBatches(_ptr(self.bptr), _ptr(self.ucol), _ptr(self.uptr), _ptr(self.occ),
                          _ptr(self.occ_row), _ptr(self.occ_u), _ptr(self.unext), self.U_host)


def pdb_strerror(code: int) -> str:
    return load().pdb_strerror(code).decode()


def pdb_schedule_workspace_bytes(n: int, d: int, nnz: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().pdb_schedule_workspace_bytes(n, d, nnz, ctypes.byref(out)),
           "pdb_schedule_workspace_bytes")
    return out.value


def pdb_epoch_workspace_bytes(d: int = 0) -> int:
    out = ctypes.c_size_t(0)
    _check(load().pdb_epoch_workspace_bytes(d, ctypes.byref(out)), "pdb_epoch_workspace_bytes")
    return out.value


def workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def pdb_schedule(csr: Csr, labels, n: int, d: int, levels: Levels, method: int = PDB_SCHED_AUTO,
                 ws: torch.Tensor | None = None, stream=None, opt=None) -> dict:
    if ws is None:
        ws = workspace(pdb_schedule_workspace_bytes(n, d, csr.nnz), csr.device)
    lv = levels.c()
    info = PdbScheduleInfo()
    _check(load().pdb_schedule(ctypes.byref(csr.c()), _ptr(labels), n, d, ctypes.byref(lv),
                               method, ctypes.byref(info), _ptr(ws), ws.numel(), _opt(opt),
                               _stream(stream, csr.device)), "pdb_schedule")
    levels.L_host, levels.max_width_host = lv.L_host, lv.max_width_host
    return dict(method_used=info.method_used, rounds=info.rounds, n_levels=info.n_levels,
                max_width=info.max_width)


def pdb_sgd_epoch(csr: Csr, labels: torch.Tensor, n: int, d: int, w: torch.Tensor, lr: float,
                  loss: int, levels: Levels, ws: torch.Tensor | None = None, stream=None,
                  opt=None):
    if w.dtype != torch.float32 or labels.dtype != torch.float32:
        raise TypeError("w and labels must be float32")
    if w.numel() < d or labels.numel() < n:
        raise ValueError("w must hold d entries and labels n entries")
    if ws is None:
        ws = workspace(pdb_epoch_workspace_bytes(d), csr.device)
    _check(load().pdb_sgd_epoch(ctypes.byref(csr.c()), _ptr(labels), n, d, _ptr(w),
                                ctypes.c_float(lr), loss, ctypes.byref(levels.c()), _ptr(ws),
                                ws.numel(), _opt(opt), _stream(stream, csr.device)),
           "pdb_sgd_epoch")
    return ws


def pdb_sgd_epoch_noalloc(csr: Csr, labels: torch.Tensor, n: int, d: int, w: torch.Tensor,
                          lr: float, loss: int, levels: Levels, status: torch.Tensor | None = None,
                          stream=None, opt=None):
    """pdb_sgd_epoch on the library's own scratch (no workspace); status: an
    int32 device tensor of one element that receives the device error code."""
    if w.dtype != torch.float32 or labels.dtype != torch.float32:
        raise TypeError("w and labels must be float32")
    if w.numel() < d or labels.numel() < n:
        raise ValueError("w must hold d entries and labels n entries")
    if status is not None and (status.dtype != torch.int32 or status.numel() < 1):
        raise TypeError("status must be an int32 device tensor")
    _check(load().pdb_sgd_epoch_noalloc(ctypes.byref(csr.c()), _ptr(labels), n, d, _ptr(w),
                                        ctypes.c_float(lr), loss, ctypes.byref(levels.c()),
                                        _ptr(status), _opt(opt), _stream(stream, csr.device)),
           "pdb_sgd_epoch_noalloc")


def pdb_mf_epoch(user, item, rating, n: int, U, n_users: int, V, n_items: int, rank: int,
                 lr: float, reg: float, levels: Levels, ws=None, stream=None, opt=None):
    for t, name in ((user, "user"), (item, "item")):
        if t.dtype != torch.int32 or t.numel() < n:
            raise TypeError("%s must be int32[n]" % name)
    if U.numel() < n_users * rank or V.numel() < n_items * rank:
        raise ValueError("U / V too small")
    if ws is None:
        ws = workspace(pdb_epoch_workspace_bytes((n_users + n_items) * rank), U.device)
    _check(load().pdb_mf_epoch(_ptr(user), _ptr(item), _ptr(rating), n, _ptr(U), n_users,
                               _ptr(V), n_items, rank, ctypes.c_float(lr), ctypes.c_float(reg),
                               ctypes.byref(levels.c()), _ptr(ws), ws.numel(), _opt(opt),
                               _stream(stream, U.device)), "pdb_mf_epoch")
    return ws


def pdb_batch_schedule(csr: Csr, n: int, d: int, batches: Batches, levels: Levels,
                       method: int = PDB_SCHED_AUTO, ws: torch.Tensor | None = None,
                       stream=None, opt=None) -> dict:
    """levels: a Levels for nb = ceil(n / batch) rows and (for prev_nz) nnz entries."""
    if ws is None:
        ws = workspace(pdb_schedule_workspace_bytes(n, d, csr.nnz), csr.device)
    bt = batches.c()
    lv = levels.c()
    info = PdbScheduleInfo()
    _check(load().pdb_batch_schedule(ctypes.byref(csr.c()), n, d, batches.batch, ctypes.byref(bt),
                                     ctypes.byref(lv), method, ctypes.byref(info), _ptr(ws),
                                     ws.numel(), _opt(opt), _stream(stream, csr.device)),
           "pdb_batch_schedule")
    batches.U_host = bt.U_host
    levels.L_host, levels.max_width_host = lv.L_host, lv.max_width_host
    return dict(method_used=info.method_used, rounds=info.rounds, n_levels=info.n_levels,
                max_width=info.max_width)


def pdb_batch_epoch(csr: Csr, labels: torch.Tensor, n: int, d: int, w: torch.Tensor, lr: float,
                    loss: int, batches: Batches, levels: Levels, ws: torch.Tensor | None = None,
                    stream=None, opt=None):
    if w.dtype != torch.float32 or labels.dtype != torch.float32:
        raise TypeError("w and labels must be float32")
    if w.numel() < d or labels.numel() < n:
        raise ValueError("w must hold d entries and labels n entries")
    if ws is None:
        ws = workspace(pdb_epoch_workspace_bytes(d), csr.device)
    _check(load().pdb_batch_epoch(ctypes.byref(csr.c()), _ptr(labels), n, d, batches.batch, _ptr(w),
                                  ctypes.c_float(lr), loss, ctypes.byref(batches.c()),
                                  ctypes.byref(levels.c()), _ptr(ws), ws.numel(), _opt(opt),
                                  _stream(stream, csr.device)), "pdb_batch_epoch")
    return ws


def pdb_stale_workspace_bytes(nnz: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().pdb_stale_workspace_bytes(nnz, ctypes.byref(out)), "pdb_stale_workspace_bytes")
    return out.value


def pdb_stale_epoch(csr: Csr, labels: torch.Tensor, n: int, d: int, w: torch.Tensor, lr: float,
                    loss: int, delay: int, levels: Levels, ws: torch.Tensor | None = None,
                    stream=None, opt=None):
    """levels: from pdb_schedule on the same CSR (its prev_nz is used)."""
    if w.dtype != torch.float32 or labels.dtype != torch.float32:
        raise TypeError("w and labels must be float32")
    if w.numel() < d or labels.numel() < n:
        raise ValueError("w must hold d entries and labels n entries")
    if levels.prev_nz is None and csr.nnz > 0:
        raise ValueError("the levels must carry prev_nz")
    if ws is None:
        ws = workspace(pdb_stale_workspace_bytes(csr.nnz), csr.device)
    _check(load().pdb_stale_epoch(ctypes.byref(csr.c()), _ptr(labels), n, d, _ptr(w),
                                  ctypes.c_float(lr), loss, delay, _ptr(levels.prev_nz), _ptr(ws),
                                  ws.numel(), _opt(opt), _stream(stream, csr.device)),
           "pdb_stale_epoch")
    return ws


def pdb_dense_plan(n: int, d: int, workers: int = 0) -> tuple[int, int]:
    """(row_block, col_block) for n x d on `workers` workers (0: the device's CUs)."""
    rb, cb = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(load().pdb_dense_plan(n, d, workers, ctypes.byref(rb), ctypes.byref(cb)),
           "pdb_dense_plan")
    return rb.value, cb.value


def pdb_dense_workspace_bytes(n: int, d: int, row_block: int, col_block: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().pdb_dense_workspace_bytes(n, d, row_block, col_block, ctypes.byref(out)),
           "pdb_dense_workspace_bytes")
    return out.value


def pdb_dense_gd(X: torch.Tensor, labels: torch.Tensor, w: torch.Tensor, lr: float, loss: int,
                 iters: int, row_block: int = 0, col_block: int = 0,
                 ws: torch.Tensor | None = None, stream=None, opt=None):
    """X: float32 device matrix n x d with unit column stride (any row stride
    >= d).  row_block = col_block = 0 takes pdb_dense_plan's blocking."""
    if X.dtype != torch.float32 or w.dtype != torch.float32 or labels.dtype != torch.float32:
        raise TypeError("X, w and labels must be float32")
    if X.dim() != 2 or (X.shape[0] > 1 and X.shape[1] > 0 and X.stride(1) != 1):
        raise ValueError("X must be a matrix with unit column stride")
    n, d = X.shape
    ldx = X.stride(0) if n > 1 else d
    if w.numel() < d or labels.numel() < n:
        raise ValueError("w must hold d entries and labels n entries")
    if row_block == 0 and col_block == 0:
        row_block, col_block = pdb_dense_plan(n, d)
    if ws is None:
        ws = workspace(pdb_dense_workspace_bytes(n, d, row_block, col_block), X.device)
    if not X.is_cuda:
        raise ValueError("expected a device tensor")
    _check(load().pdb_dense_gd(X.data_ptr() if X.numel() else None, ldx, _ptr(labels), n, d, _ptr(w), ctypes.c_float(lr), loss,
                               iters, row_block, col_block, _ptr(ws), ws.numel(), _opt(opt),
                               _stream(stream, X.device)), "pdb_dense_gd")
    return ws


def pdb_validate_csr(csr: Csr, n: int, d: int, ws=None, stream=None) -> int:
    """Returns the status code (PDB_OK or PDB_ERR_BAD_CSR); raises on other errors."""
    if ws is None:
        ws = workspace(pdb_epoch_workspace_bytes(), csr.device)
    rc = load().pdb_validate_csr(ctypes.byref(csr.c()), n, d, _ptr(ws), ws.numel(),
                                 _stream(stream, csr.device))
    if rc not in (PDB_OK, PDB_ERR_BAD_CSR):
        raise PdbError(rc, "pdb_validate_csr")
    return rc


def pdb_validate_schedule(csr: Csr, n: int, d: int, levels: Levels, ws=None, stream=None) -> int:
    """Returns PDB_OK or PDB_ERR_DEVICE (a schedule the epoch may not run);
    raises on other errors."""
    if ws is None:
        ws = workspace(pdb_schedule_workspace_bytes(n, d, csr.nnz), csr.device)
    rc = load().pdb_validate_schedule(ctypes.byref(csr.c()), n, d, ctypes.byref(levels.c()),
                                      _ptr(ws), ws.numel(), _stream(stream, csr.device))
    if rc not in (PDB_OK, PDB_ERR_DEVICE):
        raise PdbError(rc, "pdb_validate_schedule")
    return rc


def pdb_workspace_status(ws: torch.Tensor, stream=None) -> int:
    return load().pdb_workspace_status(_ptr(ws), _stream(stream, ws.device))


def pdb_transpose(csr: Csr, n: int, d: int, col_ptr, csc_row, ws=None, stream=None):
    if ws is None:
        ws = workspace(pdb_schedule_workspace_bytes(n, d, csr.nnz), csr.device)
    _check(load().pdb_transpose(ctypes.byref(csr.c()), n, d, _ptr(col_ptr), _ptr(csc_row),
                                _ptr(ws), ws.numel(), _stream(stream, csr.device)),
           "pdb_transpose")


def pdb_prev_writer(csr: Csr, n: int, d: int, prev_row, prev_nz=None, ws=None, stream=None):
    if ws is None:
        ws = workspace(pdb_schedule_workspace_bytes(n, d, csr.nnz), csr.device)
    _check(load().pdb_prev_writer(ctypes.byref(csr.c()), n, d, _ptr(prev_row), _ptr(prev_nz),
                                  _ptr(ws), ws.numel(), _stream(stream, csr.device)),
           "pdb_prev_writer")


def pdb_check_reciprocal(lo_bits: int, hi_bits: int, device, ws=None, stream=None):
    """(mismatches, first mismatching bit pattern or 0xFFFFFFFF)."""
    if ws is None:
        ws = workspace(pdb_epoch_workspace_bytes(), device)
    bad = ctypes.c_uint64(0)
    first = ctypes.c_uint32(0)
    _check(load().pdb_check_reciprocal(lo_bits, hi_bits, ctypes.byref(bad), ctypes.byref(first),
                                       _ptr(ws), ws.numel(), _stream(stream, device)),
           "pdb_check_reciprocal")
    return bad.value, first.value


# ---------------------------------------------------------------------------
# microbenchmarks (include/pdb_mb.h)

def pdb_mb_workspace_bytes() -> int:
    out = ctypes.c_size_t(0)
    _check(load().pdb_mb_workspace_bytes(ctypes.byref(out)), "pdb_mb_workspace_bytes")
    return out.value


def pdb_mb_copy(src: torch.Tensor, dst: torch.Tensor, stream=None):
    """Streams src into dst (same byte size, a multiple of 16) with the
    library's copy kernel."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("src and dst must have the same size")
    _check(load().pdb_mb_copy(_ptr(src), _ptr(dst), nbytes, _stream(stream, src.device)),
           "pdb_mb_copy")


def pdb_mb_hop(rounds: int, partner: int, device, ws=None, stream=None, opt=None):
    """(ns per round trip, XCD of block 0, XCD of the partner block)."""
    if ws is None:
        ws = workspace(pdb_mb_workspace_bytes(), device)
    ns = ctypes.c_double(0)
    xa, xb = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(load().pdb_mb_hop(rounds, partner, _ptr(ws), ws.numel(), ctypes.byref(ns),
                             ctypes.byref(xa), ctypes.byref(xb), _opt(opt),
                             _stream(stream, device)), "pdb_mb_hop")
    return ns.value, xa.value, xb.value


def pdb_mb_barrier(rounds: int, blocks: int, device, ws=None, stream=None, opt=None) -> float:
    """ns per grid-wide barrier over `blocks` resident blocks."""
    if ws is None:
        ws = workspace(pdb_mb_workspace_bytes(), device)
    ns = ctypes.c_double(0)
    _check(load().pdb_mb_barrier(rounds, blocks, _ptr(ws), ws.numel(), ctypes.byref(ns),
                                 _opt(opt), _stream(stream, device)), "pdb_mb_barrier")
    return ns.value
