"""CPU oracle for sequentially-correct sparse SGD -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never does, and the two share no code.

What it computes (all single-threaded, binary32 arithmetic, see oracle.c):
  * ``levels_brute`` / ``levels_seq``: the conflict level of each example,
    i.e. the position of the example in the earliest layering that keeps every
    feature's accesses in example order (read/write constraints, Sec. 4.4 and
    Theorem 2, with one feature per partition);
  * ``bucket``: examples grouped by level;
  * ``prev_writer`` / ``transpose``: per-entry previous example on the same
    feature, and per-feature occurrence lists;
  * ``sgd_epoch`` / ``mf_epoch``: the sequential computation of Algorithm 1,
    one example per iteration (Sec. 6.3), with the gradient step of Sec. 2.
  * ``batch_levels_brute`` / ``batch_levels_seq`` / ``batch_union`` /
    ``batch_epoch``: the same with a mini-batch of B examples per iteration
    (Sec. 6.3's mini-batch gradient descent): batch levels, each batch's
    union of features with its occurrences in example order, and the
    sequential mini-batch epoch.
  * ``stale_epoch`` / ``stale_snapshot``: the bounded-delay relaxation of
    Sec. 7, in the execution that reads as early as its read constraint
    allows (example alpha computes z against the weights after examples
    0 .. alpha - delay - 1; updates applied in example order).
  * ``dense_gd``: full-batch gradient descent on a dense example matrix
    (every example in every iteration, the update of Sec. 2 as in the dense
    workloads of Sec. 6.1-6.2).
  * ``history``: the execution-history predicates of Definition 4 and
    Sec. 4.3-4.4 (see ``oracle.history``).

Parity of the paper's speed-up numbers is unpinned (no code, no figures).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

NATURAL, MATCHED = 0, 1
LOGISTIC, SQUARED = 0, 1


def build(force: bool = True) -> str:
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11",
                               "-shared", "-fPIC", "-o", tmp, src, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=False)
    lib = ctypes.CDLL(_LIB_PATH)
    P, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    lib.orc_exp.argtypes = [f32]
    lib.orc_exp.restype = f32
    lib.orc_sigmoid.argtypes = [f32]
    lib.orc_sigmoid.restype = f32
    lib.orc_levels_brute.argtypes = [i64, P, P, P]
    lib.orc_levels_brute.restype = i32
    lib.orc_levels_seq.argtypes = [i64, i64, P, P, P]
    lib.orc_levels_seq.restype = i32
    lib.orc_bucket.argtypes = [i64, P, i32, P, P]
    lib.orc_bucket.restype = ctypes.c_int
    lib.orc_prev_writer.argtypes = [i64, i64, P, P, P]
    lib.orc_prev_writer.restype = ctypes.c_int
    lib.orc_transpose.argtypes = [i64, i64, P, P, P, P]
    lib.orc_transpose.restype = ctypes.c_int
    lib.orc_sgd_apply.argtypes = [i64, P, P, P, P, P, P, f32, i32, i32]
    lib.orc_sgd_apply.restype = None
    lib.orc_mf_apply.argtypes = [i64, P, P, P, P, P, P, i32, f32, f32, i32]
    lib.orc_mf_apply.restype = None
    lib.orc_batch_levels_brute.argtypes = [i64, P, P, i64, P]
    lib.orc_batch_levels_brute.restype = i32
    lib.orc_batch_levels_seq.argtypes = [i64, i64, P, P, i64, P]
    lib.orc_batch_levels_seq.restype = i32
    lib.orc_batch_union.argtypes = [i64, i64, P, P, i64, P, P, P, P]
    lib.orc_batch_union.restype = i64
    lib.orc_batch_apply.argtypes = [i64, i64, P, P, P, P, P, P, f32, i32, i32, i64]
    lib.orc_batch_apply.restype = ctypes.c_int
    lib.orc_stale_snapshot.argtypes = [i64, i64, P, P, P, P, P, f32, i32, i32, i64]
    lib.orc_stale_snapshot.restype = ctypes.c_int
    lib.orc_stale_apply.argtypes = [i64, i64, P, P, P, P, P, f32, i32, i32, i64]
    lib.orc_dense_gd.argtypes = [i64, i64, P, i64, P, P, f32, i32, i32, i64, i64, i64, i64]
    lib.orc_dense_gd.restype = ctypes.c_int
    lib.orc_stale_apply.restype = ctypes.c_int
    _lib = lib
    return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data


def exp(x: float) -> np.float32:
    """e^x by Cody-Waite reduction and the degree-7 Taylor polynomial (binary32)."""
    return np.float32(_load().orc_exp(np.float32(x)))


def sigmoid(z: float) -> np.float32:
    """The logistic function of the matched mode: 1/(1 + exp(min(-z, 87)))."""
    return np.float32(_load().orc_sigmoid(np.float32(z)))


def levels_brute(row_ptr, col, n=None):
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1 if n is None else n
    level = np.empty(n, dtype=np.int32)
    L = _load().orc_levels_brute(n, _ptr(row_ptr), _ptr(col), _ptr(level))
    return level, int(L)


def levels_seq(row_ptr, col, d, n=None):
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1 if n is None else n
    level = np.empty(n, dtype=np.int32)
    L = _load().orc_levels_seq(n, d, _ptr(row_ptr), _ptr(col), _ptr(level))
    if L < 0:
        raise MemoryError
    return level, int(L)


def bucket(level, L):
    level = _c(level, np.int32)
    n = len(level)
    perm = np.empty(n, dtype=np.int32)
    level_ptr = np.empty(L + 1, dtype=np.int64)
    if _load().orc_bucket(n, _ptr(level), L, _ptr(perm), _ptr(level_ptr)) != 0:
        raise ValueError("level out of range")
    return perm, level_ptr


def schedule(row_ptr, col, d):
    """levels, perm, level_ptr, L as one call."""
    level, L = levels_seq(row_ptr, col, d)
    perm, level_ptr = bucket(level, L)
    return level, perm, level_ptr, L


def prev_writer(row_ptr, col, d):
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1
    prev = np.empty(len(col), dtype=np.int32)
    if _load().orc_prev_writer(n, d, _ptr(row_ptr), _ptr(col), _ptr(prev)) != 0:
        raise MemoryError
    return prev


def transpose(row_ptr, col, d):
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1
    col_ptr = np.empty(d + 1, dtype=np.int64)
    csc_row = np.empty(len(col), dtype=np.int32)
    if _load().orc_transpose(n, d, _ptr(row_ptr), _ptr(col), _ptr(col_ptr), _ptr(csc_row)) != 0:
        raise MemoryError
    return col_ptr, csc_row


def sgd_epoch(row_ptr, col, val, y, w, lr, loss=LOGISTIC, mode=MATCHED, order=None, count=None):
    """Apply one epoch in place on a copy of w and return it.

    order: None = example order 0..n-1 (the sequential computation); otherwise
    the sequence of example indices to apply.  count limits the number of
    steps (a prefix of the order)."""
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    val = None if val is None else _c(val, np.float32)
    y = _c(y, np.float32)
    w = np.array(w, dtype=np.float32, copy=True)
    n = len(row_ptr) - 1
    if order is not None:
        order = _c(order, np.int32)
        cnt = len(order) if count is None else count
    else:
        cnt = n if count is None else count
    _load().orc_sgd_apply(cnt, _ptr(order), _ptr(row_ptr), _ptr(col), _ptr(val), _ptr(y),
                          _ptr(w), np.float32(lr), loss, mode)
    return w


def mf_epoch(user, item, rating, U, V, lr, reg, mode=MATCHED, order=None, count=None):
    user = _c(user, np.int32)
    item = _c(item, np.int32)
    rating = _c(rating, np.float32)
    U = np.array(U, dtype=np.float32, copy=True, order="C")
    V = np.array(V, dtype=np.float32, copy=True, order="C")
    rank = U.shape[1]
    if V.shape[1] != rank or rank > 64 or rank & (rank - 1):
        raise ValueError("rank must be a power of two <= 64 and equal for U and V")
    if order is not None:
        order = _c(order, np.int32)
        cnt = len(order) if count is None else count
    else:
        cnt = len(user) if count is None else count
    _load().orc_mf_apply(cnt, _ptr(order), _ptr(user), _ptr(item), _ptr(rating), _ptr(U), _ptr(V),
                         rank, np.float32(lr), np.float32(reg), mode)
    return U, V


def n_batches(n, B):
    return (n + B - 1) // B


def batch_levels_brute(row_ptr, col, B):
    """Batch levels from the definition (tiny inputs)."""
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1
    level = np.empty(n_batches(n, B), dtype=np.int32)
    L = _load().orc_batch_levels_brute(n, _ptr(row_ptr), _ptr(col), B, _ptr(level))
    return level, int(L)


def batch_levels_seq(row_ptr, col, d, B):
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1
    level = np.empty(n_batches(n, B), dtype=np.int32)
    L = _load().orc_batch_levels_seq(n, d, _ptr(row_ptr), _ptr(col), B, _ptr(level))
    if L < 0:
        raise MemoryError
    return level, int(L)


def batch_schedule(row_ptr, col, d, B):
    """Batch levels, batches grouped by level (perm, level_ptr), L."""
    level, L = batch_levels_seq(row_ptr, col, d, B)
    perm, level_ptr = bucket(level, L)
    return level, perm, level_ptr, L


def batch_union(row_ptr, col, d, B):
    """(bptr, ucol, uptr, occ): batch b's union features are ucol[bptr[b]:bptr[b+1]],
    ascending; union entry u's occurrences are the CSR entries occ[uptr[u]:uptr[u+1]]
    in example order."""
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    n = len(row_ptr) - 1
    nnz = len(col)
    bptr = np.empty(n_batches(n, B) + 1, dtype=np.int64)
    ucol = np.empty(max(nnz, 1), dtype=np.int32)
    uptr = np.empty(nnz + 1, dtype=np.int64)
    occ = np.empty(max(nnz, 1), dtype=np.int32)
    U = _load().orc_batch_union(n, d, _ptr(row_ptr), _ptr(col), B, _ptr(bptr), _ptr(ucol),
                                _ptr(uptr), _ptr(occ))
    if U < 0:
        raise MemoryError
    return bptr, ucol[:U], uptr[:U + 1], occ[:nnz]


def batch_epoch(row_ptr, col, val, y, w, lr, loss=LOGISTIC, mode=MATCHED, B=100, order=None):
    """One epoch of mini-batch gradient descent on a copy of w.  order: None =
    batches 0..nb-1 (the sequential computation), else the batch sequence."""
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    val = None if val is None else _c(val, np.float32)
    y = _c(y, np.float32)
    w = np.array(w, dtype=np.float32, copy=True)
    n = len(row_ptr) - 1
    if order is not None:
        order = _c(order, np.int32)
        cnt = len(order)
    else:
        cnt = n_batches(n, B)
    if _load().orc_batch_apply(n, cnt, _ptr(order), _ptr(row_ptr), _ptr(col), _ptr(val), _ptr(y),
                               _ptr(w), np.float32(lr), loss, mode, B) != 0:
        raise MemoryError
    return w


def _stale(fn, row_ptr, col, val, y, w, d, lr, loss, mode, delay):
    row_ptr = _c(row_ptr, np.int64)
    col = _c(col, np.int32)
    val = None if val is None else _c(val, np.float32)
    y = _c(y, np.float32)
    w = np.array(w, dtype=np.float32, copy=True)
    n = len(row_ptr) - 1
    if fn(n, d, _ptr(row_ptr), _ptr(col), _ptr(val), _ptr(y), _ptr(w), np.float32(lr), loss, mode,
          int(delay)) != 0:
        raise MemoryError
    return w


def stale_epoch(row_ptr, col, val, y, w, lr, loss=LOGISTIC, mode=MATCHED, delay=0):
    """One epoch of delay-stale SGD (per-entry written values)."""
    return _stale(_load().orc_stale_apply, row_ptr, col, val, y, w, len(w), lr, loss, mode, delay)


def stale_snapshot(row_ptr, col, val, y, w, lr, loss=LOGISTIC, mode=MATCHED, delay=0):
    """The same from full weight snapshots after every example (tiny inputs)."""
    return _stale(_load().orc_stale_snapshot, row_ptr, col, val, y, w, len(w), lr, loss, mode, delay)


def dense_gd(X, y, w, lr, loss=SQUARED, mode=MATCHED, iters=1, row_block=None, col_block=None,
             row_chunk=None):
    """Full-batch gradient descent on the rows of X (n x d, float32), iters
    iterations, on a copy of w.  Matched mode sums in the blocked order given
    by row_block, col_block and row_chunk (default: one block each way, one
    chunk per row block)."""
    X = np.asarray(X, dtype=np.float32)
    if X.ndim != 2 or X.strides[1] != 4 or X.strides[0] % 4:
        X = np.ascontiguousarray(X)
    n, d = X.shape
    ldx = X.strides[0] // 4 if n > 0 else d
    y = _c(y, np.float32)
    w = np.array(w, dtype=np.float32, copy=True)
    rb = max(n, 1) if row_block is None else int(row_block)
    cb = max(d, 1) if col_block is None else int(col_block)
    rc = rb if row_chunk is None else int(row_chunk)
    if _load().orc_dense_gd(n, d, X.ctypes.data, ldx, _ptr(y), _ptr(w), np.float32(lr), loss, mode,
                            int(iters), rb, cb, rc) != 0:
        raise ValueError("bad blocking or out of memory")
    return w
