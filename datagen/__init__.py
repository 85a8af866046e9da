"""Seeded synthetic inputs shaped like the paper's sparse SGD workloads.

Input generation only: nothing here computes any part of the method (no
levels, no gradients).  Both the GPU path and the CPU oracle consume these
arrays.  The C source (``gen.c``) draws every number from Philox4x32-10 keyed
by (seed, stream) with the row index in the counter, so results do not depend
on the number of threads.

The five workloads follow the paper's setting of one training example per SGD
iteration (Sec. 6.3) on sparse data, the case its conclusion of Sec. 6.3
singles out ("data sparsity") as the next step.  They stand in for the paper's
real data set (150,360 features x 16,087 examples, Sec. 6.3), which is not
available; the sizes and distributions are stated in ``CONFIGS``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libpdbgen.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile gen.c into libpdbgen.so (gcc, OpenMP)."""
    src = os.path.join(_HERE, "gen.c")
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-shared", "-fPIC", "-o", tmp, src, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=False)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64, u64, f64, i32 = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_int32
    lib.gen_row_ptr.argtypes = [P, P, ctypes.c_int]
    lib.gen_row_ptr.restype = i64
    lib.gen_fill.argtypes = [P, P, P, P, P, ctypes.c_int]
    lib.gen_fill.restype = ctypes.c_int
    lib.gen_mf.argtypes = [u64, i64, i64, i64, f64, f64, i32, f64, f64, P, P, P, P, P, ctypes.c_int]
    lib.gen_mf.restype = ctypes.c_int
    lib.gen_philox_block.argtypes = [P, P, P]
    lib.gen_uniform.argtypes = [u64, ctypes.c_uint32, i64, P]
    lib.gen_zipf_sample.argtypes = [u64, i64, f64, i64, P]
    lib.gen_poisson_sample.argtypes = [u64, f64, i64, P]
    lib.gen_wstar.argtypes = [u64, i64, P, ctypes.c_int]
    lib.gen_dense.argtypes = [u64, i64, i64, i64, i32, f64, P, P, ctypes.c_int]
    lib.gen_dense.restype = ctypes.c_int
    _lib = lib
    return lib


class _Params(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64), ("d", ctypes.c_int64),
        ("nnz_kind", ctypes.c_int32), ("id_kind", ctypes.c_int32),
        ("nnz_a", ctypes.c_int64), ("nnz_b", ctypes.c_int64),
        ("nnz_mean", ctypes.c_double), ("alpha", ctypes.c_double),
        ("val_kind", ctypes.c_int32), ("label_kind", ctypes.c_int32),
        ("val_s", ctypes.c_double), ("label_p", ctypes.c_double),
        ("seed", ctypes.c_uint64),
    ]


LOGISTIC, SQUARED = 0, 1


@dataclass(frozen=True)
class SparseConfig:
    name: str
    n: int
    d: int
    nnz_kind: int          # 0 fixed, 1 uniform int, 2 Poisson clipped
    nnz_a: int
    nnz_b: int
    nnz_mean: float
    id_kind: int           # 0 Zipf, 1 uniform
    alpha: float
    val_kind: int          # 0 N(0,1), 1 +-lognormal, 2 ones (binary)
    val_s: float
    label_kind: int        # 0 sign with flips, 1 linear + noise
    label_p: float
    loss: int
    lr: float


@dataclass(frozen=True)
class MFConfig:
    name: str
    n: int
    n_users: int
    n_items: int
    alpha_u: float
    alpha_i: float
    rank: int
    factor_sd: float
    noise_sd: float
    lr: float
    reg: float


CONFIGS = {
    1: SparseConfig("logreg-10k-1k-zipf1.0", 10_000, 1_000, 0, 10, 10, 0.0, 0, 1.0, 0, 0.0, 0, 0.05,
                    LOGISTIC, 0.1),
    2: SparseConfig("logreg-1m-100k-zipf1.1", 1_000_000, 100_000, 1, 20, 40, 0.0, 0, 1.1, 1, 0.5, 0,
                    0.05, LOGISTIC, 0.05),
    3: SparseConfig("logreg-10m-1m-zipf1.2-binary", 10_000_000, 1_000_000, 0, 50, 50, 0.0, 0, 1.2, 2,
                    0.0, 0, 0.10, LOGISTIC, 0.01),
    4: SparseConfig("lsq-5m-2m-uniform-poisson80", 5_000_000, 2_000_000, 2, 1, 400, 80.0, 1, 0.0, 0,
                    0.0, 1, 0.1, SQUARED, 0.001),
    5: MFConfig("mf-20m-1mx200k-r32", 20_000_000, 1_000_000, 200_000, 1.0, 1.0, 32,
                1.0 / np.sqrt(32.0), 0.5, 0.005, 0.02),
}


@dataclass(frozen=True)
class DenseConfig:
    name: str
    n: int
    d: int
    label_kind: int        # 0 sign with flips, 1 linear + noise
    label_p: float
    loss: int
    lr: float
    iters: int


# Dense full-batch gradient descent (the linear-regression experiments of
# Sec. 6.1-6.2): 960 features over 5000 examples, and the widest of
# a sweep over the number of features at 500 examples.  The step sizes keep
# the summed-gradient iteration contractive: lr times the largest eigenvalue
# of X^T X, about (sqrt(n) + sqrt(d))^2, stays near 1.
DENSE = {
    1: DenseConfig("lsq-dense-5000x960", 5000, 960, 1, 0.1, SQUARED, 1e-4, 200),
    2: DenseConfig("lsq-dense-500x1m", 500, 1_000_000, 1, 0.1, SQUARED, 1e-6, 50),
}


def seed_for(cfg_id: int) -> int:
    return 1000 + cfg_id


def _threads(nthreads):
    if nthreads:
        return int(nthreads)
    return min(16, os.cpu_count() or 1)


def generate(cfg_id: int, n: int | None = None, d: int | None = None, seed: int | None = None,
             nthreads: int | None = None, values: bool = True) -> dict:
    """CSR workload for configs 1-4 (optionally with n, d shrunk for tests).

    Returns a dict with row_ptr (int64[n+1]), col (int32[nnz]), val (float32[nnz]
    or None for binary values), y (float32[n]), n, d, nnz, loss, lr, name, seed.
    """
    cfg = CONFIGS[cfg_id]
    if not isinstance(cfg, SparseConfig):
        raise ValueError("config %d is matrix completion; use generate_mf" % cfg_id)
    lib = _load()
    n = cfg.n if n is None else int(n)
    d = cfg.d if d is None else int(d)
    seed = seed_for(cfg_id) if seed is None else int(seed)
    p = _Params(n, d, cfg.nnz_kind, cfg.id_kind, cfg.nnz_a, cfg.nnz_b, cfg.nnz_mean, cfg.alpha,
                cfg.val_kind, cfg.label_kind, cfg.val_s, cfg.label_p, seed)
    nt = _threads(nthreads)
    row_ptr = np.empty(n + 1, dtype=np.int64)
    nnz = lib.gen_row_ptr(ctypes.byref(p), row_ptr.ctypes.data, nt)
    if nnz < 0:
        raise ValueError("bad generator parameters")
    col = np.empty(nnz, dtype=np.int32)
    binary = cfg.val_kind == 2
    val = None if (binary or not values) else np.empty(nnz, dtype=np.float32)
    y = np.empty(n, dtype=np.float32)
    rc = lib.gen_fill(ctypes.byref(p), row_ptr.ctypes.data, col.ctypes.data,
                      None if val is None else val.ctypes.data, y.ctypes.data, nt)
    if rc != 0:
        raise MemoryError("generator failed")
    return dict(row_ptr=row_ptr, col=col, val=val, y=y, n=n, d=d, nnz=int(nnz), loss=cfg.loss,
                lr=np.float32(cfg.lr), name=cfg.name, seed=seed, cfg=cfg_id)


def generate_mf(cfg_id: int = 5, n: int | None = None, n_users: int | None = None,
                n_items: int | None = None, seed: int | None = None,
                nthreads: int | None = None) -> dict:
    """Matrix-completion workload: user, item (int32[n]), rating (float32[n]),
    U0 (float32[n_users, rank]), V0 (float32[n_items, rank]) and the conflict
    CSR in which rating i touches features {user_i, n_users + item_i}."""
    cfg = CONFIGS[cfg_id]
    if not isinstance(cfg, MFConfig):
        raise ValueError("config %d is not matrix completion" % cfg_id)
    lib = _load()
    n = cfg.n if n is None else int(n)
    nu = cfg.n_users if n_users is None else int(n_users)
    ni = cfg.n_items if n_items is None else int(n_items)
    seed = seed_for(cfg_id) if seed is None else int(seed)
    user = np.empty(n, dtype=np.int32)
    item = np.empty(n, dtype=np.int32)
    rating = np.empty(n, dtype=np.float32)
    U0 = np.empty((nu, cfg.rank), dtype=np.float32)
    V0 = np.empty((ni, cfg.rank), dtype=np.float32)
    rc = lib.gen_mf(seed, n, nu, ni, cfg.alpha_u, cfg.alpha_i, cfg.rank, cfg.factor_sd,
                    cfg.noise_sd, user.ctypes.data, item.ctypes.data, rating.ctypes.data,
                    U0.ctypes.data, V0.ctypes.data, _threads(nthreads))
    if rc != 0:
        raise MemoryError("generator failed")
    row_ptr = np.arange(0, 2 * n + 1, 2, dtype=np.int64)
    col = np.empty(2 * n, dtype=np.int32)
    col[0::2] = user
    col[1::2] = item + np.int32(nu)
    return dict(user=user, item=item, rating=rating, U0=U0, V0=V0, n=n, n_users=nu, n_items=ni,
                rank=cfg.rank, lr=np.float32(cfg.lr), reg=np.float32(cfg.reg), row_ptr=row_ptr,
                col=col, d=nu + ni, nnz=2 * n, name=cfg.name, seed=seed, cfg=cfg_id)


def generate_dense(cfg_id: int, n: int | None = None, d: int | None = None,
                   seed: int | None = None, loss: int | None = None, ldx: int | None = None,
                   nthreads: int | None = None) -> dict:
    """Dense workload: X (float32, n x d, row stride ldx >= d; the view of the
    first d columns), y (float32[n]), and the config's loss, lr, iters."""
    cfg = DENSE[cfg_id]
    n = cfg.n if n is None else int(n)
    d = cfg.d if d is None else int(d)
    loss = cfg.loss if loss is None else int(loss)
    ldx = d if ldx is None else int(ldx)
    if ldx < d:
        raise ValueError("row stride below the row length")
    seed = 2000 + cfg_id if seed is None else int(seed)
    label_kind, label_p = (cfg.label_kind, cfg.label_p) if loss == SQUARED else (0, 0.05)
    buf = np.zeros((n, ldx), dtype=np.float32)
    y = np.empty(n, dtype=np.float32)
    if _load().gen_dense(seed, n, d, ldx, label_kind, label_p, buf.ctypes.data, y.ctypes.data,
                         _threads(nthreads)) != 0:
        raise MemoryError("generator failed")
    return dict(X=buf[:, :d], y=y, n=n, d=d, ldx=ldx, loss=loss, lr=np.float32(cfg.lr),
                iters=cfg.iters, name=cfg.name, seed=seed)


def philox_block(ctr, key):
    lib = _load()
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    lib.gen_philox_block(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def uniform_sample(seed: int, count: int, stream: int = 97) -> np.ndarray:
    out = np.empty(count, dtype=np.float64)
    _load().gen_uniform(seed, stream, count, out.ctypes.data)
    return out


def zipf_sample(seed: int, d: int, alpha: float, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.int64)
    _load().gen_zipf_sample(seed, d, alpha, count, out.ctypes.data)
    return out


def poisson_sample(seed: int, mu: float, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.int64)
    _load().gen_poisson_sample(seed, mu, count, out.ctypes.data)
    return out


def w_init(cfg_or_d) -> np.ndarray:
    """Initial weights of the logistic / least-squares workloads: w0 = 0."""
    d = cfg_or_d["d"] if isinstance(cfg_or_d, dict) else int(cfg_or_d)
    return np.zeros(d, dtype=np.float32)
