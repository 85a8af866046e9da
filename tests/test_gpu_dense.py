"""GPU parity of dense full-batch gradient descent (pdb_dense_gd) against the
CPU oracle on the same seeded inputs: weights bitwise equal to the oracle's
matched order for the same blocking, and close to its natural order.

The natural-order bound: every iteration sums n products per gradient entry
and d per dot product in another order; each sum differs by at most
(n + d) 2^-24 times the sum of magnitudes, and the contractive iteration does
not amplify it.  The tests take 1e-4 of the largest weight (plus 1e-6)."""
import numpy as np
import pytest

import datagen
import oracle

pytestmark = pytest.mark.gpu

ROW_CHUNK = 32  # rows per fma chain of a partial gradient (the documented order)


def native_mod():
    from paper_1508_00703_amd import native
    return native


def run_gpu(native, dev, X, y, w0, lr, loss, iters, rb=0, cb=0, ws=None, opt=None):
    import torch

    Xt = torch.from_numpy(np.ascontiguousarray(X)).to(dev) if X.flags.c_contiguous or X.size == 0 \
        else None
    if Xt is None:
        # keep the caller's row stride: copy the whole buffer, then view
        base = X.base if X.base is not None else X
        off = (X.__array_interface__["data"][0] - base.__array_interface__["data"][0]) // 4
        bt = torch.from_numpy(np.ascontiguousarray(base)).to(dev).view(-1)
        Xt = bt.as_strided(X.shape, (X.strides[0] // 4, 1), off)
    yt = torch.from_numpy(np.ascontiguousarray(y, dtype=np.float32)).to(dev)
    wt = torch.from_numpy(np.array(w0, dtype=np.float32)).to(dev)
    ws = native.pdb_dense_gd(Xt, yt, wt, float(lr), loss, iters, rb, cb, ws=ws, opt=opt)
    torch.cuda.synchronize()
    assert native.pdb_workspace_status(ws) == native.PDB_OK
    return wt.cpu().numpy(), ws


def check_dense(native, dev, X, y, w0, lr, loss, iters, rb=0, cb=0, natural=True, opt=None):
    n, d = X.shape
    if rb == 0 and cb == 0:
        rb, cb = native.pdb_dense_plan(n, d)
    got, _ = run_gpu(native, dev, X, y, w0, lr, loss, iters, rb, cb, opt=opt)
    ref = oracle.dense_gd(X, y, w0, lr, loss, oracle.MATCHED, iters, rb, cb, ROW_CHUNK)
    bad = np.nonzero(got.view(np.int32) != ref.view(np.int32))[0]
    assert len(bad) == 0, "blocks %dx%d, first mismatches %s: gpu %s oracle %s" % (
        rb, cb, bad[:5], got[bad[:5]], ref[bad[:5]])
    if natural:
        nat = oracle.dense_gd(X, y, w0, lr, loss, oracle.NATURAL, iters)
        assert np.max(np.abs(got - nat), initial=0.0) <= 1e-4 * np.abs(nat).max(initial=0.0) + 1e-6
    return got


def problem(n, d, loss, seed):
    g = datagen.generate_dense(1, n=n, d=d, seed=seed, loss=loss)
    lr = np.float32(0.5 / (np.sqrt(n) + np.sqrt(d)) ** 2)
    w0 = (0.1 * np.random.default_rng(seed).normal(size=d)).astype(np.float32)
    return g["X"], g["y"], w0, lr


# (n, d, row_block, col_block); 0, 0 = the plan for this device
CASES = [
    (37, 301, 0, 0), (37, 301, 5, 16), (37, 301, 37, 304), (37, 301, 1, 64),
    (5, 4, 0, 0), (1, 1, 0, 0), (1, 1, 1, 4), (64, 3, 8, 4), (300, 1000, 0, 0),
    (300, 1000, 20, 256), (1000, 257, 70, 32), (4096, 8, 4096, 8), (3, 20000, 1, 16384),
    (2000, 40, 100, 8), (130, 64, 130, 64),
]


@pytest.mark.parametrize("n,d,rb,cb", CASES)
@pytest.mark.parametrize("loss", [oracle.SQUARED, oracle.LOGISTIC])
@pytest.mark.parametrize("iters", [1, 4])
def test_dense_blockings(gpu, n, d, rb, cb, loss, iters):
    native = native_mod()
    X, y, w0, lr = problem(n, d, loss, n + d + iters)
    check_dense(native, gpu, X, y, w0, lr, loss, iters, rb, cb)


@pytest.mark.parametrize("n,d,rb,cb", [(37, 301, 5, 16), (300, 1000, 0, 0), (200, 96, 10, 32)])
def test_streaming_equals_resident(gpu, n, d, rb, cb):
    # the same blocking with the tile kept in LDS and streamed every iteration
    native = native_mod()
    X, y, w0, lr = problem(n, d, oracle.SQUARED, 3)
    a = check_dense(native, gpu, X, y, w0, lr, oracle.SQUARED, 5, rb, cb, natural=False)
    b = check_dense(native, gpu, X, y, w0, lr, oracle.SQUARED, 5, rb, cb, natural=False,
                    opt=dict(dense_stream=1))
    assert np.array_equal(a.view(np.int32), b.view(np.int32))


@pytest.mark.parametrize("stream", [0, 1])
def test_strided_and_unaligned_rows(gpu, stream):
    # row stride not a multiple of 4, and a start one float past 16 bytes:
    # the scalar-load variants
    opt = dict(dense_stream=stream)
    native = native_mod()
    g = datagen.generate_dense(1, n=90, d=130, ldx=133, seed=7)
    X, y = g["X"], g["y"]
    lr = np.float32(0.002)
    w0 = np.zeros(130, np.float32)
    check_dense(native, gpu, X, y, w0, lr, oracle.SQUARED, 3, 9, 32, opt=opt)
    buf = np.zeros((90, 136), np.float32)
    buf[:, 1:131] = X
    check_dense(native, gpu, buf[:, 1:131], y, w0, lr, oracle.SQUARED, 3, 9, 32, opt=opt)


def test_calls_compose(gpu):
    # two calls of 3 iterations on one workspace = one call of 6
    native = native_mod()
    X, y, w0, lr = problem(120, 200, oracle.SQUARED, 9)
    rb, cb = native.pdb_dense_plan(120, 200)
    w3, ws = run_gpu(native, gpu, X, y, w0, lr, oracle.SQUARED, 3, rb, cb)
    w33, _ = run_gpu(native, gpu, X, y, w3, lr, oracle.SQUARED, 3, rb, cb, ws=ws)
    w6, _ = run_gpu(native, gpu, X, y, w0, lr, oracle.SQUARED, 6, rb, cb)
    assert np.array_equal(w33.view(np.int32), w6.view(np.int32))
    ref = oracle.dense_gd(X, y, w0, lr, oracle.SQUARED, oracle.MATCHED, 6, rb, cb, ROW_CHUNK)
    assert np.array_equal(w6.view(np.int32), ref.view(np.int32))


def test_degenerate_and_errors(gpu):
    import torch

    native = native_mod()
    X, y, w0, lr = problem(10, 12, oracle.SQUARED, 4)
    for iters in (0,):
        got, _ = run_gpu(native, gpu, X, y, w0, lr, oracle.SQUARED, iters)
        assert np.array_equal(got, w0)
    got, _ = run_gpu(native, gpu, np.zeros((0, 12), np.float32), np.zeros(0, np.float32), w0, lr,
                     oracle.SQUARED, 3)
    assert np.array_equal(got, w0)
    Xt = torch.from_numpy(X).to(gpu)
    yt = torch.from_numpy(y).to(gpu)
    wt = torch.from_numpy(w0).to(gpu)
    for kw, code in [(dict(loss=7), native.PDB_ERR_INVALID_ARG),
                     (dict(iters=-1), native.PDB_ERR_INVALID_ARG),
                     (dict(row_block=2, col_block=6), native.PDB_ERR_INVALID_ARG),
                     (dict(row_block=5000, col_block=4), native.PDB_ERR_UNSUPPORTED)]:
        args = dict(loss=oracle.SQUARED, iters=1, row_block=0, col_block=0)
        args.update(kw)
        with pytest.raises(native.PdbError) as e:
            native.pdb_dense_gd(Xt, yt, wt, float(lr), args["loss"], args["iters"],
                                args["row_block"], args["col_block"])
        assert e.value.code == code
    # more workers than compute units cannot all be resident
    Xb = torch.zeros((400, 400), dtype=torch.float32, device=gpu)
    with pytest.raises(native.PdbError) as e:
        native.pdb_dense_gd(Xb, torch.zeros(400, device=gpu), torch.zeros(400, device=gpu), 0.1,
                            oracle.SQUARED, 1, 1, 4)
    assert e.value.code == native.PDB_ERR_UNSUPPORTED
    with pytest.raises(native.PdbError) as e:
        native.pdb_dense_gd(Xt, yt, wt, float(lr), oracle.SQUARED, 1,
                            ws=native.workspace(64, gpu))
    assert e.value.code == native.PDB_ERR_WORKSPACE
    assert np.array_equal(wt.cpu().numpy(), w0)


def test_full_size_sec61(gpu):
    # 5000 examples x 960 features, the launch configuration bench.py --dense 1 times
    native = native_mod()
    g = datagen.generate_dense(1)
    rb, cb = native.pdb_dense_plan(g["n"], g["d"])
    print("5000 x 960: blocks %d x %d" % (rb, cb), flush=True)
    check_dense(native, gpu, g["X"], g["y"], np.zeros(g["d"], np.float32), g["lr"], g["loss"],
                g["iters"], rb, cb)


def test_full_size_sec62(gpu):
    # 500 examples x 1M features, the blocking bench.py --dense 2 times, two iterations
    native = native_mod()
    g = datagen.generate_dense(2)
    rb, cb = native.pdb_dense_plan(g["n"], g["d"])
    print("500 x 1M: blocks %d x %d" % (rb, cb), flush=True)
    check_dense(native, gpu, g["X"], g["y"], np.zeros(g["d"], np.float32), g["lr"], g["loss"], 2,
                rb, cb)
