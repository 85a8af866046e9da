"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Levels, perm and level_ptr must be bit-exact; weights
bitwise equal to the oracle's matched summation order and within 1e-5 of its
natural order."""
import numpy as np
import pytest

import datagen
import oracle
from pdbtest import check_mf, check_schedule, check_sgd, csr_from_rows, gpu_schedule

pytestmark = pytest.mark.gpu

METHODS = [0, 1, 2, 3, 4, 5, 6]  # auto, chain-scan, dataflow, spine, chain, walk, short


def native_mod():
    from paper_1508_00703_amd import native
    return native


def structured_cases():
    n = 300
    return {
        "single": [{3}],
        "fully_conflicting": [{0, 1 + i % 7} for i in range(n)],
        "disjoint": [{2 * i, 2 * i + 1} for i in range(n)],
        "chain": [{i, i + 1} for i in range(n)],
        "interleaved": [{i % 2} for i in range(n)],
        "empty_rows": [set() if i % 3 == 0 else {i % 5, 7} for i in range(n)],
        "wide_rows": [set(range(i % 4, 200 + i % 4, 1 + i % 3)) for i in range(40)],
        "row_64_65": [set(range(64)), set(range(64, 129)), set(range(1, 66)), set(range(200, 263))],
        "one_feature": [{0}] * 50,
    }


@pytest.mark.parametrize("name", sorted(structured_cases()))
@pytest.mark.parametrize("method", METHODS)
def test_structured_schedules(gpu, name, method):
    rows = structured_cases()[name]
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1 if len(col) else 1
    check_schedule(native_mod(), gpu, row_ptr, col, d, method)


def test_no_stored_entries(gpu):
    row_ptr = np.zeros(17, np.int64)
    col = np.zeros(0, np.int32)
    lv, _ = check_schedule(native_mod(), gpu, row_ptr, col, 5, 0)
    assert lv.L_host == 1


def test_no_examples(gpu):
    native = native_mod()
    lv, info = gpu_schedule(native, gpu, np.zeros(1, np.int64), np.zeros(0, np.int32), 4, 0)
    assert lv.L_host == 0 and int(lv.n_levels.item()) == 0


EPOCH_MODES = [1, 2]  # level by level, sync-free


@pytest.mark.parametrize("name", sorted(structured_cases()))
@pytest.mark.parametrize("loss", [0, 1])
@pytest.mark.parametrize("with_val", [True, False])
@pytest.mark.parametrize("mode", EPOCH_MODES)
def test_structured_epochs(gpu, name, loss, with_val, mode):
    native = native_mod()
    rows = structured_cases()[name]
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1 if len(col) else 1
    n = len(rows)
    rng = np.random.default_rng(len(col) + loss)
    val = rng.normal(size=len(col)).astype(np.float32) if with_val else None
    # a step size that keeps the iteration contractive (lr * |x|^2 < 1/2):
    # diverging weights would make every summation order disagree
    sq = np.bincount(np.repeat(np.arange(n), np.diff(row_ptr)),
                     weights=(val.astype(np.float64) ** 2 if with_val else np.ones(len(col))),
                     minlength=n)
    lr = np.float32(min(0.05, 0.5 / max(sq.max(), 1.0)))
    g = dict(row_ptr=row_ptr, col=col, n=n, d=d, loss=loss, lr=lr, val=val,
             y=(np.sign(rng.normal(size=n)) if loss == 0 else rng.normal(size=n)).astype(np.float32))
    lv, _ = check_schedule(native, gpu, row_ptr, col, d, 0)
    w0 = (0.1 * rng.normal(size=d)).astype(np.float32)
    check_sgd(native, gpu, g, lv, w0=w0, opt=dict(epoch_mode=mode))


SCALED = {
    1: dict(),                                  # the full 10k x 1k workload
    2: dict(n=60_000, d=6_000),
    3: dict(n=30_000, d=30_000),
    4: dict(n=30_000, d=12_000),
}


@pytest.mark.parametrize("cfg", sorted(SCALED))
@pytest.mark.parametrize("method", METHODS)
def test_config_schedules(gpu, cfg, method):
    g = datagen.generate(cfg, **SCALED[cfg])
    check_schedule(native_mod(), gpu, g["row_ptr"], g["col"], g["d"], method)


@pytest.mark.parametrize("cfg", sorted(SCALED))
@pytest.mark.parametrize("mode", [0] + EPOCH_MODES)
def test_config_epochs(gpu, cfg, mode):
    native = native_mod()
    g = datagen.generate(cfg, **SCALED[cfg])
    lv, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_sgd(native, gpu, g, lv, opt=dict(epoch_mode=mode))


@pytest.mark.parametrize("cfg", [1, 4])
def test_epoch_with_oracle_schedule(gpu, cfg):
    """The apply kernel alone, fed the oracle's grouping."""
    native = native_mod()
    g = datagen.generate(cfg, **SCALED[cfg])
    level, perm, level_ptr, L = oracle.schedule(g["row_ptr"], g["col"], g["d"])
    lv = native.Levels.from_host(level, perm, level_ptr, gpu)
    check_sgd(native, gpu, g, lv)


# (epoch_mode, mf_one_cu): auto, level by level, sync-free over the device
# and sync-free on one compute unit
MF_RUNS = [(0, -1), (1, -1), (2, 0), (2, 1)]


@pytest.mark.parametrize("mode,one_cu", MF_RUNS)
def test_mf_scaled(gpu, mode, one_cu):
    native = native_mod()
    g = datagen.generate_mf(5, n=300_000, n_users=15_000, n_items=3_000)
    lv, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_mf(native, gpu, g, lv, opt=dict(epoch_mode=mode, mf_one_cu=one_cu))


@pytest.mark.parametrize("n,nu,ni", [(1, 1, 1), (2, 1, 1), (7, 3, 2), (4097, 5, 3000),
                                     (30_001, 2_000, 700)])
def test_mf_one_cu_shapes(gpu, n, nu, ni):
    """The one-compute-unit execution on odd counts, fewer rows than the LDS
    holds (every row hot), more items than it holds (hot and cold rows in one
    rating), and a ring that wraps many times."""
    native = native_mod()
    g = datagen.generate_mf(5, n=n, n_users=nu, n_items=ni)
    lv, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    check_mf(native, gpu, g, lv, opt=dict(epoch_mode=2, mf_one_cu=1))


def test_transpose_and_prev_writer(gpu):
    import torch

    native = native_mod()
    for cfg in (1, 3):
        g = datagen.generate(cfg, **SCALED[cfg])
        csr = native.Csr.from_numpy(g["row_ptr"], g["col"], None, gpu)
        col_ptr = torch.empty(g["d"] + 1, dtype=torch.int64, device=gpu)
        csc_row = torch.empty(g["nnz"], dtype=torch.int32, device=gpu)
        native.pdb_transpose(csr, g["n"], g["d"], col_ptr, csc_row)
        ref_ptr, ref_row = oracle.transpose(g["row_ptr"], g["col"], g["d"])
        assert np.array_equal(col_ptr.cpu().numpy(), ref_ptr)
        assert np.array_equal(csc_row.cpu().numpy(), ref_row)
        prev_row = torch.empty(g["nnz"], dtype=torch.int32, device=gpu)
        prev_nz = torch.empty(g["nnz"], dtype=torch.int32, device=gpu)
        native.pdb_prev_writer(csr, g["n"], g["d"], prev_row, prev_nz)
        ref_prev = oracle.prev_writer(g["row_ptr"], g["col"], g["d"])
        pr, pn = prev_row.cpu().numpy(), prev_nz.cpu().numpy()
        assert np.array_equal(pr, ref_prev)
        has = pn >= 0
        assert np.array_equal(has, ref_prev >= 0)
        # prev_nz points at the same feature in the previous writer's row
        assert np.array_equal(g["col"][pn[has]], g["col"][has])
        rows = np.searchsorted(g["row_ptr"], pn[has], side="right") - 1
        assert np.array_equal(rows, ref_prev[has])


def test_deterministic_repeat(gpu):
    native = native_mod()
    g = datagen.generate(2, **SCALED[2])
    lv1, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 2)
    from pdbtest import gpu_sgd
    a = gpu_sgd(native, gpu, g, lv1)
    b = gpu_sgd(native, gpu, g, lv1)
    assert np.array_equal(a.view(np.int32), b.view(np.int32))


def test_bad_csr_and_arguments(gpu):
    import torch

    native = native_mod()
    ok_rows = [{0, 2}, {1}, {2, 3}]
    row_ptr, col = csr_from_rows(ok_rows)
    assert native.pdb_validate_csr(native.Csr.from_numpy(row_ptr, col, None, gpu), 3, 4) == 0
    bad = [
        (row_ptr, np.array([0, 2, 1, 2, 5], np.int32), 4),     # column out of range
        (row_ptr, np.array([2, 0, 1, 2, 3], np.int32), 4),     # unsorted in a row
        (row_ptr, np.array([0, 0, 1, 2, 3], np.int32), 4),     # duplicate in a row
        (np.array([0, 3, 2, 5], np.int64), col, 4),            # row_ptr not monotone
        (np.array([0, 2, 3, 4], np.int64), col, 4),            # row_ptr[n] != nnz
        (np.array([1, 2, 3, 5], np.int64), col, 4),            # row_ptr[0] != 0
        (row_ptr, np.array([0, 2, -1, 2, 3], np.int32), 4),    # negative column
    ]
    for rp, c, d in bad:
        assert native.pdb_validate_csr(native.Csr.from_numpy(rp, c, None, gpu), 3, d) == \
            native.PDB_ERR_BAD_CSR
    csr = native.Csr.from_numpy(row_ptr, col, None, gpu)
    lv = native.Levels(3, len(col), gpu)
    small = torch.empty(16, dtype=torch.uint8, device=gpu)
    with pytest.raises(native.PdbError) as e:
        native.pdb_schedule(csr, None, 3, 4, lv, ws=small)
    assert e.value.code == native.PDB_ERR_WORKSPACE
    with pytest.raises(native.PdbError) as e:
        native.pdb_schedule(csr, None, 3, 4, lv, method=7)
    assert e.value.code == native.PDB_ERR_INVALID_ARG
    native.pdb_schedule(csr, None, 3, 4, lv)
    w = torch.zeros(4, dtype=torch.float32, device=gpu)
    y = torch.ones(3, dtype=torch.float32, device=gpu)
    with pytest.raises(native.PdbError) as e:
        native.pdb_sgd_epoch(csr, y, 3, 4, w, 0.1, 5, lv)
    assert e.value.code == native.PDB_ERR_INVALID_ARG
    with pytest.raises(native.PdbError) as e:
        U = torch.zeros(4 * 16, device=gpu)
        native.pdb_mf_epoch(torch.zeros(3, dtype=torch.int32, device=gpu),
                            torch.zeros(3, dtype=torch.int32, device=gpu), y, 3, U, 4, U, 4, 16,
                            0.1, 0.0, lv)
    assert e.value.code == native.PDB_ERR_INVALID_ARG


@pytest.mark.parametrize("hot", [0, 5, 64, -1])
@pytest.mark.parametrize("cfg", [1, 2, 3])
@pytest.mark.parametrize("width", [1, 4, 16])
def test_width1_pipeline_hot_and_cold(gpu, cfg, hot, width):
    """Runs of narrow levels (at most `width` examples each) through the
    staged pipeline, with the LDS weight cache shrunk so that cold features
    (ring, prefetch, forwarding) appear."""
    native = native_mod()
    g = datagen.generate(cfg, **SCALED[cfg])
    lv, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    assert lv.prev_nz is not None
    check_sgd(native, gpu, g, lv, opt=dict(hot_features=hot, pipeline_width=width))


@pytest.mark.parametrize("width", [2, 4, 8])
@pytest.mark.parametrize("hot", [0, -1])
def test_pipeline_runs_of_narrow_levels(gpu, width, hot):
    """Levels of 1 to 5 examples (disjoint pairs and triples between shared
    features), with consecutive rows and without: the pipeline takes the
    examples of a run in level order, and the result is the sequential one."""
    native = native_mod()
    rng = np.random.default_rng(int(width))
    rows = []
    for b in range(150):
        base, m = 100 * b + 10, 1 + b % 5
        rows.append({0, base})                                  # width 1
        rows.append({0} | {base + 1 + j for j in range(m)})     # width 1
        rows += [{base + 1 + j, base + 50 + j} for j in range(m)]  # one level of m
        rows.append({0, base + 50, base + 50 + m - 1})          # width 1
        if b % 7 == 3:
            rows = rows[:-1] + [set()] + rows[-1:]              # an empty example (level 1)
    row_ptr, col = csr_from_rows(rows)
    n, d = len(rows), int(col.max()) + 1
    val = (0.5 * rng.normal(size=len(col))).astype(np.float32)
    g = dict(row_ptr=row_ptr, col=col, n=n, d=d, loss=0, lr=np.float32(0.05), val=val,
             y=np.sign(rng.normal(size=n)).astype(np.float32))
    lv, _ = check_schedule(native, gpu, row_ptr, col, d, 0)
    widths = set(np.diff(lv.level_ptr.cpu().numpy()[:lv.L_host + 1]).tolist())
    assert {1, 2, 3, 4, 5} <= widths
    check_sgd(native, gpu, g, lv, w0=(0.1 * rng.normal(size=d)).astype(np.float32),
              opt=dict(hot_features=hot, pipeline_width=width))


def test_plain_path_matches_pipeline(gpu):
    native = native_mod()
    g = datagen.generate(3, **SCALED[3])
    lv, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    from pdbtest import gpu_sgd
    a = gpu_sgd(native, gpu, g, lv)
    b = gpu_sgd(native, gpu, g, lv, opt=dict(pipeline=0))
    assert np.array_equal(a.view(np.int32), b.view(np.int32))


def test_pipeline_index_order_when_every_level_is_narrow(gpu):
    """Config 1 (levels 1-3 wide, level order not index order): with every
    level at most pipeline_width wide the epoch is one pipeline run over the
    rows in index order (the control block counts one run of n rows), and the
    weights are bitwise the matched oracle's; with pipeline_width 1 the same
    levels run as width-1 and narrow runs in level order, to the same bits
    (Theorem 2: both orders give every weight the same updates in the same
    order)."""
    import torch

    native = native_mod()
    g = datagen.generate(1)
    lv, _ = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    perm = lv.perm.cpu().numpy()
    assert not np.array_equal(perm, np.arange(g["n"]))      # level order is not index order
    assert 2 <= lv.max_width_host <= 4
    ref = oracle.sgd_epoch(g["row_ptr"], g["col"], g["val"], g["y"], np.zeros(g["d"], np.float32),
                           g["lr"], g["loss"], oracle.MATCHED)
    csr = native.Csr.from_numpy(g["row_ptr"], g["col"], g["val"], gpu)
    y = torch.from_numpy(g["y"]).to(gpu)
    runs = {}
    for width in (4, 1):
        w = torch.zeros(g["d"], dtype=torch.float32, device=gpu)
        ws = native.pdb_sgd_epoch(csr, y, g["n"], g["d"], w, float(g["lr"]), g["loss"], lv,
                                  opt=dict(epoch_mode=native.PDB_EPOCH_LEVELS, pipeline_width=width))
        torch.cuda.synchronize()
        assert np.array_equal(w.cpu().numpy().view(np.int32), ref.view(np.int32)), width
        # control block: examples run and runs started by the pipeline (int64 8 and 9)
        st = ws[:512].cpu().numpy().view(np.int64)
        runs[width] = (int(st[8]), int(st[9]))
    assert runs[4] == (g["n"], 1)
    assert runs[1][1] > 1


@pytest.mark.parametrize("hot", [0, 40, -1])
@pytest.mark.parametrize("with_val", [True, False])
def test_width1_pipeline_long_rows(gpu, hot, with_val):
    """A chain (feature 0 everywhere) mixing 50- and 70-entry examples: the
    pipeline stops at each example over 64 entries and resumes after it."""
    native = native_mod()
    rows = [{0} | set(range(1 + i % 11, 1 + i % 11 + (69 if i % 5 == 3 else 49)))
            for i in range(400)]
    row_ptr, col = csr_from_rows(rows)
    n, d = len(rows), int(col.max()) + 1
    rng = np.random.default_rng(9)
    val = (0.3 * rng.normal(size=len(col))).astype(np.float32) if with_val else None
    g = dict(row_ptr=row_ptr, col=col, n=n, d=d, loss=0, lr=np.float32(0.01), val=val,
             y=np.sign(rng.normal(size=n)).astype(np.float32))
    lv, _ = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert lv.L_host == n
    check_sgd(native, gpu, g, lv, w0=(0.1 * rng.normal(size=d)).astype(np.float32),
              opt=dict(hot_features=hot))


@pytest.mark.parametrize("name", ["pairs_1_before_32", "pairs_16_before_32"])
def test_summation_order_adversarial(gpu, name):
    """Rows whose dot product depends on the pairing order of the butterfly."""
    import sys, os
    sys.path.insert(0, os.path.dirname(__file__))
    from test_oracle_apply import ADVERSARIAL_LANES, adversarial_order_row
    native = native_mod()
    row_ptr, col, x, w0 = adversarial_order_row(ADVERSARIAL_LANES[name])
    g = dict(row_ptr=row_ptr, col=col, n=1, d=65, loss=1, lr=np.float32(1.0), val=x,
             y=np.zeros(1, np.float32))
    lv, _ = check_schedule(native, gpu, row_ptr, col, 65, 0)
    from pdbtest import gpu_sgd
    got = gpu_sgd(native, gpu, g, lv, w0=w0)
    assert got[64] == -1.0
    check_sgd(native, gpu, g, lv, w0=w0, tol=float("inf"))


def test_reciprocal_exhaustive(gpu):
    """The division of the logistic step equals IEEE 1/b for every binary32 b
    in [1, 2^126), the range of 1 + exp(min(-z, 87))."""
    native = native_mod()
    bad, first = native.pdb_check_reciprocal(0x3F800000, 0x7E800000, gpu)
    assert bad == 0, "first mismatch at bits %#x" % first
    with pytest.raises(native.PdbError):
        native.pdb_check_reciprocal(0x3F000000, 0x3F800000, gpu)   # below 1


@pytest.mark.parametrize("hot", [0, -1])
def test_extreme_logits(gpu, hot):
    """Logistic steps whose logits pass the exponent cap (z < -87), overflow
    exp (z > 88.7) or round the logistic value to 0 or 1, on both the plain
    path and the pipeline."""
    native = native_mod()
    zs = [-1e30, -200.0, -104.5, -88.0, -87.5, -87.0, -86.9, -30.0, -17.0, -1e-3, 0.0, 1e-3,
          17.0, 30.0, 88.8, 103.9, 104.5, 200.0, 1e30]
    # a chain through feature 0 (weight 0 throughout: x0 = 0) plus one fresh
    # feature per example carrying the logit
    rows = [{0, 1 + i} for i in range(len(zs) * 3)]
    row_ptr, col = csr_from_rows(rows)
    n, d = len(rows), len(rows) + 1
    val = np.zeros(len(col), np.float32)
    val[1::2] = 1.0
    w0 = np.zeros(d, np.float32)
    w0[1:] = np.tile(np.float32(zs), 3)
    y = np.tile(np.float32([1.0, -1.0, 1.0]), len(zs))[:n]
    g = dict(row_ptr=row_ptr, col=col, n=n, d=d, loss=0, lr=np.float32(0.5), val=val, y=y)
    lv, _ = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert lv.L_host == n
    check_sgd(native, gpu, g, lv, w0=w0, opt=dict(hot_features=hot))


@pytest.mark.parametrize("hot", [0, 3, -1])
def test_width1_pipeline_rows_with_gaps(gpu, hot):
    """A run of width-1 levels whose examples are not consecutive rows (rows
    in between sit on level 1 with fresh features), so the pipeline matches
    each entry against the preceding examples' entry ranges."""
    native = native_mod()
    rng = np.random.default_rng(21)
    rows = []
    for i in range(600):
        if i >= 10 and i % 2 == 1:
            rows.append({5000 + i})
        else:
            k = int(rng.integers(1, 40))
            rows.append({0} | set(rng.choice(np.arange(1, 300), size=k, replace=False).tolist()))
    row_ptr, col = csr_from_rows(rows)
    n, d = len(rows), int(col.max()) + 1
    val = (0.5 * rng.normal(size=len(col))).astype(np.float32)
    y = np.sign(rng.normal(size=n)).astype(np.float32)
    g = dict(row_ptr=row_ptr, col=col, n=n, d=d, loss=0, lr=np.float32(0.05), val=val, y=y)
    lv, _ = check_schedule(native, gpu, row_ptr, col, d, 0)
    widths = np.diff(lv.level_ptr.cpu().numpy()[:lv.L_host + 1])
    assert widths[0] > 1 and np.all(widths[1:] == 1) and lv.L_host > 300
    check_sgd(native, gpu, g, lv, w0=(0.1 * rng.normal(size=d)).astype(np.float32),
              opt=dict(hot_features=hot))


def test_spine_selection_and_fallback(gpu):
    """Auto takes the spine when the most frequent feature misses few rows;
    with more exceptional rows (or entries) than the solver holds, both auto
    and an explicit spine request run dataflow.  Levels are exact each time."""
    native = native_mod()
    rng = np.random.default_rng(5)
    # feature 0 in all rows but every 37th; the others chain through 1..6
    rows = [({0} if i % 37 else set()) | {1 + int(rng.integers(0, 6)), 10 + int(rng.integers(0, 500))}
            for i in range(3000)]
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1
    _, info = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert info["method_used"] in (3, 4)   # the chain check runs first
    _, info = check_schedule(native, gpu, row_ptr, col, d, 3)
    assert info["method_used"] == 3 and info["rounds"] >= 1
    # 1500 exceptional rows
    rows = [{0, 1 + i % 5} if i % 2 else {6 + i % 9} for i in range(3000)]
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1
    _, info = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert info["method_used"] == 6        # rows of at most 4 entries: the short-row walk
    _, info = check_schedule(native, gpu, row_ptr, col, d, 3)
    assert info["method_used"] == 2
    # 100 exceptional rows with 60 entries each
    rows = [{0, 1 + i % 3} if i % 30 else set(range(100 + i % 7, 160 + i % 7)) for i in range(3000)]
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1
    _, info = check_schedule(native, gpu, row_ptr, col, d, 3)
    assert info["method_used"] == 2


def test_walk_selection_windows_and_fallback(gpu):
    """Auto walks chain-like inputs (a few examples share nothing with their
    predecessor); the walk's windows of 512 rows see writers in the same
    window, the one before and further back.  A row longer than a window
    falls back to dataflow.  Levels are exact each time."""
    native = native_mod()
    rng = np.random.default_rng(3)
    n = 5000
    rows = []
    for i in range(n):
        # features 0 and 1 take turns chaining runs of 700 rows, so no one
        # feature covers all rows but a few (no spine)
        r = {(i // 700) % 2} if i % 97 else {2 + i % 5}
        r |= {10 + int(x) for x in rng.integers(0, 3000, size=rng.integers(0, 6))}
        if i % 700 == 3:
            r.add(5000)                                # a writer many windows back
        rows.append(r)
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1
    lv, info = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert info["method_used"] == 5
    lv, info = check_schedule(native, gpu, row_ptr, col, d, 5)
    assert info["method_used"] == 5
    # windows cut by entries, not rows: rows of 100 entries (163 per window)
    wide = [set(range(i % 3, i % 3 + 100)) | {1000 + i} for i in range(1200)]
    row_ptr, col = csr_from_rows(wide)
    lv, info = check_schedule(native, gpu, row_ptr, col, int(col.max()) + 1, 5)
    assert info["method_used"] == 5
    # a row of 20000 entries does not fit a window
    big = [{0, 1}, set(range(2, 20002)), {1, 3}, {3, 7}]
    row_ptr, col = csr_from_rows(big)
    lv, info = check_schedule(native, gpu, row_ptr, col, int(col.max()) + 1, 5)
    assert info["method_used"] == 2


@pytest.mark.parametrize("run_len", [700, 300])
def test_walk_few_runs(gpu, run_len):
    """Chain-like rows in runs (features 0 and 1 take turns every run_len
    rows, so no feature covers nearly all rows and the spine does not apply)
    with cold features whose previous writers lie many runs back.  With at
    most one run per 512 rows (run_len 700) auto settles the runs one after
    another over a grid; with more (run_len 300) it walks windows of rows.
    Empty rows make runs of a single row.  Levels equal the oracle's either
    way."""
    native = native_mod()
    rng = np.random.default_rng(run_len)
    n = 100_000
    rows = []
    for i in range(n):
        r = {(i // run_len) % 2}
        r |= {10 + int(x) for x in rng.integers(0, 20000, size=rng.integers(0, 6))}
        rows.append(r)
    # 20 empty rows: runs of one row each (shorter than the grid's blocks),
    # and the rows after them start runs too
    for i in range(1234, n, 4999):
        rows[i] = set()
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1
    for method in (0, 5):
        _, info = check_schedule(native, gpu, row_ptr, col, d, method)
        assert info["method_used"] == 5


@pytest.mark.parametrize("n,width", [(1, 4), (1023, 4), (1024, 4), (1025, 4), (5000, 4), (12295, 4),
                                     (40000, 4), (40000, 2), (5000, 2)])
def test_short_selection_chunks_and_fallback(gpu, n, width):
    """Rows of at most 4 entries take the short-row walk under auto: one block
    settles 64-row sub-chunks in order, a wave taking several consecutive ones
    per turn, by rounds of lane shuffles, with writers in the same sub-chunk,
    the last 256 sub-chunks (an LDS ring) and older ones (loaded a turn of
    every wave ahead; 40000 rows are 625 sub-chunks, and cold features recur
    about 16000 rows apart).  Rows of at most 2 entries take the kernel's
    two-writer form.  Hot features make long chains inside a sub-chunk;
    empty rows, ragged sub-chunks and ragged turns are included.  A row of 5
    entries falls back to dataflow."""
    native = native_mod()
    rng = np.random.default_rng(n + width)
    rows = []
    for i in range(n):
        k = int(rng.integers(0, width + 1))           # 0..width entries
        r = set()
        for _ in range(k):
            u = rng.random()
            # a hot feature (long chains), a warm one, or one of many cold ones
            r.add(0 if u < 0.08 else (1 + int(rng.integers(0, 50)) if u < 0.4
                                      else 100 + int(rng.integers(0, 20000))))
        rows.append(r)
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1 if len(col) else 1
    for method in (0, 6):
        lv, info = check_schedule(native, gpu, row_ptr, col, d, method)
        assert info["method_used"] in ((6, 4, 3) if method == 0 else (6,))
    rows[n // 2] = {0, 1, 2, 3, 4}
    row_ptr, col = csr_from_rows(rows)
    _, info = check_schedule(native, gpu, row_ptr, col, max(d, 5), 6)
    assert info["method_used"] == 2


@pytest.mark.parametrize("prefix_breaks", [True, False])
def test_chain_check_prefix(gpu, prefix_breaks):
    """The chain check reads a 65536-row prefix first.  Rows chain through
    features c_i (row i holds c_i and c_i+1 and four rarely shared ones); a
    break row drops c_i.  Breaks in every other row of the prefix only: the
    prefix decides 'not chain-like' without reading the rest, so dataflow
    runs although the whole input breaks in fewer than a quarter of its rows
    (the walk's rule); breaks in every eighth row after the prefix only: the
    full count decides, and the walk runs.  Every method is exact: levels equal the oracle's."""
    native = native_mod()
    rng = np.random.default_rng(17)
    n, prefix = 200_000, 65_536
    rows = []
    extra = rng.integers(0, 1 << 22, size=(n, 4)) + (n + 2)
    for i in range(n):
        # every other row of the prefix, or every eighth row after it
        brk = i > 0 and ((i < prefix and prefix_breaks and i % 2 == 1) or
                         (i >= prefix and not prefix_breaks and i % 8 == 1))
        r = {i + 1} | set(int(x) for x in extra[i])
        if not brk:
            r.add(i)
        rows.append(r)
    row_ptr, col = csr_from_rows(rows)
    d = int(col.max()) + 1
    _, info = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert info["method_used"] == (2 if prefix_breaks else 5)


@pytest.mark.parametrize("seed", range(3))
def test_dataflow_wave_per_example(gpu, seed):
    """Auto on long rows with wide levels (most examples share nothing with
    the one before): dataflow runs a wave per example.  Rows of 0 to 300
    entries (one, two and three 128-entry rounds), a few hot features for
    long dependence chains.  Levels exact."""
    native = native_mod()
    rng = np.random.default_rng(40 + seed)
    n, d = 4000, 200_000
    rows = []
    for i in range(n):
        k = int(rng.choice([0, 3, 20, 64, 65, 127, 128, 129, 300]))
        r = set(int(x) for x in rng.integers(50, d, size=k))
        if rng.random() < 0.05:
            r.add(int(rng.integers(0, 50)))           # hot features chain a few rows
        rows.append(r)
    row_ptr, col = csr_from_rows(rows)
    lv, info = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert info["method_used"] == 2


def test_chain_selection_and_fallback(gpu):
    """Auto takes the chain when every example conflicts with the one before
    it (levels 1..n); when one does not, auto and an explicit chain request
    both fall back.  Levels are exact each time."""
    native = native_mod()
    n = 4000
    chain = [{i, i + 1, 5000 + i % 3} for i in range(n)]   # row i shares feature i with row i-1
    row_ptr, col = csr_from_rows(chain)
    d = int(col.max()) + 1
    for method in (0, 4):
        lv, info = check_schedule(native, gpu, row_ptr, col, d, method)
        assert info["method_used"] == 4 and lv.L_host == n
    # one example (row 2500) shares nothing with row 2499
    broken = [set(r) for r in chain]
    broken[2500] = {n + 10, 5003}
    broken[2501] = {2501, 2502, 5000 + 2501 % 3}
    row_ptr, col = csr_from_rows(broken)
    d = int(col.max()) + 1
    for method in (0, 4):
        lv, info = check_schedule(native, gpu, row_ptr, col, d, method)
        assert info["method_used"] != 4 and lv.L_host < n
    # an empty row breaks the chain too
    holed = [set(r) for r in chain]
    holed[17] = set()
    row_ptr, col = csr_from_rows(holed)
    lv, info = check_schedule(native, gpu, row_ptr, col, int(col.max()) + 1, 4)
    assert info["method_used"] != 4


@pytest.mark.parametrize("seed", range(6))
def test_spine_random_exceptions(gpu, seed):
    """Spine levels where exceptional rows feed the spine and each other:
    random rows over a few features, feature 0 added to all but ~1%."""
    native = native_mod()
    rng = np.random.default_rng(100 + seed)
    n, d = 5000, 6
    rows = []
    for i in range(n):
        r = set(rng.choice(np.arange(1, d), size=int(rng.integers(0, 4)), replace=False).tolist())
        if rng.random() > 0.01:
            r.add(0)
        rows.append(r)
    row_ptr, col = csr_from_rows(rows)
    lv, info = check_schedule(native, gpu, row_ptr, col, d, 3)
    assert info["method_used"] == 3
    # exceptional rows raised the spine above its own length
    assert lv.L_host > np.bincount(col).max()


@pytest.mark.parametrize("mode,one_cu", MF_RUNS[1:])
def test_mf_structured_pairs(gpu, mode, one_cu):
    """Ratings whose neighbours share a user or an item (a wave takes two
    ratings at once only when the second does not depend on the first),
    repeated users and items, and a hot item."""
    native = native_mod()
    rng = np.random.default_rng(77)
    n, nu, ni = 2000, 40, 25
    user = rng.integers(0, nu, size=n).astype(np.int32)
    item = rng.integers(0, ni, size=n).astype(np.int32)
    user[1::7] = user[0::7][:len(user[1::7])]      # same user as the rating before
    item[2::5] = item[1::5][:len(item[2::5])]      # same item as the rating before
    item[::3] = 0                                  # a hot item
    row_ptr = np.arange(0, 2 * n + 1, 2, dtype=np.int64)
    col = np.empty(2 * n, np.int32)
    col[0::2] = user
    col[1::2] = item + nu
    g = dict(user=user, item=item, rating=rng.normal(size=n).astype(np.float32),
             U0=(0.2 * rng.normal(size=(nu, 32))).astype(np.float32),
             V0=(0.2 * rng.normal(size=(ni, 32))).astype(np.float32),
             n=n, n_users=nu, n_items=ni, rank=32, lr=np.float32(0.01), reg=np.float32(0.05))
    lv, _ = check_schedule(native, gpu, row_ptr, col, nu + ni, 0)
    check_mf(native, gpu, g, lv, opt=dict(epoch_mode=mode, mf_one_cu=one_cu))


@pytest.mark.parametrize("case,fast", [("plain", 1), ("valued", 1), ("negzero", 0),
                                       ("nan_w0", 0), ("inf_x", 0), ("huge_lr", 0),
                                       ("squares", 0)])
def test_pipeline_select_free_guard(gpu, case, fast):
    """The width-1 pipeline's select-free step runs only when the epoch's
    check shows it exact (logistic loss; w0 finite with no -0; x finite;
    n |lr| max|x| bounded): the control block records the decision, and
    where the run is finite the weights are bitwise the matched oracle's.
    A -0 in w0 on a feature read from memory would turn into +0 on the
    select-free step, so that case must take the selecting step."""
    import torch

    native = native_mod()
    rng = np.random.default_rng(31)
    n, d = 3000, 400
    # a chain through feature 0, plus three features per row from the rest
    rows = [{0} | set((1 + rng.choice(d - 1, 3, replace=False)).tolist()) for _ in range(n)]
    row_ptr, col = csr_from_rows(rows)
    val = None
    if case in ("valued", "inf_x"):
        val = (0.5 * rng.normal(size=len(col))).astype(np.float32)
        if case == "inf_x":
            val[len(col) // 2] = np.inf
    w0 = (0.1 * rng.normal(size=d)).astype(np.float32)
    if case == "negzero":
        w0[1::7] = -0.0
    if case == "nan_w0":
        w0[5] = np.nan
    lr = np.float32(1e30 if case == "huge_lr" else 0.05)
    loss = 1 if case == "squares" else 0
    y = np.sign(rng.normal(size=n)).astype(np.float32)
    g = dict(row_ptr=row_ptr, col=col, n=n, d=d, loss=loss, lr=lr, val=val, y=y)
    lv, _ = check_schedule(native, gpu, row_ptr, col, d, 0)
    assert lv.L_host == n
    csr = native.Csr.from_numpy(row_ptr, col, val, gpu)
    w = torch.from_numpy(w0.copy()).to(gpu)
    ws = native.pdb_sgd_epoch(csr, torch.from_numpy(y).to(gpu), n, d, w, float(lr), loss, lv,
                              opt=dict(epoch_mode=native.PDB_EPOCH_LEVELS))
    torch.cuda.synchronize()
    # control block: pipe_bad at byte 112, pipe_fast at byte 116
    ctrl = ws[:512].cpu().numpy().view(np.int32)
    assert ctrl[29] == fast, (case, ctrl[26:30])
    if case in ("plain", "valued", "negzero", "squares"):
        ref = oracle.sgd_epoch(row_ptr, col, val, y, w0, lr, loss, oracle.MATCHED)
        assert np.array_equal(w.cpu().numpy().view(np.int32), ref.view(np.int32))
