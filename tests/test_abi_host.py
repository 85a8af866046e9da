"""Host-side checks of the C ABI (no GPU needed, no kernel launched):
the library loads, exports every function that include/pdb.h declares, the
binding names the same set, and the host-only entry points behave."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")


def declared_functions():
    """Every pdb_* function declared in include/*.h."""
    names = set()
    for f in sorted(os.listdir(INCLUDE)):
        if f.endswith(".h"):
            text = open(os.path.join(INCLUDE, f)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(pdb_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    from paper_1508_00703_amd import native

    if not os.path.exists(native.LIB_PATH):
        pytest.fail("libpdb.so is not built (run __graft_entry__.build())")
    return native.load()


def test_header_declares_the_binding_exports():
    from paper_1508_00703_amd import native

    assert declared_functions() == sorted(native.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_options_defaults_and_layout(lib, tmp_path):
    """pdb_options_init gives the documented defaults, and the binding's
    struct has the header's size and field offsets (checked by a C program
    compiled against include/pdb.h)."""
    import subprocess

    from paper_1508_00703_amd import native

    o = native.options()
    assert (o.epoch_mode, o.pipeline, o.pipeline_width, o.thin_max, o.hot_features,
            o.spin_timeout_us, o.batch_thin_max, o.batch_syncfree_blocks, o.stale_mode,
            o.dense_stream, o.mf_one_cu) == (0, 1, 4, 16, -1, 20000000, 2, 32, 0, 0, -1)
    fields = [f for f, _ in native.PdbOptions._fields_]
    src = tmp_path / "layout.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "pdb.h"\nint main(void) {\n'
                   '  printf("%zu", sizeof(pdb_options));\n'
                   + "".join('  printf(" %%zu", offsetof(pdb_options, %s));\n' % f for f in fields)
                   + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    want = [ctypes.sizeof(native.PdbOptions)] + [getattr(native.PdbOptions, f).offset
                                                 for f in fields]
    assert got == want


@pytest.mark.parametrize("field,value", [("epoch_mode", 3), ("epoch_mode", -1), ("pipeline", 2),
                                         ("pipeline_width", 0), ("thin_max", 0),
                                         ("hot_features", -2), ("spin_timeout_us", -1),
                                         ("spin_timeout_us", 10 ** 12), ("batch_thin_max", 0),
                                         ("batch_syncfree_blocks", 0), ("stale_mode", 3),
                                         ("dense_stream", 2), ("mf_one_cu", 2),
                                         ("mf_one_cu", -2)])
def test_options_out_of_range_are_rejected(lib, field, value):
    """Checked on the host before any device work: with no examples a valid
    option set returns PDB_OK without touching the device, an invalid one
    PDB_ERR_INVALID_ARG."""
    from paper_1508_00703_amd import native

    csr = native.PdbCsr(None, None, None, 0)
    lv = native.PdbLevels(None, None, None, None, None, 0, 0)
    ws = ctypes.c_void_p(0x1000)  # never dereferenced: n = 0
    good = native.options()
    assert lib.pdb_sgd_epoch(ctypes.byref(csr), None, 0, 0, None, ctypes.c_float(0.1), 0,
                             ctypes.byref(lv), ws, 4096, ctypes.byref(good), None) == native.PDB_OK
    bad = native.options()
    setattr(bad, field, value)
    assert (lib.pdb_sgd_epoch(ctypes.byref(csr), None, 0, 0, None, ctypes.c_float(0.1), 0,
                              ctypes.byref(lv), ws, 4096, ctypes.byref(bad), None)
            == native.PDB_ERR_INVALID_ARG)


def test_strerror_covers_every_status(lib):
    texts = [lib.pdb_strerror(c).decode() for c in range(0, -7, -1)]
    assert len(set(texts)) == 7 and all(texts)
    assert lib.pdb_strerror(-99)          # unknown codes still give text


def test_workspace_size_queries(lib):
    from paper_1508_00703_amd import native

    sz = ctypes.c_size_t(0)
    assert lib.pdb_epoch_workspace_bytes(0, ctypes.byref(sz)) == native.PDB_OK and sz.value >= 512
    small = sz.value
    assert lib.pdb_epoch_workspace_bytes(10 ** 6, ctypes.byref(sz)) == native.PDB_OK
    assert sz.value >= small + 8 * 10 ** 6     # one packed word per feature
    assert lib.pdb_epoch_workspace_bytes(-1, ctypes.byref(sz)) == native.PDB_ERR_INVALID_ARG
    prev = 0
    for nnz in (0, 1000, 10 ** 6, 5 * 10 ** 8):
        assert lib.pdb_schedule_workspace_bytes(10 ** 4, 10 ** 3, nnz, ctypes.byref(sz)) == 0
        assert sz.value >= prev and sz.value % 256 == 0
        prev = sz.value
    assert lib.pdb_schedule_workspace_bytes(-1, 10, 10, ctypes.byref(sz)) == native.PDB_ERR_INVALID_ARG
    assert lib.pdb_schedule_workspace_bytes(10, 10, 10, None) == native.PDB_ERR_INVALID_ARG
    assert (lib.pdb_schedule_workspace_bytes(2 ** 31, 10, 10, ctypes.byref(sz))
            == native.PDB_ERR_UNSUPPORTED)


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    from paper_1508_00703_amd import native

    monkeypatch.setattr(native, "_lib", None)
    monkeypatch.setattr(native, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        native.load()


def test_dense_plan_and_workspace(lib):
    # host-only arithmetic when the worker count is given
    from paper_1508_00703_amd import native

    rb, cb = ctypes.c_int64(0), ctypes.c_int64(0)
    sz = ctypes.c_size_t(0)
    for n, d, workers in [(5000, 960, 256), (500, 10 ** 6, 256), (37, 301, 256), (1, 1, 256),
                          (10 ** 6, 10, 256), (7, 5, 3), (0, 10, 256), (10, 0, 256)]:
        assert lib.pdb_dense_plan(n, d, workers, ctypes.byref(rb), ctypes.byref(cb)) == 0
        R = -(-max(n, 1) // rb.value)
        C = -(-max(d, 1) // cb.value)
        assert cb.value % 4 == 0 and rb.value >= 1
        assert R * C <= workers, (n, d, rb.value, cb.value)
        assert lib.pdb_dense_workspace_bytes(n, d, rb.value, cb.value, ctypes.byref(sz)) == 0
        assert sz.value >= 512 + 16 * (C * n + R * d)
    assert lib.pdb_dense_plan(5000, 960, 256, ctypes.byref(rb), ctypes.byref(cb)) == 0
    assert (rb.value, cb.value) == (209, 96)
    bad = native.PDB_ERR_INVALID_ARG
    assert lib.pdb_dense_plan(-1, 4, 8, ctypes.byref(rb), ctypes.byref(cb)) == bad
    assert lib.pdb_dense_workspace_bytes(10, 10, 4, 6, ctypes.byref(sz)) == bad   # cb % 4
    assert lib.pdb_dense_workspace_bytes(10, 10, 0, 4, ctypes.byref(sz)) == bad
    assert (lib.pdb_dense_workspace_bytes(10, 10, 5000, 4, ctypes.byref(sz))
            == native.PDB_ERR_UNSUPPORTED)
    assert (lib.pdb_dense_plan(10 ** 7, 1, 256, ctypes.byref(rb), ctypes.byref(cb))
            == native.PDB_ERR_UNSUPPORTED)
