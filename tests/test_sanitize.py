"""The oracle and the input generator built with AddressSanitizer and
UndefinedBehaviorSanitizer (gcc, host code only), run over every entry point
on small workloads in a child process.  Any sanitizer report fails the run,
and the sanitized builds must return the same bytes as the normal ones."""
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SANITIZE = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=all", "-ffp-contract=off", "-fno-fast-math", "-shared", "-fPIC"]

# Runs in the child (and in this process, for the reference digest): every
# oracle and generator entry point on small inputs, hashed.
SCENARIO = r'''
import hashlib
import numpy as np
import datagen, oracle

def scenario():
    h = hashlib.sha256()
    def put(*arrs):
        for a in arrs:
            h.update(np.ascontiguousarray(a).tobytes())
    for cfg, kw in ((1, dict(n=3000, d=400)), (2, dict(n=2000, d=300)), (3, dict(n=1500, d=800)),
                    (4, dict(n=1200, d=2000))):
        g = datagen.generate(cfg, **kw)
        rp, col, val, y, d = g["row_ptr"], g["col"], g["val"], g["y"], g["d"]
        put(rp, col, y)
        if val is not None:
            put(val)
        level, perm, level_ptr, L = oracle.schedule(rp, col, d)
        put(level, perm, level_ptr)
        put(oracle.levels_brute(rp[:301], col[:rp[300]])[0])
        put(oracle.prev_writer(rp, col, d), *oracle.transpose(rp, col, d))
        for mode in (oracle.NATURAL, oracle.MATCHED):
            put(oracle.sgd_epoch(rp, col, val, y, np.zeros(d, np.float32), g["lr"], g["loss"], mode))
            for B in (1, 7, 100):
                put(oracle.batch_epoch(rp, col, val, y, np.zeros(d, np.float32), g["lr"] / B,
                                       g["loss"], mode, B))
            for delay in (0, 3):
                put(oracle.stale_epoch(rp, col, val, y, np.zeros(d, np.float32), g["lr"],
                                       g["loss"], mode, delay))
        put(*oracle.batch_schedule(rp, col, d, 7)[:3])
        put(*oracle.batch_union(rp, col, d, 7))
        put(oracle.batch_levels_brute(rp[:201], col[:rp[200]], 3)[0])
        small = rp[:41]
        put(oracle.stale_snapshot(small, col[:small[-1]], None if val is None else val[:small[-1]],
                                  y[:40], np.zeros(d, np.float32), g["lr"], g["loss"],
                                  oracle.MATCHED, 2))
    m = datagen.generate_mf(5, n=5000, n_users=300, n_items=80)
    put(m["user"], m["item"], m["rating"], m["U0"], m["V0"])
    for mode in (oracle.NATURAL, oracle.MATCHED):
        put(*oracle.mf_epoch(m["user"], m["item"], m["rating"], m["U0"], m["V0"], m["lr"],
                             m["reg"], mode))
    dg = datagen.generate_dense(1, n=70, d=90, ldx=93, seed=3)
    for mode, rb, cb in ((oracle.NATURAL, None, None), (oracle.MATCHED, 9, 32)):
        put(oracle.dense_gd(dg["X"], dg["y"], np.zeros(90, np.float32), np.float32(1e-3),
                            oracle.SQUARED, mode, 3, rb, cb, 32))
    put(np.float32([oracle.exp(x) for x in (-104.0, -1.5, 0.0, 0.3, 88.0)]))
    put(np.float32([oracle.sigmoid(z) for z in (-90.0, -2.0, 0.0, 2.0, 90.0)]))
    put(datagen.philox_block([1, 2, 3, 4], [5, 6]), datagen.uniform_sample(9, 100),
        datagen.zipf_sample(9, 1000, 1.1, 100), datagen.poisson_sample(9, 80.0, 100))
    return h.hexdigest()
'''


def runtime(name):
    path = subprocess.run(["gcc", "-print-file-name=%s" % name], capture_output=True, text=True,
                          check=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("gcc has no %s" % name)
    return path


@pytest.mark.slow
def test_oracle_and_generator_under_asan_ubsan(tmp_path):
    asan, ubsan = runtime("libasan.so"), runtime("libubsan.so")
    lib_oracle = tmp_path / "liboracle_san.so"
    lib_gen = tmp_path / "libpdbgen_san.so"
    subprocess.run(["gcc", *SANITIZE, "-std=c11", "-o", str(lib_oracle),
                    os.path.join(ROOT, "oracle", "oracle.c"), "-lm"], check=True)
    subprocess.run(["gcc", *SANITIZE, "-fopenmp", "-o", str(lib_gen),
                    os.path.join(ROOT, "datagen", "gen.c"), "-lm"], check=True)
    child = tmp_path / "child.py"
    child.write_text(
        "import sys\nsys.path.insert(0, %r)\n" % ROOT + SCENARIO +
        "import oracle, datagen\n"
        "oracle._LIB_PATH = %r\ndatagen._LIB_PATH = %r\n" % (str(lib_oracle), str(lib_gen)) +
        "print(scenario())\n")
    env = dict(os.environ)
    env["LD_PRELOAD"] = "%s:%s" % (asan, ubsan)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["OMP_NUM_THREADS"] = "4"
    r = subprocess.run([sys.executable, str(child)], capture_output=True, text=True, env=env,
                       timeout=600)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    ns = {}
    exec(SCENARIO, ns)
    assert r.stdout.strip().splitlines()[-1] == ns["scenario"]()
