"""GPU parity at the full sizes of the five workloads, in the launch
configuration bench.py times (default schedule method, default tuning):
levels, grouping and previous writers bit-exact, weights bitwise equal to the
oracle's matched order and within 1e-5 of its natural order."""
import numpy as np
import pytest

import datagen
from pdbtest import check_mf, check_schedule, check_sgd

pytestmark = pytest.mark.gpu


def native_mod():
    from paper_1508_00703_amd import native
    return native


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_full_size_sgd(gpu, cfg):
    native = native_mod()
    g = datagen.generate(cfg)
    lv, info = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    print("config %d: L=%d max width=%d method=%d rounds=%d" % (
        cfg, lv.L_host, lv.max_width_host, info["method_used"], info["rounds"]), flush=True)
    check_sgd(native, gpu, g, lv)


def test_full_size_mf(gpu):
    native = native_mod()
    g = datagen.generate_mf(5)
    lv, info = check_schedule(native, gpu, g["row_ptr"], g["col"], g["d"], 0)
    print("config 5: L=%d max width=%d" % (lv.L_host, lv.max_width_host), flush=True)
    check_mf(native, gpu, g, lv)
