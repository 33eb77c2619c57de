"""The C-ABI library without a GPU: it loads, exports every function
include/dd.h declares, and rejects bad arguments before touching HIP."""
import ctypes
import os

import pytest

from paper_2006_03318_amd import binding as B


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2006_03318_amd import build
        build.build()
    return B.lib()


def test_exports_every_declared_symbol(lib):
    names = B.declared_symbols()
    assert len(names) >= 11
    raw = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_status_strings(lib):
    assert [B.dd_status_str(i) for i in range(len(B.STATUS_NAMES))] == B.STATUS_NAMES
    assert B.dd_status_str(99) == "DD_UNKNOWN"


def test_argument_errors_without_device(lib):
    vp = ctypes.c_void_p
    out = vp()
    assert lib.dd_graph_load(-1, 1, None, None, None, None, None, None, None, None, None,
                             ctypes.byref(out)) == B.DD_EINVAL
    assert "n < 0" in B.dd_last_error()
    assert lib.dd_graph_load(1, 0, None, None, None, None, None, None, None, None, None,
                             ctypes.byref(out)) == B.DD_EINVAL
    assert lib.dd_graph_load(1, 1, None, None, None, None, None, None, None, None, None,
                             None) == B.DD_EINVAL
    steps = ctypes.c_int64()
    assert lib.dd_levelize(None, 1, B.DD_PHASES, None, ctypes.byref(out),
                           ctypes.byref(steps)) == B.DD_EINVAL
    assert lib.dd_apply_transforms(None, 1, 1, None, None, None, None,
                                   ctypes.byref(out)) == B.DD_EINVAL
    assert lib.dd_simulate_batch(None, None, None, None, None, None, None) == B.DD_EINVAL
    # launch shapes: 0, 1, 2, 4, 8, 16 (one workgroup per variant strip),
    # -1, -2, -4, -8 (the few-variant path); the value is checked first
    for bad in (3, -3, -16, 32, -32):
        assert lib.dd_simulate_batch_vs(None, None, None, None, None, None, bad, None) == B.DD_EINVAL
        assert "variants_per_wg" in B.dd_last_error()
    for good in (0, 1, 16, -1, -8):
        assert lib.dd_simulate_batch_vs(None, None, None, None, None, None, good, None) == B.DD_EINVAL
        assert "NULL handle" in B.dd_last_error()
    assert lib.dd_sched_task_steps(None, None, None) == B.DD_EINVAL
    assert lib.dd_sched_info(None, None, None, None, None) == B.DD_EINVAL
    # freeing NULL handles is a no-op
    lib.dd_graph_free(None)
    lib.dd_sched_free(None)
    lib.dd_variants_free(None)


def test_binding_checks_dtypes(lib):
    import numpy as np
    with pytest.raises(TypeError):
        B.dd_graph_load(1, 1, np.zeros(2, np.int32), None, None, np.zeros(1, np.int32),
                        np.zeros(1, np.int32), np.zeros(1, np.int64), np.zeros(1, np.int64),
                        None)
