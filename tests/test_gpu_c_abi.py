"""The C ABI used from plain C (tests/c_abi/dl_example.c, no torch): hipMalloc'd
buffers, a GDN layer stepped through three merge cycles with dl_append_step beside a
dense copy stepped with dl_eager_step, then flushed.  The example returns 0 when every
step's outputs and the flushed state agree within 1e-4 (relative Frobenius)."""

import ctypes
import os

import pytest

from gpu_harness import log

pytestmark = pytest.mark.gpu

LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "libdl_example.so")


def test_pure_c_caller_matches_eager():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB)
    lib.dl_example_run.argtypes = [ctypes.POINTER(ctypes.c_double)]
    lib.dl_example_run.restype = ctypes.c_int
    err = ctypes.c_double(-1.0)
    rc = lib.dl_example_run(ctypes.byref(err))
    log(f"pure-C ABI example: rc {rc}, max rel err DeltaLog vs eager {err.value:.2e}")
    assert rc == 0, f"dl_example_run returned {rc} (max rel err {err.value:.3e})"
    assert 0.0 <= err.value <= 1e-4
