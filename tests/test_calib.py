"""The matrix-core calibration library (context for the roofline, not part of
libmalt): it loads and rejects bad arguments on the CPU; on the GPU, random
operands run slower than constant ones (either MFMA shape) and every rate stays below the
datasheet figure at the measured clock."""
import ctypes
import os

import pytest

from paper_2608_05088_amd import calib


def test_calib_library_loads_and_rejects_bad_arguments():
    if not os.path.exists(calib.LIB_PATH):
        pytest.skip("libmalt_calib.so not built")
    lib = calib.lib()
    d = ctypes.c_double()
    # Argument checks return -1 before any device call.
    assert lib.malt_calib_mfma(3, 10, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d)) == -1
    assert lib.malt_calib_mfma(0, 0, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d)) == -1
    assert lib.malt_calib_mfma(0, 10, None, ctypes.byref(d), ctypes.byref(d)) == -1
    assert lib.malt_calib_mfma_shape(2, 0, 10, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d)) == -1
    assert lib.malt_calib_mfma_shape(-1, 0, 10, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d)) == -1


@pytest.mark.gpu
def test_random_operands_bound_the_matrix_cores_below_constant_ones():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    for shape in calib.SHAPES:
        r = calib.mfma_ceiling("random", shape, iters=1000)
        one = calib.mfma_ceiling("ones", shape, iters=1000)
        print(r, one)
        for x in (r, one):
            assert 500.0 < x["clock_MHz"] < 3000.0
            assert 0.0 < x["TFLOP_per_s"] <= 2500.0 * x["clock_MHz"] / 2400.0 * 1.05
        assert r["TFLOP_per_s"] < one["TFLOP_per_s"]
