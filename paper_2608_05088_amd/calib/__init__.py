"""Matrix-core ceiling of this GPU under its power budget (calibration only).

``mfma_ceiling(kind, shape)`` runs an MFMA-only kernel (no memory traffic) on
every CU and returns the sustained bf16 rate and the shader clock. The
datasheet's 2.5 PFLOP/s assumes 2.4 GHz; with random operands the power budget
holds the clock, and the rate, below that, by an amount that depends on the
instruction. The bench reports the ceiling of the instruction its kernels
issue (16x16x32) beside the datasheet peak, which stays the roofline's
``peak``.

    python -m paper_2608_05088_amd.calib      # both shapes; random, constant and zero operands
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "lib", "libmalt_calib.so")
KINDS = {"random": 0, "ones": 1, "zeros": 2}
SHAPES = {"32x32x16": 0, "16x16x32": 1}
_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        # torch carries its own HIP runtime, the library links ROCm's: torch's
        # must reach the device first, or it finds none afterwards.
        import torch
        torch.cuda.is_available()
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} not found: build it with python -m paper_2608_05088_amd.build")
        _lib = ctypes.CDLL(LIB_PATH)
        _lib.malt_calib_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
        _lib.malt_calib_mfma.restype = ctypes.c_int
        _lib.malt_calib_mfma_shape.argtypes = [ctypes.c_int] + _lib.malt_calib_mfma.argtypes
        _lib.malt_calib_mfma_shape.restype = ctypes.c_int
    return _lib


def mfma_ceiling(kind: str = "random", shape: str = "16x16x32", iters: int = 4000) -> dict:
    """Sustained rate (TFLOP/s) and clock (MHz) of v_mfma_f32_<shape>_bf16 for
    operands of `kind` ("random": seeded N(0, 1) bf16, "ones", "zeros"), the
    fastest of three timed launches after a warm-up one."""
    tf, mhz, ms = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    rc = lib().malt_calib_mfma_shape(SHAPES[shape], KINDS[kind], int(iters), ctypes.byref(tf), ctypes.byref(mhz),
                                     ctypes.byref(ms))
    if rc != 0:
        raise RuntimeError(f"malt_calib_mfma_shape failed ({rc})")
    return {"instruction": f"v_mfma_f32_{shape}_bf16", "operands": kind, "TFLOP_per_s": round(tf.value, 1),
            "clock_MHz": round(mhz.value, 0), "ms": round(ms.value, 3)}
