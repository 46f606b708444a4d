"""Matrix-core ceiling of this GPU under its power budget (calibration only).

``mfma_ceiling(kind)`` runs an MFMA-only kernel (no memory traffic) on every CU
and returns the sustained bf16 rate and the shader clock. The datasheet's
2.5 PFLOP/s assumes 2.4 GHz; with random operands the power budget holds the
clock, and the rate, well below that. The bench reports this beside the
datasheet peak, which stays the roofline's ``peak``.

    python -m paper_2608_05088_amd.calib      # random, constant and zero operands
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "lib", "libmalt_calib.so")
KINDS = {"random": 0, "ones": 1, "zeros": 2}
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
    return _lib


def mfma_ceiling(kind: str = "random", iters: int = 4000) -> dict:
    """Sustained v_mfma_f32_32x32x16_bf16 rate (TFLOP/s) and clock (MHz) for
    operands of `kind` ("random": seeded N(0, 1) bf16, "ones", "zeros")."""
    tf, mhz, ms = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    rc = lib().malt_calib_mfma(KINDS[kind], int(iters), ctypes.byref(tf), ctypes.byref(mhz), ctypes.byref(ms))
    if rc != 0:
        raise RuntimeError(f"malt_calib_mfma failed ({rc})")
    return {"operands": kind, "TFLOP_per_s": round(tf.value, 1), "clock_MHz": round(mhz.value, 0),
            "ms": round(ms.value, 3)}
