"""ctypes binding of libmalt (the C ABI declared in include/libmalt.h).

Argument marshalling only: every step of the optimizer runs in the HIP
kernels of libmalt.so.  PyTorch is used to allocate device memory and to
supply HIP streams.  If the shared library is missing this module raises on
use; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_int32, c_int64, c_size_t, c_void_p
from typing import List, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libmalt.so")

MALT_OK = 0
MALT_ERR_INVALID_ARG = 1
MALT_ERR_SHAPE = 2
MALT_ERR_ALIGNMENT = 3
MALT_ERR_STATE_MISMATCH = 4
MALT_ERR_HIP = 5
MALT_ERR_ALIAS = 6
MALT_ERR_SCRATCH_SIZE = 7
MALT_ERR_BOUNDS = 8
MALT_SCRATCH_BYTES = 64 << 20

MALT_VARIANT_MALT = 0
MALT_VARIANT_MALTER = 1
VARIANTS = {"malt": MALT_VARIANT_MALT, "malter": MALT_VARIANT_MALTER}

NUM_PHASES = 9
PHASE_NAMES = ("momentum_rowcol", "precond_finalize", "scale_convert", "norm_scalars",
               "ns_gram", "ns_poly", "ns_update", "graft_scalars", "backmap_write")

# Order of the float64 per-matrix scalar slots (malt_debug_layout_t.scalars).
SCALAR_NAMES = ("s", "sigma", "nu", "alpha", "o2", "d2", "graft", "coef")


class malt_shape_t(ctypes.Structure):
    _fields_ = [("rows", c_int64), ("cols", c_int64)]


class malt_hparams_t(ctypes.Structure):
    _fields_ = [("lr", c_double), ("mu1", c_double), ("mu2", c_double), ("eps", c_double),
                ("weight_decay", c_double), ("ns_steps", c_int32), ("ns_a", c_double),
                ("ns_b", c_double), ("ns_c", c_double), ("ns_eps", c_double),
                ("precond_identity", c_int32)]


class malt_state_layout_t(ctypes.Structure):
    _fields_ = [("M", c_int64), ("l", c_int64), ("r", c_int64), ("nu", c_int64)]


class malt_debug_layout_t(ctypes.Structure):
    _fields_ = [("Lv", c_int64), ("Rv", c_int64), ("O", c_int64), ("X0", c_int64),
                ("scalars", c_int64), ("O_pitch", c_int64), ("O_transposed", c_int64),
                ("A", c_int64), ("B", c_int64), ("AB_pitch", c_int64), ("B_split", c_int64)]


class malt_profile_t(ctypes.Structure):
    _fields_ = [("ms", c_double * NUM_PHASES), ("launches", c_int64 * NUM_PHASES),
                ("bytes", c_double * NUM_PHASES), ("flops", c_double * NUM_PHASES)]


class MaltError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


_lib: Optional[ctypes.CDLL] = None

# (name, restype, argtypes) for every entry point of include/libmalt.h.
_SIGNATURES = [
    ("malt_hparams_default", None, [POINTER(malt_hparams_t)]),
    ("malt_state_size", c_int32, [POINTER(malt_shape_t), c_int32, c_int32, POINTER(c_size_t),
                                  POINTER(c_size_t)]),
    ("malt_init_state", c_int32, [POINTER(c_void_p), POINTER(malt_shape_t), c_int32, c_int32,
                                  c_void_p, c_void_p, c_int32, c_int64, c_void_p]),
    ("malt_init_state_scratch", c_int32, [POINTER(c_void_p), POINTER(malt_shape_t), c_int32, c_int32,
                                          c_void_p, c_int32, c_int64, c_void_p]),
    ("malt_step", c_int32, [c_void_p, POINTER(c_void_p), POINTER(c_void_p), POINTER(malt_shape_t),
                            c_int32, POINTER(malt_hparams_t), c_void_p]),
    ("malt_state_layout", c_int32, [c_void_p, c_int32, POINTER(malt_state_layout_t)]),
    ("malt_debug_layout", c_int32, [c_void_p, c_int32, POINTER(malt_debug_layout_t)]),
    ("malt_plan_step", c_int64, [c_void_p]),
    ("malt_precond_condition", c_int32, [c_void_p, c_void_p, c_void_p]),
    ("malt_check_bounds", c_int32, [POINTER(malt_shape_t), c_int32, c_int32, c_int64, POINTER(c_int64)]),
    ("malt_profile_enable", c_int32, [c_void_p, c_int32]),
    ("malt_profile_read", c_int32, [c_void_p, POINTER(malt_profile_t), c_int32]),
    ("malt_destroy_state", None, [c_void_p]),
    ("malt_status_string", c_char_p, [c_int32]),
    ("malt_last_error", c_char_p, []),
    ("malt_version", c_char_p, []),
]
EXPORTED = tuple(name for name, _, _ in _SIGNATURES)


def lib() -> ctypes.CDLL:
    """The loaded libmalt.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libmalt.so not found at {LIB_PATH}: build it with "
                               "`python -m paper_2608_05088_amd.build` (there is no CPU fallback)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, res, args in _SIGNATURES:
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_string(status: int) -> str:
    return lib().malt_status_string(status).decode()


def last_error() -> str:
    return lib().malt_last_error().decode()


def _check(status: int) -> None:
    if status != MALT_OK:
        raise MaltError(status, last_error())


def _shapes(shapes: Sequence[Tuple[int, int]]):
    arr = (malt_shape_t * max(1, len(shapes)))()
    for i, (m, n) in enumerate(shapes):
        arr[i].rows = int(m)
        arr[i].cols = int(n)
    return arr


def hparams_default() -> malt_hparams_t:
    hp = malt_hparams_t()
    lib().malt_hparams_default(ctypes.byref(hp))
    return hp


def make_hparams(**kw) -> malt_hparams_t:
    hp = hparams_default()
    for k, v in kw.items():
        if not hasattr(hp, k):
            raise TypeError(f"unknown hyper-parameter {k!r}")
        setattr(hp, k, int(v) if k in ("ns_steps", "precond_identity") else float(v))
    return hp


def malt_state_size(shapes: Sequence[Tuple[int, int]], variant: str = "malt") -> Tuple[int, int]:
    sb, wb = c_size_t(0), c_size_t(0)
    _check(lib().malt_state_size(_shapes(shapes), len(shapes), VARIANTS[variant], ctypes.byref(sb),
                                 ctypes.byref(wb)))
    return sb.value, wb.value


def check_bounds(shapes: Sequence[Tuple[int, int]], variant: str = "malt", shrink_bytes: int = 0) -> int:
    """malt_check_bounds: the number of address ranges proved in bounds for a
    plan over `shapes`; raises MaltError (MALT_ERR_BOUNDS) naming the first
    range that is not.  Host only."""
    checked = c_int64(0)
    _check(lib().malt_check_bounds(_shapes(shapes), len(shapes), VARIANTS[variant], int(shrink_bytes),
                                   ctypes.byref(checked)))
    return checked.value


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Plan:
    """A libmalt plan over torch-allocated state and workspace buffers.

    scratch=True builds the plan with malt_init_state_scratch: no workspace
    tensor is allocated, the library's static per-device scratch array serves
    instead (debug_views are then unavailable)."""

    def __init__(self, shapes: Sequence[Tuple[int, int]], variant: str = "malt", device=None,
                 stream=None, state=None, from_existing: bool = False, step: int = 0,
                 scratch: bool = False):
        import torch
        self.shapes: List[Tuple[int, int]] = [(int(m), int(n)) for m, n in shapes]
        self.variant = variant
        dev = torch.device(device if device is not None else "cuda")
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        sb, wb = malt_state_size(self.shapes, variant)
        self.state_bytes, self.workspace_bytes = sb, wb
        if state is None:
            state = torch.empty(sb, dtype=torch.uint8, device=self.device)
        elif state.numel() * state.element_size() < sb:
            raise ValueError("state buffer too small")
        self.state = state
        self.scratch = bool(scratch)
        self._c_shapes = _shapes(self.shapes)
        handle = c_void_p()
        with torch.cuda.device(self.device):   # the plan's device is current during set-up
            if self.scratch:
                self.workspace = None
                _check(lib().malt_init_state_scratch(ctypes.byref(handle), self._c_shapes, len(self.shapes),
                                                     VARIANTS[variant], c_void_p(self.state.data_ptr()),
                                                     int(from_existing), int(step),
                                                     c_void_p(_stream_handle(stream))))
            else:
                self.workspace = torch.empty(wb, dtype=torch.uint8, device=self.device)
                _check(lib().malt_init_state(ctypes.byref(handle), self._c_shapes, len(self.shapes),
                                             VARIANTS[variant], c_void_p(self.state.data_ptr()),
                                             c_void_p(self.workspace.data_ptr()), int(from_existing),
                                             int(step), c_void_p(_stream_handle(stream))))
        self._h = handle

    # -- stepping ----------------------------------------------------------------
    def step(self, params: Sequence, grads: Sequence, hp: Optional[malt_hparams_t] = None,
             stream=None) -> None:
        import torch
        n = len(self.shapes)
        if len(params) != n or len(grads) != n:
            raise ValueError(f"expected {n} params and grads")
        # The C ABI sees raw pointers: check here what it cannot (dtype,
        # layout, device, shape), so a wrong tensor fails instead of being read
        # as float32 rows.
        for i, (p, g) in enumerate(zip(params, grads)):
            for what, x in (("param", p), ("grad", g)):
                if (x.dtype != torch.float32 or not x.is_contiguous() or x.device != self.device
                        or tuple(x.shape) != self.shapes[i]):
                    raise ValueError(f"matrix {i}: {what} must be a contiguous float32 tensor of shape "
                                     f"{self.shapes[i]} on {self.device} (got {x.dtype}, {tuple(x.shape)}, "
                                     f"{x.device}, contiguous={x.is_contiguous()})")
        self._step_ptrs(params, grads, hp, stream)

    def _step_ptrs(self, params: Sequence, grads: Sequence, hp: Optional[malt_hparams_t] = None,
                   stream=None) -> None:
        """malt_step on the tensors' data pointers, without the checks of step():
        only the C library's own validation applies."""
        n = len(self.shapes)
        P = (c_void_p * n)(*[c_void_p(p.data_ptr()) for p in params])
        G = (c_void_p * n)(*[c_void_p(g.data_ptr()) for g in grads])
        hp = hp if hp is not None else hparams_default()
        _check(lib().malt_step(self._h, P, G, self._c_shapes, n, ctypes.byref(hp),
                               c_void_p(_stream_handle(stream))))

    @property
    def t(self) -> int:
        return int(lib().malt_plan_step(self._h))

    # -- views -------------------------------------------------------------------
    def state_layout(self, i: int) -> malt_state_layout_t:
        out = malt_state_layout_t()
        _check(lib().malt_state_layout(self._h, i, ctypes.byref(out)))
        return out

    def state_views(self, i: int):
        """(M, l, r, nu) torch views into the state buffer (nu is None for MALT)."""
        L = self.state_layout(i)
        m, n = self.shapes[i]
        f = self.state.view(-1)[: self.state_bytes].view(__import__("torch").float32)
        M = f[L.M: L.M + m * n].view(m, n)
        nu = f[L.nu: L.nu + 1] if L.nu >= 0 else None
        return M, f[L.l: L.l + m], f[L.r: L.r + n], nu

    def debug_layout(self, i: int) -> malt_debug_layout_t:
        out = malt_debug_layout_t()
        _check(lib().malt_debug_layout(self._h, i, ctypes.byref(out)))
        return out

    def debug_views(self, i: int) -> dict:
        """Torch views of matrix i's last-step intermediates in the workspace."""
        import torch
        if self.workspace is None:
            raise RuntimeError("debug_views need a caller workspace (this plan uses the static scratch)")
        L = self.debug_layout(i)
        m, n = self.shapes[i]
        w = self.workspace
        mc, nc = min(m, n), max(m, n)
        rows_alloc = -(-mc // 256) * 256

        def bf16(off):
            canon = w[off: off + 2 * rows_alloc * L.O_pitch].view(torch.bfloat16).view(
                rows_alloc, L.O_pitch)[:mc, :nc]
            return canon.t() if L.O_transposed else canon

        sc = w[L.scalars: L.scalars + 8 * 16].view(torch.float64)
        views = {"Lv": w[L.Lv: L.Lv + 4 * m].view(torch.float32),
                 "Rv": w[L.Rv: L.Rv + 4 * n].view(torch.float32),
                 "O": bf16(L.O), "X0": bf16(L.X0),
                 "scalars": {k: sc[j] for j, k in enumerate(SCALAR_NAMES)}}
        if L.AB_pitch:   # bf16 Newton-Schulz path: the last iteration's A and B' (padded)
            p = L.AB_pitch
            views["A"] = w[L.A: L.A + 2 * p * p].view(torch.bfloat16).view(p, p)
            bw = 2 * p if L.B_split else p
            b = w[L.B: L.B + 2 * p * bw].view(torch.bfloat16).view(p, bw)
            views["B"] = b[:, :p]
            if L.B_split:
                views["B_lo"] = b[:, p:]
        return views

    def precond_condition(self, stream=None):
        """malt_precond_condition: an (n, 2) float64 device tensor of
        (kappa(diag l), kappa(diag r)) per matrix, enqueued on the stream."""
        import torch
        out = torch.empty((len(self.shapes), 2), dtype=torch.float64, device=self.device)
        _check(lib().malt_precond_condition(self._h, c_void_p(out.data_ptr()),
                                            c_void_p(_stream_handle(stream))))
        return out

    # -- profiling ---------------------------------------------------------------
    def profile_enable(self, enable: bool = True) -> None:
        _check(lib().malt_profile_enable(self._h, int(enable)))

    def profile_read(self, reset: bool = True) -> dict:
        out = malt_profile_t()
        _check(lib().malt_profile_read(self._h, ctypes.byref(out), int(reset)))
        return {name: {"ms": out.ms[k], "launches": int(out.launches[k]), "bytes": out.bytes[k],
                       "flops": out.flops[k]} for k, name in enumerate(PHASE_NAMES)}

    def close(self) -> None:
        if getattr(self, "_h", None):
            lib().malt_destroy_state(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
