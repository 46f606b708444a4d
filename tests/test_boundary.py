"""Host-side tests of the libmalt C ABI (no GPU needed).

The library must load, export every function include/libmalt.h declares, size
the state exactly as the paper's memory-complexity table says, and reject bad
arguments on the host before touching the device.
"""
import ctypes
import os
import re
from ctypes import c_size_t, c_void_p

import pytest

from paper_2608_05088_amd import libmalt as lm
from paper_2608_05088_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lm.LIB_PATH):
        from paper_2608_05088_amd import build
        build.build()
    return lm.lib()


def _header_functions():
    src = open(os.path.join(ROOT, "include", "libmalt.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(malt_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(L):
    declared = _header_functions()
    assert len(declared) >= 12
    for name in declared:
        assert hasattr(L, name), f"libmalt.so does not export {name}"
    assert sorted(lm.EXPORTED) == declared


def test_version_and_status_strings(L):
    assert "gfx950" in lm.lib().malt_version().decode()
    assert lm.status_string(lm.MALT_OK) == "MALT_OK"
    assert lm.status_string(lm.MALT_ERR_SHAPE) == "MALT_ERR_SHAPE"
    assert lm.status_string(99) == "MALT_ERR_UNKNOWN"


def test_default_hparams_match_reading(L):
    from oracle import OracleHparams
    hp = lm.hparams_default()
    o = OracleHparams()
    assert (hp.mu1, hp.mu2, hp.eps, hp.weight_decay) == (o.mu1, o.mu2, o.eps, o.weight_decay)
    assert (hp.ns_steps, hp.ns_a, hp.ns_b, hp.ns_c, hp.ns_eps) == (o.ns_steps, o.ns_a, o.ns_b, o.ns_c, o.ns_eps)
    assert hp.precond_identity == 0


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_state_size_is_paper_accounting(L, cid):
    w = workloads.WORKLOADS[cid]
    for variant in ("malt", "malter"):
        sb, wb = lm.malt_state_size(w.shapes, variant)
        vals = sum(m * n + m + n for m, n in w.shapes) + (len(w.shapes) if variant == "malter" else 0)
        assert sb == 4 * vals
        assert wb % 256 == 0 and wb > 0


def test_workspace_scales_with_ns_buffers(L):
    # bf16 NS buffers: X double-buffered + A + B' (B' as a hi/lo pair when the
    # short side is <= 128), everything padded to multiples of 256.
    sb, wb = lm.malt_state_size([(512, 1024)])
    ns = 2 * (2 * 512 * 1024 + 2 * 512 * 512)
    assert ns <= wb < ns + 4 * 1024 * 1024
    sb, wb = lm.malt_state_size([(100, 300)])
    ns = 2 * (2 * 256 * 512 + 256 * 256 + 2 * 256 * 256)
    assert ns <= wb < ns + 1024 * 1024


@pytest.mark.parametrize("shapes,code", [
    ([], lm.MALT_ERR_INVALID_ARG),
    ([(0, 5)], lm.MALT_ERR_SHAPE),
    ([(5, -1)], lm.MALT_ERR_SHAPE),
    ([(1 << 21, 2)], lm.MALT_ERR_SHAPE),
    ([(40000, 40000)], lm.MALT_ERR_SHAPE),
    ([(65536, 65536)], lm.MALT_ERR_SHAPE),
    ([(2047, 1 << 20)], lm.MALT_ERR_SHAPE),   # < 2^31 elements, 2^31 once padded to 256
])
def test_state_size_rejects_bad_shapes(L, shapes, code):
    sb, wb = c_size_t(0), c_size_t(0)
    st = L.malt_state_size(lm._shapes(shapes), len(shapes), 0, ctypes.byref(sb), ctypes.byref(wb))
    assert st == code
    assert lm.last_error()


def test_state_size_rejects_bad_variant_and_null(L):
    sb, wb = c_size_t(0), c_size_t(0)
    assert L.malt_state_size(lm._shapes([(4, 4)]), 1, 7, ctypes.byref(sb), ctypes.byref(wb)) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_state_size(None, 1, 0, ctypes.byref(sb), ctypes.byref(wb)) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_state_size(lm._shapes([(4, 4)]), 1, 0, None, ctypes.byref(wb)) == lm.MALT_ERR_INVALID_ARG


def test_init_rejects_bad_pointers_before_device_work(L):
    shapes = lm._shapes([(8, 8)])
    out = c_void_p()
    # NULL buffers, misaligned state / workspace, overlapping state and workspace.
    assert L.malt_init_state(ctypes.byref(out), shapes, 1, 0, None, c_void_p(0x10000), 0, 0, None) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_init_state(ctypes.byref(out), shapes, 1, 0, c_void_p(0x10004), c_void_p(0x100000), 0, 0, None) == lm.MALT_ERR_ALIGNMENT
    assert L.malt_init_state(ctypes.byref(out), shapes, 1, 0, c_void_p(0x10000), c_void_p(0x100010), 0, 0, None) == lm.MALT_ERR_ALIGNMENT
    assert L.malt_init_state(ctypes.byref(out), shapes, 1, 0, c_void_p(0x10000), c_void_p(0x10000), 0, 0, None) == lm.MALT_ERR_ALIAS
    assert L.malt_init_state(ctypes.byref(out), shapes, 1, 0, c_void_p(0x10000), c_void_p(0x100000), 2, 0, None) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_init_state(ctypes.byref(out), shapes, 1, 0, c_void_p(0x10000), c_void_p(0x100000), 1, -3, None) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_init_state(None, shapes, 1, 0, c_void_p(0x10000), c_void_p(0x100000), 0, 0, None) == lm.MALT_ERR_INVALID_ARG
    assert out.value is None


def test_scratch_init_rejects_before_device_work(L):
    # The static scratch holds MALT_SCRATCH_BYTES; larger workspaces, NULL or
    # misaligned state are refused on the host.
    out = c_void_p()
    big = lm._shapes([(4096, 4096)])
    assert lm.malt_state_size([(4096, 4096)])[1] > lm.MALT_SCRATCH_BYTES
    assert L.malt_init_state_scratch(ctypes.byref(out), big, 1, 0, c_void_p(0x10000), 0, 0, None) == lm.MALT_ERR_SCRATCH_SIZE
    assert "static scratch" in lm.last_error()
    small = lm._shapes([(8, 8)])
    assert L.malt_init_state_scratch(ctypes.byref(out), small, 1, 0, None, 0, 0, None) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_init_state_scratch(ctypes.byref(out), small, 1, 0, c_void_p(0x10004), 0, 0, None) == lm.MALT_ERR_ALIGNMENT
    assert L.malt_init_state_scratch(None, small, 1, 0, c_void_p(0x10000), 0, 0, None) == lm.MALT_ERR_INVALID_ARG
    assert lm.status_string(lm.MALT_ERR_SCRATCH_SIZE) == "MALT_ERR_SCRATCH_SIZE"
    assert out.value is None


def test_step_rejects_null_plan_and_bad_hparams(L):
    shapes = lm._shapes([(8, 8)])
    P = (c_void_p * 1)(c_void_p(0x1000))
    hp = lm.hparams_default()
    assert L.malt_step(None, P, P, shapes, 1, ctypes.byref(hp), None) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_plan_step(None) == -1
    L.malt_destroy_state(None)   # no-op


def test_layout_queries_reject_null(L):
    out = lm.malt_state_layout_t()
    assert L.malt_state_layout(None, 0, ctypes.byref(out)) == lm.MALT_ERR_INVALID_ARG
    dout = lm.malt_debug_layout_t()
    assert L.malt_debug_layout(None, 0, ctypes.byref(dout)) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_profile_enable(None, 1) == lm.MALT_ERR_INVALID_ARG


def test_make_hparams_rejects_unknown_names(L):
    with pytest.raises(TypeError):
        lm.make_hparams(learning_rate=1.0)
    hp = lm.make_hparams(lr=0.5, ns_steps=3)
    assert hp.lr == 0.5 and hp.ns_steps == 3


def test_product_path_does_not_import_oracle():
    pkg = os.path.join(ROOT, "paper_2608_05088_amd")
    pat = re.compile(r"^\s*(from\s+oracle\b|import\s+oracle\b|#\s*include\s*[<\"].*oracle)|"
                     r"(import_module|__import__)\(\s*[\"']oracle", re.M)
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                src = open(os.path.join(dirpath, f)).read()
                assert not pat.search(src), f"{f} reaches the oracle"
