"""Host-side bounds check of every kernel's address ranges (no GPU).

malt_check_bounds rebuilds the work lists a plan over the given shapes would
use, padding entries of the XCD-ordered Newton-Schulz lists included, and
derives with the kernels' own address functions every byte range each kernel
can address: direct-load spans of both operands over the whole contraction,
output tiles and mirrors, partial slots, the workspace layout.  Every range
must lie inside its buffer, and the Newton-Schulz operand offsets (32-bit
buffer offsets, hardware range check off) below 4 GiB.  The check must also
be tight: with the Newton-Schulz buffers 16 bytes shorter it has to fail,
because the kernels read and write their last bytes.
"""
import os

import pytest

from paper_2608_05088_amd import libmalt as lm
from paper_2608_05088_amd import workloads as wl

CASES = {
    **{wl.WORKLOADS[c].name: list(wl.WORKLOADS[c].shapes) for c in range(1, 6)},
    "ragged": [(300, 200), (1, 257), (257, 1), (129, 513), (64, 64), (3, 1000), (513, 129), (1, 1), (250, 250)],
    "mixed_split_tall_wide": [(100, 2900), (700, 1500), (1500, 300), (64, 5000)] * 8,
    "short_sides": [(5, 5), (32, 4000), (4000, 32), (33, 600), (2, 3), (17, 70000), (31, 31)],
    "extreme_aspect": [(1, 1 << 20), (1 << 20, 2), (3, 700000)],
    "max_min_dim": [(32768, 32768)],
    "max_tall": [(1 << 20, 1792)],
    "max_wide_padded": [(2047, 1 << 19), (1792, 1 << 20)],
    "matrix_core_extremes": [(33, 1 << 20), (1 << 20, 129), (128, 128), (129, 129)],
}


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lm.LIB_PATH):
        from paper_2608_05088_amd import build
        build.build()
    return lm.lib()


@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_every_kernel_range_is_inside_its_buffer(L, name, variant):
    shapes = CASES[name]
    checked = lm.check_bounds(shapes, variant)
    # At least one check per work-list entry of every matrix.
    assert checked >= len(shapes)
    matrix_core = any(min(s) > 32 for s in shapes)
    if matrix_core:
        with pytest.raises(lm.MaltError) as ei:
            lm.check_bounds(shapes, variant, shrink_bytes=16)
        assert ei.value.status == lm.MALT_ERR_BOUNDS
        assert "ns_" in str(ei.value)
    else:
        # Only the fp32 path: no buffer-resource operands to shrink.
        assert lm.check_bounds(shapes, variant, shrink_bytes=16) == checked


def test_gpt2_large_counts_every_tile(L):
    # 144 matrices: every Gram / polynomial / update tile contributes at least
    # its operand, output and partial-slot ranges.
    w = wl.WORKLOADS[4]
    T = 1280 // 256
    sym = len(w.shapes) * T * (T + 1) // 2
    upd = sum((min(s) // 256) * (max(s) // 256) for s in w.shapes)
    assert lm.check_bounds(w.shapes) >= 3 * sym + 4 * upd


def test_rejects_bad_arguments(L):
    import ctypes
    n = ctypes.c_int64(0)
    assert L.malt_check_bounds(lm._shapes([(8, 8)]), 1, 0, -1, ctypes.byref(n)) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_check_bounds(lm._shapes([(8, 8)]), 1, 5, 0, ctypes.byref(n)) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_check_bounds(lm._shapes([(8, 8)]), 1, 0, 0, None) == lm.MALT_ERR_INVALID_ARG
    assert L.malt_check_bounds(lm._shapes([(0, 8)]), 1, 0, 0, ctypes.byref(n)) == lm.MALT_ERR_SHAPE
    assert lm.status_string(lm.MALT_ERR_BOUNDS) == "MALT_ERR_BOUNDS"
