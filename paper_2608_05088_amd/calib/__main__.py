"""python -m paper_2608_05088_amd.calib: the matrix-core ceiling of both bf16
MFMA shapes for random, constant and zero operands."""
from paper_2608_05088_amd.calib import KINDS, SHAPES, mfma_ceiling

for shape in SHAPES:
    for k in KINDS:
        r = mfma_ceiling(k, shape)
        print(f"{shape} {k:>7}: {r['TFLOP_per_s']:8.1f} TFLOP/s ({r['TFLOP_per_s'] / 25.0:5.1f}% of 2500) "
              f"at {r['clock_MHz']:6.0f} MHz, {r['ms']:.3f} ms", flush=True)
