"""Seeded synthetic workloads for the MALT / MALTER step.

This module only draws random numbers and names matrix shapes; it contains none
of the optimizer's arithmetic.  Both the HIP path (through the tests and the
benchmark) and the fp64 oracle consume the same float32 buffers it produces.

Shapes follow the GPT-2 modules the paper names in its preconditioner
condition-number study (attn.c_attn, attn.c_proj, mlp.c_fc, mlp.c_proj) at the
Small / Medium / Large widths of its experiments (Sec. 5.1), written
rows x cols; learning rates come from its optimal-learning-rate table and
mu1 = 0.95, mu2 = 0.99, eps = 1e-8 from its hyper-parameter table.  The
OpenWebText gradients of the paper's runs are replaced by seeded synthetic
gradients of the stated distributions.

Host generator: NumPy PCG64 seeded with SeedSequence([config_id, step, matrix]);
every matrix can be regenerated on its own, values are drawn in float64 and
rounded to float32.  Device generator (benchmark only, for speed): torch's
Philox generator on the GPU, seeded from the same triple; it draws the same
distributions but not the same numbers.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

WEIGHT_KEY = 2_000_000_001     # SeedSequence key for initial weights
ROWSCALE_KEY = 2_000_000_002   # SeedSequence key for per-row gradient scales
LOWRANK_KEY = 2_000_000_003    # SeedSequence key for the low-rank factors
GRAD_SCALE = 1e-2
WEIGHT_STD = 0.02

Shape = Tuple[int, int]


def gpt2_matrix_shapes(n_layer: int, d: int) -> List[Shape]:
    """Per transformer block: attn.c_attn (d x 3d), attn.c_proj (d x d),
    mlp.c_fc (d x 4d), mlp.c_proj (4d x d)."""
    per_layer = [(d, 3 * d), (d, d), (d, 4 * d), (4 * d, d)]
    return [s for _ in range(n_layer) for s in per_layer]


@dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    shapes: Tuple[Shape, ...]
    variant: str          # "malt" or "malter"
    lr: float
    steps: int
    dist: str             # "normal", "row_loguniform", "student_t3"
    mu1: float = 0.95
    mu2: float = 0.99
    eps: float = 1e-8

    @property
    def numel(self) -> int:
        return sum(m * n for m, n in self.shapes)


WORKLOADS = {
    1: Workload(1, "single_256x512", ((256, 512),), "malt", 1.3e-3, 3, "normal"),
    2: Workload(2, "gpt2_small", tuple(gpt2_matrix_shapes(12, 768)), "malt", 1.3e-3, 1, "normal"),
    3: Workload(3, "gpt2_medium", tuple(gpt2_matrix_shapes(24, 1024)), "malter", 9e-3, 1,
                "row_loguniform"),
    4: Workload(4, "gpt2_large", tuple(gpt2_matrix_shapes(36, 1280)), "malt", 7e-4, 10, "normal"),
    5: Workload(5, "stress_4096", tuple([(4096, 4096), (4096, 11008)] * 64), "malter", 6e-3, 1,
                "student_t3"),
}


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


def row_scales(cid: int, idx: int, rows: int) -> np.ndarray:
    """Per-row scales 10**U(-3, 0), drawn once per matrix (curvature anisotropy)."""
    return 10.0 ** _rng(cid, ROWSCALE_KEY, idx).uniform(-3.0, 0.0, size=rows)


def grad(cid: int, step: int, idx: int, shape: Shape, dist: str = "normal",
         scale: float = GRAD_SCALE) -> np.ndarray:
    """Seeded float32 gradient for (config, 1-based step, matrix index)."""
    m, n = shape
    g = _rng(cid, step, idx)
    if dist == "normal":
        x = g.standard_normal((m, n))
        x *= scale
    elif dist == "row_loguniform":
        x = g.standard_normal((m, n))
        x *= (scale * row_scales(cid, idx, m))[:, None]
    elif dist == "student_t3":
        x = g.standard_t(3.0, size=(m, n))
        x *= scale
    elif dist.startswith("lowrank"):
        x = lowrank(cid, idx, shape, dist, g)
        x *= scale
    elif dist == "zero":
        x = np.zeros((m, n))
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return x.astype(np.float32)


def lowrank(cid: int, idx: int, shape: Shape, dist: str, g: np.random.Generator) -> np.ndarray:
    """"lowrank<r>_<noise>": a rank-r matrix U V^T (factors N(0,1), drawn once per
    matrix, so successive steps share the dominant subspace, as the gradients
    of a real layer do) plus `noise` times an N(0, r) matrix drawn per step:
    the noise floor sits `noise` below the low-rank part, entry for entry."""
    m, n = shape
    r_s, noise_s = dist[len("lowrank"):].split("_")
    r, noise = int(r_s), float(noise_s)
    f = _rng(cid, LOWRANK_KEY, idx)
    u = f.standard_normal((m, r))
    v = f.standard_normal((r, n))
    x = u @ v
    x += (noise * np.sqrt(r)) * g.standard_normal((m, n))
    return x


def weight(cid: int, idx: int, shape: Shape, std: float = WEIGHT_STD) -> np.ndarray:
    """Seeded float32 initial weight ~ N(0, std^2)."""
    x = _rng(cid, WEIGHT_KEY, idx).standard_normal(shape)
    x *= std
    return x.astype(np.float32)


def _pmap(fn, items, workers: int):
    if workers <= 1 or len(items) <= 1:
        return [fn(it) for it in items]
    with ThreadPoolExecutor(max_workers=workers) as ex:
        return list(ex.map(fn, items))


def grads_for(w: Workload, step: int, indices: Optional[Sequence[int]] = None,
              workers: int = 8) -> List[np.ndarray]:
    idx = list(range(len(w.shapes))) if indices is None else list(indices)
    return _pmap(lambda i: grad(w.cid, step, i, w.shapes[i], w.dist), idx, workers)


def weights_for(w: Workload, indices: Optional[Sequence[int]] = None,
                workers: int = 8) -> List[np.ndarray]:
    idx = list(range(len(w.shapes))) if indices is None else list(indices)
    return _pmap(lambda i: weight(w.cid, i, w.shapes[i]), idx, workers)


# ----------------------------------------------------------------------------
# Device-side generator (benchmark inputs; not used for parity values).
# ----------------------------------------------------------------------------

def _torch_seed(*key: int) -> int:
    return int(np.random.SeedSequence([int(k) for k in key]).generate_state(1, np.uint64)[0]
               & 0x7FFF_FFFF_FFFF_FFFF)


def grad_device(cid: int, step: int, idx: int, shape: Shape, dist: str, device, out=None,
                scale: float = GRAD_SCALE):
    """Float32 gradient drawn on `device` with torch's generator (same
    distribution family as `grad`, different numbers)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(_torch_seed(cid, step, idx))
    m, n = shape
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=device)
    if dist == "normal":
        out.normal_(0.0, scale, generator=gen)
    elif dist == "row_loguniform":
        out.normal_(0.0, 1.0, generator=gen)
        rs = torch.from_numpy(scale * row_scales(cid, idx, m)).to(device=device, dtype=torch.float32)
        out.mul_(rs[:, None])
    elif dist == "student_t3":
        # t_3 = Z / sqrt(chi2_3 / 3), chi2_3 a sum of three squared normals.
        out.normal_(0.0, 1.0, generator=gen)
        chi = torch.zeros_like(out)
        tmp = torch.empty_like(out)
        for _ in range(3):
            tmp.normal_(0.0, 1.0, generator=gen)
            chi.addcmul_(tmp, tmp)
        out.div_(torch.sqrt(chi.div_(3.0))).mul_(scale)
    elif dist == "zero":
        out.zero_()
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return out


def weight_device(cid: int, idx: int, shape: Shape, device, out=None, std: float = WEIGHT_STD):
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(_torch_seed(cid, WEIGHT_KEY, idx))
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=device)
    out.normal_(0.0, std, generator=gen)
    return out
