"""Learning-rate schedules of the paper, as multipliers of the peak rate.

Each function maps the 1-based iteration t to a factor in [0, 1]. `lambda_lr` wraps
one for torch: `LambdaLR` calls its function with the number of steps already taken,
which is t - 1.

* `linear_warmup(total, frac=0.1)`: a linear rise to the stable rate over the first
  10% of training (Sec. 5.1, training protocols), then constant. The paper names no
  decay for its GPT-2 runs.
* `wsd(warmup, stable, decay, floor=0.0)`: warmup-stable-decay. A linear rise over
  `warmup` iterations, a constant phase of `stable` iterations, then a linear fall to
  `floor` over `decay` iterations. The appendix simulation uses 500 / 3500 / 1000 with
  eta_max = 1e-3 and eta_min = 0 (Appendix B).
* `geometric(period, rho)`: rho ** floor((t - 1) / period). This is the stepped decay
  of the appendix's second setting (period 50, rho 0.5).

Reading: warm-up reaches the peak at its last iteration, so t = warmup gives 1. The
decay reaches the floor at its last iteration, so t = warmup + stable + decay gives
`floor`. Past the end the factor stays at `floor`.
"""
from __future__ import annotations

import math
from typing import Callable

Schedule = Callable[[int], float]


def linear_warmup(total: int, frac: float = 0.1) -> Schedule:
    if total < 1 or not (0.0 <= frac <= 1.0):
        raise ValueError("total >= 1 and 0 <= frac <= 1 required")
    w = int(round(frac * total))

    def f(t: int) -> float:
        if t < 1:
            raise ValueError("iterations are 1-based")
        return min(1.0, t / w) if w > 0 else 1.0
    return f


def wsd(warmup: int, stable: int, decay: int, floor: float = 0.0) -> Schedule:
    if min(warmup, stable, decay) < 0 or not (0.0 <= floor <= 1.0):
        raise ValueError("phase lengths >= 0 and 0 <= floor <= 1 required")

    def f(t: int) -> float:
        if t < 1:
            raise ValueError("iterations are 1-based")
        if t <= warmup:
            return t / warmup
        if t <= warmup + stable:
            return 1.0
        k = t - warmup - stable
        if k >= decay:
            return floor
        return floor + (1.0 - floor) * (decay - k) / decay
    return f


def geometric(period: int, rho: float) -> Schedule:
    if period < 1 or not (0.0 < rho <= 1.0):
        raise ValueError("period >= 1 and 0 < rho <= 1 required")

    def f(t: int) -> float:
        if t < 1:
            raise ValueError("iterations are 1-based")
        return rho ** math.floor((t - 1) / period)
    return f


def lambda_lr(optimizer, schedule: Schedule):
    """A torch LambdaLR that applies `schedule` to every group's rate. LambdaLR calls
    its function with the count of steps taken, so the first step uses t = 1."""
    import torch
    return torch.optim.lr_scheduler.LambdaLR(optimizer, lambda s: schedule(s + 1))
