"""Closed forms of one MALT / MALTER step (from the zero state) on structured
gradients, written from the update rule (Algorithms 1 and 2, Sec. 3.3
preconditioners, Sec. 3.5 grafting) without the oracle's code.  Test
infrastructure only.

Scaled partial permutation: G has at most one nonzero per row and per column,
G[i, pi(i)] = g_i for i in S.  Then l, r, L, R are entrywise, L M R has the
same pattern, X X^T and every Newton-Schulz polynomial are diagonal, and NS
maps each entry x of the normalised matrix through the scalar quintic
p(x) = a x + b x^3 + c x^5 (an odd map, so signs carry through).  Every entry
off the pattern stays exactly zero.
"""
from __future__ import annotations

import numpy as np

NS_A, NS_B, NS_C = 3.4445, -4.7750, 2.0315   # Muon's quintic (no coefficients in the paper)


def permutation_step(m: int, n: int, rows: np.ndarray, cols: np.ndarray, g: np.ndarray, variant: str,
                     lr: float, mu1: float = 0.95, mu2: float = 0.99, eps: float = 1e-8, ns_steps: int = 5,
                     ns_eps: float = 1e-7):
    """Returns (l, r, Lv, Rv, dW values at (rows, cols)) in float64."""
    g = np.asarray(g, np.float64)
    l = np.zeros(m)
    r = np.zeros(n)
    l[rows] = (1 - mu2) * g * g
    r[cols] = (1 - mu2) * g * g
    Lv, Rv = (l + eps) ** -0.125, (r + eps) ** -0.125
    mt = (1 - mu1) * g * Lv[rows] * Rv[cols]          # L M R on the pattern
    s = np.sqrt(np.sum(mt * mt))
    x = mt / (s + ns_eps)
    for _ in range(ns_steps):
        x = NS_A * x + NS_B * x ** 3 + NS_C * x ** 5
    d = Lv[rows] * x * Rv[cols]                       # D = L O R on the pattern
    graft = np.sqrt(np.sum(x * x)) / (np.sqrt(np.sum(d * d)) + eps)
    alpha = 1.0
    if variant == "malter":
        q = np.sum((Lv[rows] * g * Rv[cols]) ** 2)    # ||L G R||_F^2
        nu = (1 - mu2) * q
        alpha = np.sqrt(1 - mu2) / (1 - mu1 + eps) * s / (np.sqrt(nu) + eps)
    return l, r, Lv, Rv, -lr * alpha * graft * d


def random_permutation_pattern(m: int, n: int, k: int, seed: int):
    """k distinct rows and k distinct columns paired at random, values
    +-[0.5, 2] * 1e-2."""
    rng = np.random.default_rng(seed)
    rows = rng.choice(m, k, replace=False)
    cols = rng.choice(n, k, replace=False)
    g = rng.uniform(0.5, 2.0, k) * np.where(rng.random(k) < 0.5, -1.0, 1.0) * 1e-2
    return rows, cols, g
