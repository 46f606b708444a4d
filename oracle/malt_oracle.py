"""Reference oracle for the MALT / MALTER matrix-optimizer step (fp64, NumPy).

TEST INFRASTRUCTURE ONLY.  This module is a plain, slow, deliberately literal
CPU implementation of the update rule of "MALT: Lightweight Curvature-Aware
Muon via Diagonal Preconditioning".  Only the test-suite, the package smoke
check and the CPU-baseline leg of the benchmark may import it.  The product
path (the HIP library and its Python binding) never imports, links or calls
anything in this directory, and this module imports nothing from the product.

Every function works in float64 on inputs upcast from the float32 buffers that
the GPU path also consumes.  There is no blocking, fusion or reordering beyond
what the paper's algorithms state; NumPy matmul and SVD are used as library
primitives only.

Sources, by the paper's own numbering:
  * Algorithm 1 (MALT update) and Algorithm 2 (MALTER update);
  * Sec. 3.1, Eq. (2): Muon's update and the definition Orth(X) = U V^T from the
    reduced SVD, approximated in practice by Newton-Schulz iterations;
  * Sec. 3.3, Eq. (dp_preconditioner) / (two_sided_diagonal_preconditioner):
    the row/column EMAs and the (l+eps)^(-1/8) diagonal factors;
  * Sec. 3.5 (norm grafting; displayed equation for alpha_t);
  * Table "memory_complexity" (state sizes mn, mn+m+n, mn+m+n+1).

Readings taken where the paper is silent or inconsistent (all configurable):
  * Newton-Schulz coefficients / step count / normalisation are not given in
    the paper.  We use the quintic published with Muon (the method the paper
    builds on and cites): p(x) = a x + b x^3 + c x^5 with
    (a, b, c) = (3.4445, -4.7750, 2.0315), 5 iterations, input divided by
    (||X||_F + 1e-7), iterating on the orientation with rows <= cols.
  * Algorithm 2 writes eta inside alpha_t and again in the parameter update;
    the displayed equation for alpha_t (Sec. 3.5) has no eta, and we follow it:
    W <- W - eta * alpha_t * ||O||/(||D||+eps) * D.
  * nu_t uses the current L_t, R_t (after this step's l, r update).
  * The bias-correction index t is 1-based (t = 1 on the first step).
  * One eps everywhere it is written: (l+eps), ||D||+eps, 1-mu1^t+eps,
    sqrt(nu)+eps.
  * No Nesterov momentum; M_t itself is preconditioned and orthogonalised.
  * Decoupled weight decay (listed in the hyper-parameter table but absent
    from both algorithms) is optional: W <- (1 - eta*lambda) W before the
    update (the decoupled rule of AdamW, which the paper cites); lambda = 0
    by default.  Pinned to torch's AdamW on zero gradients and by its
    separation from the update (P14).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

# Muon's published quintic Newton-Schulz coefficients and defaults
# (reading for Sec. 3.1 "approximately computed using Newton-Schulz").
NS_A = 3.4445
NS_B = -4.7750
NS_C = 2.0315
NS_STEPS = 5
NS_EPS = 1e-7

VARIANT_MALT = "malt"
VARIANT_MALTER = "malter"


@dataclass
class OracleHparams:
    """Hyper-parameters of Algorithms 1 and 2 (eta, mu1, mu2, eps) plus the
    Newton-Schulz reading and the optional decoupled weight decay."""

    variant: str = VARIANT_MALT
    lr: float = 1.3e-3          # eta
    mu1: float = 0.95           # momentum EMA (table "additional_settings")
    mu2: float = 0.99           # row/col EMA and nu EMA
    eps: float = 1e-8           # damping constant
    weight_decay: float = 0.0   # lambda (not part of Algorithms 1/2)
    ns_steps: int = NS_STEPS
    ns_a: float = NS_A
    ns_b: float = NS_B
    ns_c: float = NS_C
    ns_eps: float = NS_EPS
    precond_identity: bool = False   # L = R = I: the step reduces to Muon
    orth: str = "ns"                 # "ns" (Newton-Schulz) or "svd" (exact Orth)


@dataclass
class OracleState:
    """Per-matrix optimizer state of Algorithms 1/2: M (m x n), l (m), r (n),
    nu (scalar, MALTER only), and the shared step counter t."""

    shapes: List[Tuple[int, int]]
    variant: str
    M: List[np.ndarray] = field(default_factory=list)
    l: List[np.ndarray] = field(default_factory=list)
    r: List[np.ndarray] = field(default_factory=list)
    nu: List[float] = field(default_factory=list)
    t: int = 0

    def num_state_values(self) -> int:
        """Number of stored optimizer-state scalars (Table memory_complexity):
        mn + m + n per matrix for MALT, plus one (nu) for MALTER."""
        total = 0
        for i in range(len(self.shapes)):
            total += self.M[i].size + self.l[i].size + self.r[i].size
            if self.variant == VARIANT_MALTER:
                total += 1
        return total


def oracle_init(shapes: Sequence[Tuple[int, int]], variant: str = VARIANT_MALT) -> OracleState:
    """Zero initialisation of M, l, r (and nu) as in the INITIALIZE line of
    Algorithms 1 and 2."""
    st = OracleState(shapes=[(int(m), int(n)) for m, n in shapes], variant=variant)
    for m, n in st.shapes:
        st.M.append(np.zeros((m, n), dtype=np.float64))
        st.l.append(np.zeros(m, dtype=np.float64))
        st.r.append(np.zeros(n, dtype=np.float64))
        st.nu.append(0.0)
    return st


def newton_schulz(X: np.ndarray, steps: int = NS_STEPS, a: float = NS_A, b: float = NS_B,
                  c: float = NS_C, eps: float = NS_EPS) -> np.ndarray:
    """Newton-Schulz approximation of Orth(X) (Sec. 3.1), Muon's quintic.

    X is normalised by its Frobenius norm (+eps), then each iteration forms
    A = X X^T, B = b A + c A A and X <- a X + B X, on the orientation with
    rows <= cols (transposed in and out for tall inputs).  Every singular value
    sigma of the normalised input is mapped by p(x) = a x + b x^3 + c x^5 once
    per iteration; singular vectors are unchanged.
    """
    X = np.asarray(X, dtype=np.float64)
    tall = X.shape[0] > X.shape[1]
    if tall:
        X = X.T
    X = X / (np.linalg.norm(X) + eps)
    for _ in range(steps):
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    if tall:
        X = X.T
    return X


def polar_svd(X: np.ndarray, rank_tol: float = 1e-12) -> np.ndarray:
    """Exact Orth(X) = U V^T from the reduced SVD (Sec. 3.1), singular values
    below rank_tol * sigma_max mapped to zero (they have no direction)."""
    X = np.asarray(X, dtype=np.float64)
    U, S, Vt = np.linalg.svd(X, full_matrices=False)
    if S.size == 0 or S[0] == 0.0:
        return np.zeros_like(X)
    keep = S > rank_tol * S[0]
    return (U[:, keep]) @ Vt[keep, :]


@dataclass
class StepIntermediates:
    """Per-matrix intermediates of one step, for stage-by-stage comparison."""

    Lv: np.ndarray          # diagonal of L_t
    Rv: np.ndarray          # diagonal of R_t
    M_tilde: np.ndarray     # L_t M_t R_t
    s: float                # ||M_tilde||_F
    O: np.ndarray           # Orth(M_tilde) (Newton-Schulz or exact)
    D: np.ndarray           # L_t O_t R_t
    graft: float            # ||O||_F / (||D||_F + eps)
    alpha: float            # MALTER stepsize (1 for MALT)
    nu: float               # MALTER nu_t (0 for MALT)
    dW: np.ndarray          # W_t - W_{t-1}


def oracle_step(W_list: Sequence[np.ndarray], G_list: Sequence[np.ndarray], state: OracleState,
                hp: OracleHparams) -> Tuple[List[np.ndarray], List[StepIntermediates]]:
    """One MALT (Algorithm 1) or MALTER (Algorithm 2) step over a list of
    matrices.  Mutates `state` (M, l, r, nu, t); returns the new parameters
    (float64) and the per-matrix intermediates."""
    if len(W_list) != len(state.shapes) or len(G_list) != len(state.shapes):
        raise ValueError("matrix count does not match the state")
    state.t += 1
    t = state.t
    mu1, mu2, eps = hp.mu1, hp.mu2, hp.eps
    W_out: List[np.ndarray] = []
    inter: List[StepIntermediates] = []
    for i, (m, n) in enumerate(state.shapes):
        W = np.asarray(W_list[i], dtype=np.float64)
        G = np.asarray(G_list[i], dtype=np.float64)
        if W.shape != (m, n) or G.shape != (m, n):
            raise ValueError(f"matrix {i}: shape mismatch")
        # Momentum EMA (Alg. 1/2, momentum line).
        state.M[i] = mu1 * state.M[i] + (1.0 - mu1) * G
        M = state.M[i]
        # Row / column squared-norm EMAs (Eq. dp_preconditioner).
        G2 = G * G
        state.l[i] = mu2 * state.l[i] + (1.0 - mu2) * G2.sum(axis=1)
        state.r[i] = mu2 * state.r[i] + (1.0 - mu2) * G2.sum(axis=0)
        # Diagonal preconditioners L = Diag((l+eps)^(-1/8)), R likewise.
        if hp.precond_identity:
            Lv = np.ones(m)
            Rv = np.ones(n)
        else:
            Lv = (state.l[i] + eps) ** (-1.0 / 8.0)
            Rv = (state.r[i] + eps) ** (-1.0 / 8.0)
        # Two-sided scaling M_tilde = L M R.
        M_tilde = Lv[:, None] * M * Rv[None, :]
        s = float(np.linalg.norm(M_tilde))
        # Orthogonalisation.
        if hp.orth == "svd":
            O = polar_svd(M_tilde)
        else:
            O = newton_schulz(M_tilde, hp.ns_steps, hp.ns_a, hp.ns_b, hp.ns_c, hp.ns_eps)
        # Map back D = L O R and graft the norm of O.
        D = Lv[:, None] * O * Rv[None, :]
        graft = float(np.linalg.norm(O)) / (float(np.linalg.norm(D)) + eps)
        # MALTER noise-adaptive scalar (Alg. 2; displayed equation for alpha_t).
        if state.variant == VARIANT_MALTER:
            P = Lv[:, None] * G * Rv[None, :]
            state.nu[i] = mu2 * state.nu[i] + (1.0 - mu2) * float(np.sum(P * P))
            alpha = (np.sqrt(1.0 - mu2 ** t) / (1.0 - mu1 ** t + eps)) * (s / (np.sqrt(state.nu[i]) + eps))
        else:
            alpha = 1.0
        # Parameter update (optional decoupled weight decay first).
        W_new = W - hp.lr * hp.weight_decay * W
        W_new = W_new - hp.lr * alpha * graft * D
        W_out.append(W_new)
        inter.append(StepIntermediates(Lv=Lv, Rv=Rv, M_tilde=M_tilde, s=s, O=O, D=D, graft=graft,
                                       alpha=float(alpha), nu=float(state.nu[i]), dW=W_new - W))
    return W_out, inter


def rel_fro(x: np.ndarray, ref: np.ndarray) -> float:
    """Relative Frobenius error ||x - ref|| / ||ref|| (0 when both are 0)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.linalg.norm(ref))
    num = float(np.linalg.norm(x - ref))
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den
