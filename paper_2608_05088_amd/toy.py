"""The appendix's matrix quadratic regression: Muon and MALT through libmalt,
beside the exact-whitening preconditioned Muon the paper plots (Appendix B,
Fig. 1).

Problem (Appendix B): minimise f(X) = 1/2 ||A X B^T - C||_F^2 over X (r x r),
with n = 50 and r = 5.
  * C = U S V^T, where U and V (n x r) have orthonormal columns and S (r x r) is a
    random core scaled to unit Frobenius norm.
  * A = U R1 and B = V R2, where R1 and R2 (r x r) are random with a prescribed
    condition number. Only their singular values change with kappa.
  * The Hessian in vec(X) is (B^T B) kron (A^T A), so its condition number is
    cond(R1)^2 cond(R2)^2. Here cond(R1) = cond(R2) = kappa^(1/4).
  * X0 = 0, T = 5000 iterations.
  * Schedule: warmup-stable-decay, a linear rise to eta_max = 1e-3 over 500
    iterations, 3500 constant, then a linear fall to 0 over the last 1000.
  * f* comes from the least-squares solution. C lies in the model's range, so f*
    is 0 up to rounding.

Optimizers:
  * "muon" and "malt" step X through libmalt on the GPU: one 5 x 5 matrix,
    Algorithm 1, with L = R = I for Muon.
  * "whitened" is the paper's exact-Hessian preconditioned Muon, X <- X - eta P
    Orth(P grad Q) Q with P = (A^T A)^(-1/2) and Q = (B^T B)^(-1/2). It uses the
    exact polar factor, in float64 on the host. It is the comparison the paper
    plots, not part of the library.
  * "muon_polar" is Muon as the appendix defines it: X <- X - eta Orth(grad), the
    exact polar factor with no momentum and no grafting, in float64 on the host.
    The libmalt "muon" run is instead the library's step with L = R = I
    (Newton-Schulz, momentum 0.95, grafting).

The gradient grad f = A^T (A X B^T - C) B is formed in float64 by torch on the
device for the libmalt runs. The figure's data is not printed, so the
comparison is qualitative. The paper shows Muon slowing as kappa grows and the
whitened update barely changing.

  python -m paper_2608_05088_amd.toy [--steps 5000] [--kappas 10,100,1000,10000]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
from dataclasses import dataclass

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_05088_amd.schedules import wsd  # noqa: E402

N_DEFAULT, R_DEFAULT = 50, 5
CHECKPOINTS = (0, 100, 500, 1000, 2000, 3000, 4000, 5000)


@dataclass
class Problem:
    A: np.ndarray   # n x r
    B: np.ndarray   # n x r
    C: np.ndarray   # n x n
    kappa: float

    def f(self, X: np.ndarray) -> float:
        Rs = self.A @ X @ self.B.T - self.C
        return 0.5 * float(np.sum(Rs * Rs))

    def grad(self, X: np.ndarray) -> np.ndarray:
        return self.A.T @ (self.A @ X @ self.B.T - self.C) @ self.B

    def lstsq(self) -> np.ndarray:
        """Least-squares minimiser: X = A^+ C (B^+)^T."""
        return np.linalg.pinv(self.A) @ self.C @ np.linalg.pinv(self.B).T

    def hessian_cond(self) -> float:
        sa = np.linalg.svd(self.A, compute_uv=False)
        sb = np.linalg.svd(self.B, compute_uv=False)
        return float((sa[0] / sa[-1]) ** 2 * (sb[0] / sb[-1]) ** 2)


def _orthonormal(rng: np.random.Generator, n: int, r: int) -> np.ndarray:
    q, rr = np.linalg.qr(rng.standard_normal((n, r)))
    return q * np.sign(np.diag(rr))


def make_problem(kappa: float, n: int = N_DEFAULT, r: int = R_DEFAULT, seed: int = 0) -> Problem:
    """Every random draw (U, V, S and the rotations of R1, R2) depends on the
    seed only; kappa sets the singular values of R1 and R2, geometric from 1 to
    kappa^(-1/4)."""
    rng = np.random.default_rng(seed)
    U, V = _orthonormal(rng, n, r), _orthonormal(rng, n, r)
    S = rng.standard_normal((r, r))
    S /= np.linalg.norm(S)
    rot = [_orthonormal(rng, r, r) for _ in range(4)]
    sv = np.geomspace(1.0, kappa ** -0.25, r)
    R1 = rot[0] @ np.diag(sv) @ rot[1].T
    R2 = rot[2] @ np.diag(sv) @ rot[3].T
    return Problem(A=U @ R1, B=V @ R2, C=U @ S @ V.T, kappa=kappa)


def _inv_sqrt_psd(M: np.ndarray) -> np.ndarray:
    w, Q = np.linalg.eigh(M)
    return (Q / np.sqrt(w)) @ Q.T


def _polar(G: np.ndarray) -> np.ndarray:
    u, s, vt = np.linalg.svd(G)
    keep = s > s[0] * 1e-12 if s[0] > 0 else np.zeros_like(s, dtype=bool)
    return (u[:, keep] @ vt[keep]) if keep.any() else np.zeros_like(G)


def _run_polar(p: Problem, steps: int, P: np.ndarray, Q: np.ndarray, eta_max: float) -> dict:
    """X <- X - eta_t P Orth(P grad Q) Q with the exact polar factor, no momentum
    (host, float64)."""
    sched = wsd(steps // 10, steps - steps // 10 - steps // 5, steps // 5)
    X = np.zeros((p.A.shape[1], p.B.shape[1]))
    fstar = p.f(p.lstsq())
    gaps = {0: p.f(X) - fstar}
    for t in range(1, steps + 1):
        X = X - eta_max * sched(t) * P @ _polar(P @ p.grad(X) @ Q) @ Q
        if t in CHECKPOINTS or t == steps:
            gaps[t] = p.f(X) - fstar
    return gaps


def run_whitened(p: Problem, steps: int, eta_max: float = 1e-3) -> dict:
    """The paper's exact-whitening preconditioned Muon (host, float64)."""
    return _run_polar(p, steps, _inv_sqrt_psd(p.A.T @ p.A), _inv_sqrt_psd(p.B.T @ p.B), eta_max)


def run_polar_muon(p: Problem, steps: int, eta_max: float = 1e-3) -> dict:
    """Muon as the appendix runs it: the exact polar factor of the gradient, no
    momentum, no grafting (host, float64)."""
    r = p.A.shape[1]
    return _run_polar(p, steps, np.eye(r), np.eye(r), eta_max)


def run_libmalt(p: Problem, steps: int, variant: str, eta_max: float = 1e-3, device=None) -> dict:
    """Muon (L = R = I) or MALT on the GPU through libmalt, float32 X."""
    import torch
    from paper_2608_05088_amd import libmalt as lm
    dev = torch.device(device or "cuda:0")
    sched = wsd(steps // 10, steps - steps // 10 - steps // 5, steps // 5)
    A = torch.from_numpy(p.A).to(dev)
    B = torch.from_numpy(p.B).to(dev)
    C = torch.from_numpy(p.C).to(dev)
    r = p.A.shape[1]
    X = torch.zeros((r, r), dtype=torch.float32, device=dev)
    G = torch.empty_like(X)
    plan = lm.Plan([(r, r)], "malt", device=dev)
    fstar = p.f(p.lstsq())

    def f_of(Xd) -> float:
        Rs = A @ Xd.double() @ B.T - C
        return 0.5 * float((Rs * Rs).sum())

    gaps = {0: f_of(X) - fstar}
    for t in range(1, steps + 1):
        G.copy_(A.T @ (A @ X.double() @ B.T - C) @ B)
        hp = lm.make_hparams(lr=eta_max * sched(t), precond_identity=1 if variant == "muon" else 0)
        plan.step([X], [G], hp)
        if t in CHECKPOINTS or t == steps:
            gaps[t] = f_of(X) - fstar
    plan.close()
    return gaps


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=5000)
    ap.add_argument("--kappas", default="10,100,1000,10000")
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        raise SystemExit("a GPU is required")
    for kappa in [float(k) for k in args.kappas.split(",")]:
        p = make_problem(kappa, seed=args.seed)
        row = {"kappa": kappa, "hessian_cond": round(p.hessian_cond(), 3), "steps": args.steps}
        for name in ("muon", "malt"):
            print(f"[toy] kappa {kappa:g} {name}", file=sys.stderr, flush=True)
            row[name] = {str(k): v for k, v in run_libmalt(p, args.steps, name).items()}
        row["whitened"] = {str(k): v for k, v in run_whitened(p, args.steps).items()}
        row["muon_polar"] = {str(k): v for k, v in run_polar_muon(p, args.steps).items()}
        print(json.dumps(row), flush=True)


if __name__ == "__main__":
    main()
