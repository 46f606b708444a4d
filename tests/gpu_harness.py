"""Shared helpers of the GPU parity tests: run libmalt and the oracle on the
same seeded float32 inputs and compare stage by stage.

Tolerances (relative Frobenius error against the fp64 oracle):
  * fp32 elementwise and preconditioner state (M, l, r, nu, L, R, ||Mt||,
    alpha): 1e-5;
  * bf16 Newton-Schulz output O and the final update dW: 2e-2.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from oracle import OracleHparams, oracle_init, oracle_step, rel_fro
from paper_2608_05088_amd import libmalt as lm

TOL_STATE = 1e-5
TOL_NS = 2e-2


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def torch_dev():
    import torch
    return torch.device("cuda:0")


def to_dev(arrs: Sequence[np.ndarray]):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a)).to(torch_dev()) for a in arrs]


@dataclass
class GpuStep:
    W: List[np.ndarray]
    dW: List[np.ndarray]
    M: List[np.ndarray]
    l: List[np.ndarray]
    r: List[np.ndarray]
    nu: List[Optional[float]]
    Lv: List[np.ndarray]
    Rv: List[np.ndarray]
    O: List[np.ndarray]
    X0: List[np.ndarray]
    scal: List[Dict[str, float]]


def run_gpu(shapes, variant: str, W0: Sequence[np.ndarray], grads: Sequence[Sequence[np.ndarray]],
            hp_kw: dict, collect: Optional[Sequence[int]] = None, plan: Optional[lm.Plan] = None) -> List[GpuStep]:
    """Run len(grads) steps on the GPU; collect per-step host copies of the
    matrices in `collect` (default: all)."""
    import torch
    idx = list(range(len(shapes))) if collect is None else list(collect)
    plan = plan or lm.Plan(shapes, variant)
    hp = lm.make_hparams(**hp_kw)
    Wd = to_dev(W0)
    out = []
    for Gs in grads:
        Gd = to_dev(Gs)
        before = [Wd[i].double().cpu().numpy() for i in idx]
        plan.step(Wd, Gd, hp)
        torch.cuda.synchronize()
        st = GpuStep([], [], [], [], [], [], [], [], [], [], [])
        for k, i in enumerate(idx):
            M, l, r, nu = plan.state_views(i)
            dv = plan.debug_views(i)
            Wn = Wd[i].double().cpu().numpy()
            st.W.append(Wn)
            st.dW.append(Wn - before[k])
            st.M.append(M.double().cpu().numpy())
            st.l.append(l.double().cpu().numpy())
            st.r.append(r.double().cpu().numpy())
            st.nu.append(float(nu.item()) if nu is not None else None)
            st.Lv.append(dv["Lv"].double().cpu().numpy())
            st.Rv.append(dv["Rv"].double().cpu().numpy())
            st.O.append(dv["O"].float().double().cpu().numpy())
            st.X0.append(dv["X0"].float().double().cpu().numpy())
            st.scal.append({k2: float(v.item()) for k2, v in dv["scalars"].items()})
        out.append(st)
        del Gd
    return out


def run_sampled_against_oracle(w, steps: int, sample: Sequence[int], hp_kw: dict, label: str,
                               tol_ns: float = TOL_NS, tol_state: float = TOL_STATE) -> Dict[str, float]:
    """Step every matrix of workload `w` for `steps` steps in one plan (the
    benchmark's launch configuration) and compare the sampled matrices with the
    oracle after every step (the oracle runs in lockstep, so host memory holds
    one step at a time).  The sampled matrices get the host generator's weights
    and gradients (the oracle's inputs); the others get device-drawn ones, which
    cannot affect the sampled matrices: the step is independent per matrix."""
    import torch

    from paper_2608_05088_amd import workloads as wl
    dev = torch_dev()
    shapes = list(w.shapes)
    sample = list(sample)
    plan = lm.Plan(shapes, w.variant)
    hp = lm.make_hparams(**hp_kw)
    W0h = {i: wl.weight(w.cid, i, shapes[i]) for i in sample}
    Wd = [torch.from_numpy(W0h[i]).to(dev) if i in W0h else wl.weight_device(w.cid, i, s, dev)
          for i, s in enumerate(shapes)]
    Gd = [torch.empty(s, dtype=torch.float32, device=dev) for s in shapes]
    sub = [shapes[i] for i in sample]
    ost = oracle_init(sub, w.variant)
    ohp = OracleHparams(variant=w.variant, **hp_kw)
    Wo = [W0h[i].astype(np.float64) for i in sample]
    worst: Dict[str, float] = {}
    for t in range(1, steps + 1):
        gh = {}
        for i, s in enumerate(shapes):
            if i in W0h:
                gh[i] = wl.grad(w.cid, t, i, s, w.dist)
                Gd[i].copy_(torch.from_numpy(gh[i]))
            else:
                wl.grad_device(w.cid, t, i, s, w.dist, dev, out=Gd[i])
        before = [Wd[i].double().cpu().numpy() for i in sample]
        plan.step(Wd, Gd, hp)
        torch.cuda.synchronize()
        st = GpuStep([], [], [], [], [], [], [], [], [], [], [])
        for k, i in enumerate(sample):
            M, l, r, nu = plan.state_views(i)
            dv = plan.debug_views(i)
            st.W.append(None)
            st.dW.append(Wd[i].double().cpu().numpy() - before[k])
            st.M.append(M.double().cpu().numpy())
            st.l.append(l.double().cpu().numpy())
            st.r.append(r.double().cpu().numpy())
            st.nu.append(float(nu.item()) if nu is not None else None)
            st.Lv.append(dv["Lv"].double().cpu().numpy())
            st.Rv.append(dv["Rv"].double().cpu().numpy())
            st.O.append(dv["O"].float().double().cpu().numpy())
            st.X0.append(None)
            st.scal.append({k2: float(v.item()) for k2, v in dv["scalars"].items()})
        del before
        Wo, inter = oracle_step(Wo, [gh[i] for i in sample], ost, ohp)
        orc = {"inter": inter, "M": ost.M, "l": ost.l, "r": ost.r, "nu": list(ost.nu)}
        w_t = compare([st], [orc], w.variant, tol_ns=tol_ns, tol_state=tol_state, label=f"{label} step {t}")
        for k2, v in w_t.items():
            worst[k2] = max(worst.get(k2, 0.0), v)
        say(f"[parity] {label} step {t}: dW {w_t['dW']:.3e} O {w_t['O']:.3e} M {w_t['M']:.3e}")
        del st, inter, orc
    plan.close()
    return worst


def run_oracle(shapes, variant: str, W0, grads, hp_kw: dict, collect=None):
    """The same steps through the oracle, restricted to the matrices in `collect`."""
    idx = list(range(len(shapes))) if collect is None else list(collect)
    sub = [shapes[i] for i in idx]
    st = oracle_init(sub, variant)
    ohp = OracleHparams(variant=variant, **{k: (bool(v) if k == "precond_identity" else v)
                                            for k, v in hp_kw.items()})
    W = [np.asarray(W0[i], np.float64) for i in idx]
    res = []
    for Gs in grads:
        W, inter = oracle_step(W, [Gs[i] for i in idx], st, ohp)
        res.append({"inter": inter, "M": [m.copy() for m in st.M], "l": [x.copy() for x in st.l],
                    "r": [x.copy() for x in st.r], "nu": list(st.nu)})
    return res


def compare(gpu: List[GpuStep], orc, variant: str, tol_ns: float = TOL_NS, tol_state: float = TOL_STATE,
            label: str = "") -> Dict[str, float]:
    """Assert parity step by step; returns the worst errors seen."""
    worst: Dict[str, float] = {}

    def chk(name, err, tol, where):
        worst[name] = max(worst.get(name, 0.0), err)
        assert err <= tol, f"{label} {where}: {name} rel err {err:.3e} > {tol:.1e}"

    for t, (g, o) in enumerate(zip(gpu, orc)):
        for k in range(len(g.W)):
            it = o["inter"][k]
            where = f"step {t + 1} matrix {k}"
            chk("M", rel_fro(g.M[k], o["M"][k]), tol_state, where)
            chk("l", rel_fro(g.l[k], o["l"][k]), tol_state, where)
            chk("r", rel_fro(g.r[k], o["r"][k]), tol_state, where)
            chk("Lv", rel_fro(g.Lv[k], it.Lv), tol_state, where)
            chk("Rv", rel_fro(g.Rv[k], it.Rv), tol_state, where)
            chk("s", abs(g.scal[k]["s"] - it.s) / max(it.s, 1e-300), tol_state, where)
            if variant == "malter":
                chk("nu", abs(g.nu[k] - o["nu"][k]) / max(abs(o["nu"][k]), 1e-300), tol_state, where)
                chk("alpha", abs(g.scal[k]["alpha"] - it.alpha) / max(abs(it.alpha), 1e-300), tol_state, where)
            chk("O", rel_fro(g.O[k], it.O), tol_ns, where)
            chk("dW", rel_fro(g.dW[k], it.dW), tol_ns, where)
    return worst
