"""torch.optim adapter: MALT / MALTER for matrix parameters through libmalt,
AdamW for every other parameter.

Algorithm 1 (MALT) and Algorithm 2 (MALTER) update matrix parameters; the
paper trains embeddings, norms and biases with AdamW.  This optimizer routes
every 2-D parameter (or those `matrix_filter` selects) of a parameter group
into one libmalt plan per group, so one `step()` is one grouped `malt_step`
per group, and hands the remaining parameters to an inner `torch.optim.AdamW`.

Variants:
  "malt"    Algorithm 1
  "malter"  Algorithm 2 (noise-adaptive stepsize)
  "muon"    Algorithm 1 with L = R = I: Muon's update (Sec. 3.1), the
            baseline the paper compares against

Conventions
  * Matrix parameters must be contiguous float32 CUDA tensors; their
    gradients are made contiguous float32 before the step.  A matrix
    parameter without a gradient is stepped with a zero gradient (the plan
    steps all of its matrices together).
  * `lr` is the matrix learning rate eta; schedulers that change a group's
    "lr" scale the group's AdamW learning rate by the same factor.
  * `state_dict()` holds each plan's state buffer (M, l, r, nu as float32)
    and step count t, and the inner AdamW's state; `load_state_dict` resumes
    bitwise.
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional, Tuple

import torch

from . import libmalt as lm

VARIANTS = ("malt", "malter", "muon")


def is_matrix(p: torch.Tensor) -> bool:
    """Default selection of matrix parameters: every 2-D tensor."""
    return p.dim() == 2


class MALT(torch.optim.Optimizer):
    def __init__(self, params, lr: float = 1.3e-3, mu1: float = 0.95, mu2: float = 0.99, eps: float = 1e-8,
                 weight_decay: float = 0.0, variant: str = "malt", ns_steps: int = 5,
                 adamw_lr: Optional[float] = None, adamw_betas=(0.9, 0.95), adamw_eps: float = 1e-8,
                 adamw_weight_decay: float = 0.0,
                 matrix_filter: Optional[Callable[[torch.Tensor], bool]] = None):
        if variant not in VARIANTS:
            raise ValueError(f"variant must be one of {VARIANTS}")
        defaults = dict(lr=lr, mu1=mu1, mu2=mu2, eps=eps, weight_decay=weight_decay, ns_steps=ns_steps,
                        adamw_lr=lr if adamw_lr is None else adamw_lr, adamw_betas=tuple(adamw_betas),
                        adamw_eps=adamw_eps, adamw_weight_decay=adamw_weight_decay)
        super().__init__(params, defaults)
        self.variant = variant
        self._filter = matrix_filter or is_matrix
        self._plans: List[Optional[lm.Plan]] = [None] * len(self.param_groups)
        self._resume: List[Optional[dict]] = [None] * len(self.param_groups)
        # Split each group into matrix parameters (libmalt) and the rest (AdamW).
        self._mats: List[List[torch.Tensor]] = []
        adam_groups = []
        for g in self.param_groups:
            mats = [p for p in g["params"] if self._filter(p)]
            rest = [p for p in g["params"] if not self._filter(p)]
            for p in mats:
                if p.dim() != 2:
                    raise ValueError("matrix_filter selected a parameter that is not 2-D")
            self._mats.append(mats)
            g["lr0"] = g["lr"]
            adam_groups.append(dict(params=rest, lr=g["adamw_lr"], betas=g["adamw_betas"], eps=g["adamw_eps"],
                                    weight_decay=g["adamw_weight_decay"]))
        self._adam_lr0 = [ag["lr"] for ag in adam_groups]
        self._adam = torch.optim.AdamW(adam_groups) if any(ag["params"] for ag in adam_groups) else None

    # ------------------------------------------------------------------ helpers
    def _hparams(self, g: dict):
        return lm.make_hparams(lr=g["lr"], mu1=g["mu1"], mu2=g["mu2"], eps=g["eps"],
                               weight_decay=g["weight_decay"], ns_steps=g["ns_steps"],
                               precond_identity=1 if self.variant == "muon" else 0)

    def _plan(self, k: int) -> Optional[lm.Plan]:
        mats = self._mats[k]
        if not mats:
            return None
        if self._plans[k] is None:
            for p in mats:
                if not (p.is_cuda and p.dtype == torch.float32 and p.is_contiguous()):
                    raise ValueError("matrix parameters must be contiguous float32 CUDA tensors")
            shapes = [tuple(p.shape) for p in mats]
            variant = "malter" if self.variant == "malter" else "malt"
            res = self._resume[k]
            if res is not None:
                state = res["state"].to(mats[0].device)
                self._plans[k] = lm.Plan(shapes, variant, device=mats[0].device, state=state,
                                         from_existing=True, step=int(res["t"]))
                self._resume[k] = None
            else:
                self._plans[k] = lm.Plan(shapes, variant, device=mats[0].device)
        return self._plans[k]

    # --------------------------------------------------------------------- step
    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        stream = torch.cuda.current_stream()
        for k, g in enumerate(self.param_groups):
            plan = self._plan(k)
            if plan is None:
                continue
            grads = []
            for p in self._mats[k]:
                gr = p.grad
                if gr is None:
                    gr = torch.zeros_like(p)
                elif gr.dtype != torch.float32 or not gr.is_contiguous():
                    gr = gr.float().contiguous()
                grads.append(gr)
            plan.step(self._mats[k], grads, self._hparams(g), stream=stream)
        if self._adam is not None:
            for k, g in enumerate(self.param_groups):   # follow the group's schedule
                self._adam.param_groups[k]["lr"] = self._adam_lr0[k] * (g["lr"] / g["lr0"]) if g["lr0"] else 0.0
            self._adam.step()
        return loss

    def zero_grad(self, set_to_none: bool = True):
        super().zero_grad(set_to_none=set_to_none)

    # ---------------------------------------------------------------- state I/O
    def state_dict(self) -> Dict:
        plans = []
        for k in range(len(self.param_groups)):
            p = self._plans[k]
            if p is None:
                plans.append(self._resume[k])
            else:
                torch.cuda.current_stream().synchronize()
                plans.append({"state": p.state[: p.state_bytes].detach().cpu().clone(), "t": p.t,
                              "shapes": list(p.shapes), "variant": self.variant})
        groups = [{k: v for k, v in g.items() if k != "params"} for g in self.param_groups]
        return {"variant": self.variant, "plans": plans, "groups": groups,
                "adamw": self._adam.state_dict() if self._adam is not None else None}

    def load_state_dict(self, sd: Dict) -> None:
        if sd["variant"] != self.variant:
            raise ValueError(f"state is for variant {sd['variant']}, optimizer is {self.variant}")
        if len(sd["plans"]) != len(self.param_groups):
            raise ValueError("parameter group count differs")
        for k, pl in enumerate(sd["plans"]):
            if pl is not None and [tuple(s) for s in pl["shapes"]] != [tuple(p.shape) for p in self._mats[k]]:
                raise ValueError(f"group {k}: matrix shapes differ from the saved state")
            if self._plans[k] is not None:
                self._plans[k].close()
                self._plans[k] = None
            self._resume[k] = pl
        for g, s in zip(self.param_groups, sd["groups"]):
            g.update(s)
        if self._adam is not None and sd.get("adamw") is not None:
            self._adam.load_state_dict(sd["adamw"])

    @torch.no_grad()
    def precond_condition(self) -> Dict[torch.Tensor, Tuple[float, float]]:
        """kappa(diag l) and kappa(diag r) of every matrix parameter that has
        stepped, as the paper's analysis of the diagonal preconditioners
        (Sec. 5.4) reports them per layer and module.  One small kernel per
        parameter group, then one copy to the host."""
        out: Dict[torch.Tensor, Tuple[float, float]] = {}
        for k in range(len(self.param_groups)):
            plan = self._plans[k]
            if plan is None:
                continue
            kap = plan.precond_condition(stream=torch.cuda.current_stream()).cpu()
            for p, (kl, kr) in zip(self._mats[k], kap.tolist()):
                out[p] = (kl, kr)
        return out

    def matrix_plan(self, group: int = 0) -> Optional[lm.Plan]:
        """The libmalt plan of a parameter group (built at its first step)."""
        return self._plan(group)
