"""Synthetic-token GPT-2 training loop: per-iteration cost of AdamW, Muon,
MALT and MALTER on one GPU (the counterpart of the paper's per-iteration
timing comparison of Sec. 5.5 and its table).

The model is GPT-2 Small / Medium / Large (transformers' GPT2LMHeadModel,
random initialisation, no checkpoint, dropout off), the data random token
ids (no dataset).  Matrix parameters (the four per-block matrices) go to
libmalt (MALT / MALTER / Muon), the rest to AdamW; "adamw" trains everything
with torch's AdamW.  The model trains in float32 (no autocast).  One
iteration is the paper's global batch: 480 sequences of 1024 tokens
(Sec. 5.1), here as 60 accumulated micro-batches of 8, then one optimizer
step; weight decay 0.1 on both parts (hyper-parameter table) and a linear
warm-up over the first 10% of the run (Sec. 5.1).

  python -m paper_2608_05088_amd.train --model gpt2-medium --optim adamw,muon,malt,malter

Prints one JSON line per optimizer: ms per iteration, of which optimizer
step, the optimizer state (as the paper counts it: the tensors the algorithm
keeps, and as allocated) and the peak device memory.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MODELS = {"gpt2-small": (12, 768, 12), "gpt2-medium": (24, 1024, 16), "gpt2-large": (36, 1280, 20)}


def build_model(name: str, device, seed: int = 0, n_positions: int = 1024):
    import torch
    from transformers import GPT2Config, GPT2LMHeadModel
    n_layer, n_embd, n_head = MODELS[name]
    cfg = GPT2Config(n_layer=n_layer, n_embd=n_embd, n_head=n_head, vocab_size=50257, n_positions=n_positions,
                     bos_token_id=50256, eos_token_id=50256, resid_pdrop=0.0, embd_pdrop=0.0, attn_pdrop=0.0)
    torch.manual_seed(seed)
    model = GPT2LMHeadModel(cfg).to(device)
    model.train()
    return model


def block_matrix(name: str, p) -> bool:
    """The paper's matrix parameters: attention and MLP weights of each block."""
    return p.dim() == 2 and ".h." in name and name.endswith("weight")


from .schedules import lambda_lr, linear_warmup  # noqa: E402


def make_optimizer(kind: str, model, lr: float, adamw_lr: float, weight_decay: float = 0.1):
    import torch
    from .optim import MALT
    if kind == "adamw":
        return torch.optim.AdamW(model.parameters(), lr=adamw_lr, betas=(0.9, 0.95), eps=1e-8,
                                 weight_decay=weight_decay)
    mats = {id(p) for n, p in model.named_parameters() if block_matrix(n, p)}
    return MALT(model.parameters(), lr=lr, variant=kind, adamw_lr=adamw_lr, weight_decay=weight_decay,
                adamw_weight_decay=weight_decay, matrix_filter=lambda p: id(p) in mats)


def _adam_state_bytes(opt) -> int:
    import torch
    total = 0
    for st in opt.state.values():
        for v in st.values():
            if torch.is_tensor(v) and v.dim() > 0:
                total += v.numel() * v.element_size()
    return total


def optimizer_state_bytes(opt) -> dict:
    """Optimizer state in bytes: "algorithm" counts what the method keeps
    (AdamW: two moments; Muon: M; MALT: M, l, r; MALTER: plus nu, Sec. 5.5),
    "allocated" what the implementation holds (a Muon plan keeps l and r it
    does not use)."""
    from .optim import MALT
    if not isinstance(opt, MALT):
        b = _adam_state_bytes(opt)
        return {"algorithm": b, "allocated": b}
    alg = alloc = _adam_state_bytes(opt._adam) if opt._adam is not None else 0
    for k in range(len(opt.param_groups)):
        plan = opt.matrix_plan(k)
        if plan is None:
            continue
        alloc += plan.state_bytes
        for m, n in plan.shapes:
            alg += 4 * m * n
            if opt.variant != "muon":
                alg += 4 * (m + n)
            if opt.variant == "malter":
                alg += 4
    return {"algorithm": alg, "allocated": alloc}


def run(kind: str, args, device) -> dict:
    import torch
    torch.cuda.reset_peak_memory_stats(device)
    model = build_model(args.model, device, seed=args.seed)
    opt = make_optimizer(kind, model, args.lr, args.adamw_lr, args.weight_decay)
    # The paper's protocol: linear warm-up over the first 10% of the run.
    sched = lambda_lr(opt, linear_warmup(args.warmup + args.iters))
    gen = torch.Generator(device=device)
    gen.manual_seed(args.seed)
    B, T = args.micro_batch, args.seq

    def iteration():
        for _ in range(args.accum):
            ids = torch.randint(0, 50257, (B, T), device=device, generator=gen)
            loss = model(input_ids=ids, labels=ids).loss
            (loss / args.accum).backward()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        opt.step()
        e.record()
        opt.zero_grad(set_to_none=True)
        sched.step()
        return s, e, loss

    for _ in range(args.warmup):
        iteration()
    torch.cuda.synchronize()
    it_s, it_e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    steps = []
    it_s.record()
    for _ in range(args.iters):
        s, e, loss = iteration()
        steps.append((s, e))
    it_e.record()
    torch.cuda.synchronize()
    ms_iter = it_s.elapsed_time(it_e) / args.iters
    ms_opt = sum(s.elapsed_time(e) for s, e in steps) / args.iters
    n_params = sum(p.numel() for p in model.parameters())
    n_mat = sum(p.numel() for n, p in model.named_parameters() if block_matrix(n, p))
    sb = optimizer_state_bytes(opt)
    mib = float(1 << 20)
    out = {"optimizer": kind, "model": args.model, "params": n_params, "matrix_params": n_mat,
           "micro_batch": B, "accum": args.accum, "tokens_per_iter": B * T * args.accum, "iters": args.iters,
           "ms_per_iter": round(ms_iter, 3), "optimizer_step_ms": round(ms_opt, 3),
           "forward_backward_ms": round(ms_iter - ms_opt, 3),
           "optimizer_state_MiB": round(sb["algorithm"] / mib, 2),
           "optimizer_state_allocated_MiB": round(sb["allocated"] / mib, 2),
           "peak_device_memory_GiB": round(torch.cuda.max_memory_allocated(device) / mib / 1024, 2),
           "final_loss": round(float(loss.item()), 4), "dtype": "float32", "data": "synthetic token ids"}
    del opt, model
    torch.cuda.empty_cache()
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--model", default="gpt2-medium", choices=sorted(MODELS))
    ap.add_argument("--optim", default="adamw,muon,malt,malter")
    ap.add_argument("--micro-batch", type=int, default=8)
    ap.add_argument("--seq", type=int, default=1024)
    ap.add_argument("--accum", type=int, default=60)
    ap.add_argument("--iters", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--lr", type=float, default=1.3e-3)
    ap.add_argument("--adamw-lr", type=float, default=6e-4)
    ap.add_argument("--weight-decay", type=float, default=0.1)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        raise SystemExit("a GPU is required")
    device = torch.device("cuda:0")
    torch.cuda.init()
    for kind in args.optim.split(","):
        print(f"[train] {args.model} {kind}", file=sys.stderr, flush=True)
        t0 = time.time()
        res = run(kind.strip(), args, device)
        res["wall_s"] = round(time.time() - t0, 1)
        print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
