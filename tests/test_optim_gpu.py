"""GPU tests of the torch.optim adapter (MALT / MALTER / Muon through libmalt
for matrix parameters, AdamW for the rest)."""
import copy

import numpy as np
import pytest

from gpu_harness import TOL_NS, TOL_STATE, run_oracle, say
from oracle import rel_fro

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_05088_amd import libmalt as lm
    lm.lib()


def _tiny_gpt2(seed=0):
    import torch
    from transformers import GPT2Config, GPT2LMHeadModel
    cfg = GPT2Config(n_layer=2, n_embd=256, n_head=4, vocab_size=1000, n_positions=64, bos_token_id=0,
                     eos_token_id=0, resid_pdrop=0.0, embd_pdrop=0.0, attn_pdrop=0.0)
    torch.manual_seed(seed)
    return GPT2LMHeadModel(cfg).cuda().train()


def _split(model):
    from paper_2608_05088_amd.train import block_matrix
    names = [n for n, p in model.named_parameters() if block_matrix(n, p)]
    ids = {id(p) for n, p in model.named_parameters() if n in names}
    return names, (lambda p: id(p) in ids)


def _hp_kw(variant, lr, wd=0.0):
    kw = dict(lr=lr, weight_decay=wd)
    if variant == "muon":
        kw["precond_identity"] = 1
    return kw


@pytest.mark.parametrize("variant,wd", [("malt", 0.0), ("malter", 0.0), ("muon", 0.0), ("malt", 0.1),
                                        ("malter", 0.1)])
def test_adapter_matches_oracle_and_adamw(variant, wd):
    """GPT-2 parameter set (2 blocks, d = 256) through the adapter with seeded
    synthetic matrix gradients: every matrix state and update against the
    oracle, every other parameter bitwise against torch's AdamW."""
    import torch
    from paper_2608_05088_amd import workloads as wl
    from paper_2608_05088_amd.optim import MALT
    say(f"[optim] GPT-2 parameter set, {variant} + AdamW, weight decay {wd}, 3 steps, synthetic gradients")
    model = _tiny_gpt2()
    ref = copy.deepcopy(model)
    names, filt = _split(model)
    params = dict(model.named_parameters())
    lr, alr = 2e-3, 1e-3
    opt = MALT(model.parameters(), lr=lr, variant=variant, adamw_lr=alr, weight_decay=wd, adamw_weight_decay=wd,
               matrix_filter=filt)
    ref_rest = [p for n, p in ref.named_parameters() if n not in names]
    ref_opt = torch.optim.AdamW(ref_rest, lr=alr, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    gen = torch.Generator(device="cuda").manual_seed(1)
    W0 = [params[n].detach().cpu().numpy().copy() for n in names]
    shapes = [w.shape for w in W0]
    grads = [[wl.grad(95, t, i, s) for i, s in enumerate(shapes)] for t in (1, 2, 3)]
    dW = []
    for t in range(3):
        for n, p in model.named_parameters():
            p.grad = (torch.from_numpy(grads[t][names.index(n)]).cuda() if n in names
                      else torch.randn(p.shape, device="cuda", generator=gen) * 1e-2)
        for (n, p), (_, q) in zip(model.named_parameters(), ref.named_parameters()):
            q.grad = p.grad.detach().clone()
        before = [params[n].detach().double().cpu().numpy() for n in names]
        opt.step()
        ref_opt.step()
        opt.zero_grad()
        ref_opt.zero_grad()
        dW.append([params[n].detach().double().cpu().numpy() - b for n, b in zip(names, before)])
    o = run_oracle(shapes, "malter" if variant == "malter" else "malt", W0, grads, _hp_kw(variant, lr, wd))
    plan = opt.matrix_plan()
    worst = 0.0
    for t in range(3):
        for k in range(len(names)):
            err = rel_fro(dW[t][k], o[t]["inter"][k].dW)
            worst = max(worst, err)
            assert err <= TOL_NS, f"step {t + 1} {names[k]}: dW rel err {err:.3e}"
    for k in range(len(names)):
        M, l, r, nu = plan.state_views(k)
        assert rel_fro(M.double().cpu().numpy(), o[2]["M"][k]) <= TOL_STATE
        assert rel_fro(l.double().cpu().numpy(), o[2]["l"][k]) <= TOL_STATE
        assert rel_fro(r.double().cpu().numpy(), o[2]["r"][k]) <= TOL_STATE
        if variant == "malter":
            assert abs(float(nu.item()) - o[2]["nu"][k]) <= TOL_STATE * abs(o[2]["nu"][k])
    for (n, p), (_, q) in zip(model.named_parameters(), ref.named_parameters()):
        if n not in names:
            assert torch.equal(p, q), n
    say(f"[optim] {variant} worst matrix dW err {worst:.3e}")


@pytest.mark.parametrize("variant", ["malt", "malter", "muon"])
def test_adapter_on_real_gradients_matches_direct_plan(variant):
    """A training loop on a small GPT-2: the adapter's matrix updates are
    bitwise those of a libmalt plan stepped directly with the same gradients,
    and its elementwise state (M, l, r, nu) matches the oracle.  The update
    itself is compared with the oracle above, on synthetic gradients: these
    early real gradients are rank-deficient (LayerNorm inputs, 256 tokens per
    batch), and on such inputs bf16 Newton-Schulz differs from the fp64
    iteration by a few percent whatever the implementation."""
    import torch
    from paper_2608_05088_amd import libmalt as lm
    from paper_2608_05088_amd.optim import MALT
    say(f"[optim] small GPT-2 training, {variant}: adapter vs direct plan, 3 steps")
    model = _tiny_gpt2()
    names, filt = _split(model)
    params = dict(model.named_parameters())
    lr = 2e-3
    opt = MALT(model.parameters(), lr=lr, variant=variant, adamw_lr=1e-3, matrix_filter=filt)
    mirror = [params[n].detach().clone() for n in names]
    W0 = [m.cpu().numpy().copy() for m in mirror]
    direct = lm.Plan([tuple(m.shape) for m in mirror], "malter" if variant == "malter" else "malt")
    hp = lm.make_hparams(**_hp_kw(variant, lr))
    gen = torch.Generator(device="cuda").manual_seed(1)
    grads, dW = [], []
    for t in range(3):
        ids = torch.randint(0, 1000, (4, 64), device="cuda", generator=gen)
        model(input_ids=ids, labels=ids).loss.backward()
        G = [params[n].grad.detach().clone() for n in names]
        grads.append([g.cpu().numpy() for g in G])
        before = [params[n].detach().double().cpu().numpy() for n in names]
        opt.step()
        opt.zero_grad()
        direct.step(mirror, G, hp)
        torch.cuda.synchronize()
        for n, m in zip(names, mirror):
            assert torch.equal(params[n], m), f"step {t + 1} {n}"
        dW.append([params[n].detach().double().cpu().numpy() - b for n, b in zip(names, before)])
    o = run_oracle([w.shape for w in W0], "malter" if variant == "malter" else "malt", W0, grads,
                   _hp_kw(variant, lr))
    plan = opt.matrix_plan()
    for k in range(len(names)):
        M, l, r, nu = plan.state_views(k)
        assert rel_fro(M.double().cpu().numpy(), o[2]["M"][k]) <= TOL_STATE
        assert rel_fro(l.double().cpu().numpy(), o[2]["l"][k]) <= TOL_STATE
        assert rel_fro(r.double().cpu().numpy(), o[2]["r"][k]) <= TOL_STATE
        if variant == "malter":
            assert abs(float(nu.item()) - o[2]["nu"][k]) <= TOL_STATE * abs(o[2]["nu"][k])
    errs = [rel_fro(dW[t][k], o[t]["inter"][k].dW) for t in range(3) for k in range(len(names))]
    say(f"[optim] {variant} real-gradient dW vs oracle: max {max(errs):.3e} median {np.median(errs):.3e}")


def _synthetic(seed):
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    shapes = [(96, 200), (300, 128), (64,), (128, 16, 3)]
    return [torch.randn(s, device="cuda", generator=g) * 0.02 for s in shapes]


def _set_grads(params, step):
    import torch
    g = torch.Generator(device="cuda").manual_seed(1000 + step)
    for p in params:
        p.grad = torch.randn(p.shape, device="cuda", generator=g) * 0.01


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_state_dict_resume_is_bitwise(variant):
    import torch
    from paper_2608_05088_amd.optim import MALT
    say(f"[optim] state_dict resume {variant}")
    A = [p.requires_grad_() for p in _synthetic(3)]
    B = [p.detach().clone().requires_grad_() for p in A]
    oa = MALT(A, lr=3e-3, variant=variant, adamw_lr=1e-3)
    ob = MALT(B, lr=3e-3, variant=variant, adamw_lr=1e-3)
    for s in range(2):
        _set_grads(A, s); _set_grads(B, s)
        oa.step(); ob.step()
    sd = ob.state_dict()
    oc = MALT(B, lr=3e-3, variant=variant, adamw_lr=1e-3)
    oc.load_state_dict(sd)
    for s in range(2, 4):
        _set_grads(A, s); _set_grads(B, s)
        oa.step(); oc.step()
    torch.cuda.synchronize()
    for a, b in zip(A, B):
        assert torch.equal(a, b)
    assert oc.matrix_plan().t == 4


def test_scheduler_scales_both_learning_rates():
    import torch
    from paper_2608_05088_amd.optim import MALT
    say("[optim] scheduler")
    P = [p.requires_grad_() for p in _synthetic(4)]
    Q = [p.detach().clone().requires_grad_() for p in P]
    op = MALT(P, lr=4e-3, adamw_lr=2e-3)
    oq = MALT(Q, lr=2e-3, adamw_lr=1e-3)
    sched = torch.optim.lr_scheduler.LambdaLR(op, lambda s: 0.5)   # halves lr (and adamw's)
    _set_grads(P, 0); _set_grads(Q, 0)
    before = [p.detach().clone() for p in P]
    op.step(); oq.step()
    torch.cuda.synchronize()
    for p, q, b in zip(P, Q, before):
        d1, d2 = (p - b).double(), (q - b).double()
        assert torch.allclose(d1, d2, rtol=1e-5, atol=1e-10)
    del sched
