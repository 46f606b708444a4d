"""GPU parity of libmalt against the fp64 oracle, through the C ABI.

Inputs are the seeded synthetic workloads; the HIP path and the oracle get the
same float32 buffers.  Each test prints its case before touching the GPU.
"""
import numpy as np
import pytest

from gpu_harness import (TOL_NS, TOL_STATE, compare, run_gpu, run_oracle, run_sampled_against_oracle, say,
                         to_dev)
from oracle import rel_fro
from paper_2608_05088_amd import libmalt as lm
from paper_2608_05088_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lm.lib()   # raises if the library is not built: no fallback


def _hp(w: wl.Workload, **kw):
    d = dict(lr=w.lr, mu1=w.mu1, mu2=w.mu2, eps=w.eps)
    d.update(kw)
    return d


def _inputs(w: wl.Workload, steps: int, indices=None, cid=None):
    cid = w.cid if cid is None else cid
    idx = list(range(len(w.shapes))) if indices is None else list(indices)
    W0 = [wl.weight(cid, i, w.shapes[i]) for i in idx]
    grads = [[wl.grad(cid, t, i, w.shapes[i], w.dist) for i in idx] for t in range(1, steps + 1)]
    return W0, grads


def test_c1_single_matrix_three_steps():
    w = wl.WORKLOADS[1]
    say(f"[parity] C1 {w.shapes} malt x{w.steps}")
    W0, grads = _inputs(w, w.steps)
    g = run_gpu(list(w.shapes), w.variant, W0, grads, _hp(w))
    o = run_oracle(list(w.shapes), w.variant, W0, grads, _hp(w))
    worst = compare(g, o, w.variant, label="C1")
    say(f"[parity] C1 worst {worst}")


RAGGED = [(300, 200), (1, 257), (257, 1), (129, 513), (64, 64), (3, 1000), (513, 129), (1, 1), (250, 250)]


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_ragged_shapes_multi_step(variant):
    say(f"[parity] ragged {RAGGED} {variant} x3")
    rng_shapes = RAGGED
    W0 = [wl.weight(90, i, s) for i, s in enumerate(rng_shapes)]
    grads = [[wl.grad(90, t, i, s, "row_loguniform") for i, s in enumerate(rng_shapes)] for t in (1, 2, 3)]
    hp = dict(lr=3e-3)
    g = run_gpu(rng_shapes, variant, W0, grads, hp)
    o = run_oracle(rng_shapes, variant, W0, grads, hp)
    worst = compare(g, o, variant, label="ragged")
    say(f"[parity] ragged worst {worst}")


def test_unaligned_pointers_take_scalar_path():
    # Params/grads offset by one float inside larger buffers: 4-byte aligned only.
    import torch
    shapes = [(64, 128), (96, 64)]
    say(f"[parity] unaligned {shapes}")
    W0 = [wl.weight(91, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(91, t, i, s) for i, s in enumerate(shapes)] for t in (1, 2)]
    hp = dict(lr=1e-2)
    plan = lm.Plan(shapes, "malt")
    bufW = [torch.zeros(m * n + 1, device="cuda") for m, n in shapes]
    bufG = [torch.zeros(m * n + 1, device="cuda") for m, n in shapes]
    Wd = [b[1:].view(s) for b, s in zip(bufW, shapes)]
    for wd, w0 in zip(Wd, W0):
        wd.copy_(torch.from_numpy(w0))
    o = run_oracle(shapes, "malt", W0, grads, hp)
    for t, Gs in enumerate(grads):
        Gd = [b[1:].view(s) for b, s in zip(bufG, shapes)]
        for gd, gh in zip(Gd, Gs):
            gd.copy_(torch.from_numpy(gh))
        before = [x.double().cpu().numpy() for x in Wd]
        plan.step(Wd, Gd, lm.make_hparams(**hp))
        torch.cuda.synchronize()
        for k in range(len(shapes)):
            dW = Wd[k].double().cpu().numpy() - before[k]
            assert rel_fro(dW, o[t]["inter"][k].dW) <= TOL_NS
            assert rel_fro(plan.state_views(k)[0].double().cpu().numpy(), o[t]["M"][k]) <= TOL_STATE


def test_c2_gpt2_small_full_set():
    w = wl.WORKLOADS[2]
    say(f"[parity] C2 gpt2-small {len(w.shapes)} matrices malt x1")
    W0, grads = _inputs(w, 1)
    g = run_gpu(list(w.shapes), w.variant, W0, grads, _hp(w))
    o = run_oracle(list(w.shapes), w.variant, W0, grads, _hp(w))
    worst = compare(g, o, w.variant, label="C2")
    say(f"[parity] C2 worst {worst}")


def test_c3_gpt2_medium_malter_sampled():
    w = wl.WORKLOADS[3]
    sample = [0, 1, 2, 3, 45, 50, 91, 95]
    say(f"[parity] C3 gpt2-medium {len(w.shapes)} matrices malter x3, oracle on {sample}")
    W0, grads = _inputs(w, 3)
    g = run_gpu(list(w.shapes), w.variant, W0, grads, _hp(w), collect=sample)
    o = run_oracle(list(w.shapes), w.variant, W0, grads, _hp(w), collect=sample)
    worst = compare(g, o, w.variant, label="C3")
    # MALTER's alpha departs from 1 after the first step.
    assert abs(g[0].scal[0]["alpha"] - 1.0) < 1e-5
    assert abs(g[2].scal[0]["alpha"] - 1.0) > 1e-3
    say(f"[parity] C3 worst {worst}")


def test_zero_gradients_leave_parameters_unchanged():
    shapes = [(128, 300), (300, 128)]
    say(f"[parity] zero grads {shapes}")
    for variant in ("malt", "malter"):
        W0 = [wl.weight(92, i, s) for i, s in enumerate(shapes)]
        grads = [[np.zeros(s, np.float32) for s in shapes]]
        g = run_gpu(shapes, variant, W0, grads, dict(lr=1e-2))
        for k in range(len(shapes)):
            assert np.all(np.isfinite(g[0].W[k]))
            assert np.array_equal(g[0].W[k], W0[k].astype(np.float64))
            assert g[0].scal[k]["graft"] == 0.0
            assert np.all(g[0].Lv[k] == np.float32(10.0))


def test_identity_preconditioner_matches_muon_reading():
    shapes = [(256, 768), (384, 256)]
    say(f"[parity] identity preconditioner {shapes}")
    W0 = [wl.weight(93, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(93, t, i, s) for i, s in enumerate(shapes)] for t in (1, 2)]
    hp = dict(lr=2e-2, precond_identity=1)
    g = run_gpu(shapes, "malt", W0, grads, hp)
    o = run_oracle(shapes, "malt", W0, grads, hp)
    compare(g, o, "malt", label="identity")
    for st in g:
        for k in range(len(shapes)):
            assert np.all(st.Lv[k] == 1.0) and np.all(st.Rv[k] == 1.0)
            assert abs(st.scal[k]["graft"] - 1.0) < 1e-6


def test_single_ns_iteration_exposes_scaled_input():
    # With one Newton-Schulz iteration X0 = bf16(L M R) is still in the workspace.
    shapes = [(200, 520), (520, 200)]
    say(f"[parity] ns_steps=1 {shapes}")
    W0 = [wl.weight(94, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(94, 1, i, s, "row_loguniform") for i, s in enumerate(shapes)]]
    hp = dict(lr=1e-2, ns_steps=1)
    g = run_gpu(shapes, "malt", W0, grads, hp)
    o = run_oracle(shapes, "malt", W0, grads, hp)
    compare(g, o, "malt", tol_ns=8e-3, label="ns1")
    for k in range(len(shapes)):
        # bf16 rounding only: relative error <= 2^-9 per entry.
        assert rel_fro(g[0].X0[k], o[0]["inter"][k].M_tilde) < 2.0 ** -9


def test_weight_decay_reading():
    shapes = [(256, 512)]
    say("[parity] weight decay")
    W0 = [wl.weight(95, 0, shapes[0])]
    grads = [[wl.grad(95, t, 0, shapes[0])] for t in (1, 2)]
    hp = dict(lr=1e-2, weight_decay=0.1)
    g = run_gpu(shapes, "malt", W0, grads, hp)
    o = run_oracle(shapes, "malt", W0, grads, hp)
    compare(g, o, "malt", label="wd")


def test_graft_identity_on_gpu_scalars():
    # ||dW|| = lr * alpha * ||O|| ||D|| / (||D|| + eps), with the GPU's own O.
    w = wl.WORKLOADS[2]
    idx = [0, 1, 2, 3]
    shapes = [w.shapes[i] for i in idx]
    say(f"[parity] graft identity {shapes}")
    W0 = [wl.weight(2, i, s) for i, s in zip(idx, shapes)]
    grads = [[wl.grad(2, 1, i, s) for i, s in zip(idx, shapes)]]
    g = run_gpu(shapes, "malter", W0, grads, dict(lr=w.lr))
    for k in range(len(shapes)):
        O = g[0].O[k]
        D = g[0].Lv[k][:, None] * O * g[0].Rv[k][None, :]
        nO, nD = np.linalg.norm(O), np.linalg.norm(D)
        assert abs(np.sqrt(g[0].scal[k]["o2"]) - nO) / nO < 1e-5
        assert abs(np.sqrt(g[0].scal[k]["d2"]) - nD) / nD < 1e-5
        expect = w.lr * g[0].scal[k]["alpha"] * nO * nD / (nD + 1e-8)
        assert abs(np.linalg.norm(g[0].dW[k]) - expect) / expect < 1e-3


def _bf16_rne(x32):
    """float32 -> bf16 bit patterns, round to nearest even (NaN-free input)."""
    u = np.asarray(x32, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_scale_convert_is_bitexact_rne(variant):
    # X0 = bf16((L_i * M_ij) * R_j) in float32, exactly as a host RNE of the same
    # float32 product of the GPU's own L, M, R (byte-exact work). Wide and tall
    # matrices take different kernels; rows of 47 and 201 floats are not
    # 16-byte multiples (scalar tails).
    import torch
    shapes = [(200, 520), (520, 200), (33, 47), (300, 201), (201, 300)]
    say(f"[parity] bf16 conversion bit-exact {variant} {shapes}")
    W0 = [wl.weight(99, i, s) for i, s in enumerate(shapes)]
    G = [wl.grad(99, 1, i, s, "student_t3") for i, s in enumerate(shapes)]
    plan = lm.Plan(shapes, variant)
    Wd, Gd = to_dev(W0), to_dev(G)
    plan.step(Wd, Gd, lm.make_hparams(lr=1e-2, ns_steps=1))
    torch.cuda.synchronize()
    for i, (m, n) in enumerate(shapes):
        M = plan.state_views(i)[0].cpu().numpy()
        dv = plan.debug_views(i)
        Lv, Rv = dv["Lv"].cpu().numpy(), dv["Rv"].cpu().numpy()
        x = (Lv[:, None].astype(np.float32) * M) * Rv[None, :].astype(np.float32)
        got = dv["X0"].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, _bf16_rne(x)), f"matrix {i}: bf16 conversion differs from RNE"


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_gram_and_polynomial_outputs_are_exactly_symmetric(variant):
    # A = X X^T and B' = a I + b A + c A A are symmetric. Diagonal tiles compute
    # only their blocks on and above the block diagonal and stage the rest as
    # the mirror, so both buffers must equal their transposes bitwise
    # (padding included). Shapes: 3 x 3 tiles (diagonal and off-diagonal), a
    # tall matrix, a 1280-square matrix and a split one (m' <= 128: B' as
    # [hi | lo]).
    import torch
    shapes = [(700, 1500), (1500, 300), (1280, 1280), (64, 5000)]
    say(f"[parity] A and B' exactly symmetric {variant} {shapes}")
    W0 = [wl.weight(95, i, s) for i, s in enumerate(shapes)]
    G = [wl.grad(95, 1, i, s, "row_loguniform") for i, s in enumerate(shapes)]
    plan = lm.Plan(shapes, variant)
    Wd, Gd = to_dev(W0), to_dev(G)
    plan.step(Wd, Gd, lm.make_hparams(lr=1e-2))
    torch.cuda.synchronize()
    for i, (m, n) in enumerate(shapes):
        dv = plan.debug_views(i)
        for key in ("A", "B", "B_lo"):
            if key not in dv:
                continue
            x = dv[key].contiguous().view(torch.int16)
            assert torch.equal(x, x.t().contiguous()), f"matrix {i} ({m}x{n}): {key} is not exactly symmetric"
        mc = min(m, n)
        a = dv["A"][:mc, :mc].float()
        assert float(a.abs().max().item()) > 0.0 and bool(torch.isfinite(a).all().item())
        assert float(dv["A"][mc:, :].abs().max().item() if dv["A"].shape[0] > mc else 0.0) == 0.0


def _bf16_ulp(v):
    """Spacing of bf16 numbers at |v| (8 significant bits)."""
    a = np.maximum(np.abs(v), np.finfo(np.float32).tiny)
    return np.exp2(np.floor(np.log2(a)) - 7)


def _check_rounded_product(got, ref, bound, label, split_lo=None):
    """got (bf16 values, or a hi/lo pair) against the fp64 ref: within one bf16
    spacing of ref plus the fp32 accumulation bound, and mostly the exact
    round-to-nearest of ref."""
    if split_lo is None:
        err = np.abs(got - ref)
        assert np.all(err <= _bf16_ulp(ref) + bound), f"{label}: max excess {np.max(err - _bf16_ulp(ref) - bound):.3e}"
        rne = (_bf16_rne(ref.astype(np.float32)).astype(np.uint32) << 16).view(np.float32)
        exact = float(np.mean(got == rne))
        assert exact > 0.98, f"{label}: only {exact:.4f} of the entries are the rounded product"
    else:
        err = np.abs(got + split_lo - ref)
        assert np.all(err <= 2.0 ** -15 * np.abs(ref) + bound + 1e-30), f"{label}: hi + lo off by {err.max():.3e}"


@pytest.mark.parametrize("abc,ns_steps", [((3.4445, -4.7750, 2.0315), 1), ((3.4445, -4.7750, 2.0315), 2),
                                          ((1.5, -0.5, 0.0), 1), ((2.0, -1.5, 0.5), 3)])
def test_gram_and_polynomial_against_fp64_of_their_own_inputs(abc, ns_steps):
    # Kernel-level check of the two symmetric products, on the GPU's own bf16
    # operands: the last iteration's A and B' (debug views) against A = s X X^T
    # (first iteration: X = X0, s = sigma^2) and B' = a I + b A + c A A computed
    # in fp64 from the same bf16 values.  c != 0 adds b A inside the
    # polynomial's main loop, c = 0 reloads A in its epilogue; the shapes cover
    # diagonal and off-diagonal tiles, a tall matrix, a 1280-square matrix and a
    # split one (m' <= 128: B' as a bf16 hi/lo pair).
    import torch
    a, b, c = abc
    shapes = [(700, 1500), (1500, 300), (1280, 1280), (64, 5000)]
    say(f"[parity] symmetric products vs fp64 of their inputs {abc} ns_steps={ns_steps} {shapes}")
    W0 = [wl.weight(97, i, s) for i, s in enumerate(shapes)]
    G = [wl.grad(97, 1, i, s, "row_loguniform") for i, s in enumerate(shapes)]
    plan = lm.Plan(shapes, "malt")
    Wd, Gd = to_dev(W0), to_dev(G)
    plan.step(Wd, Gd, lm.make_hparams(lr=1e-2, ns_steps=ns_steps, ns_a=a, ns_b=b, ns_c=c))
    torch.cuda.synchronize()
    u = 2.0 ** -23
    for i, (m, n) in enumerate(shapes):
        dv = plan.debug_views(i)
        A = dv["A"].float().cpu().numpy().astype(np.float64)
        p = A.shape[0]
        if ns_steps == 1:
            X = dv["X0"].float().cpu().numpy().astype(np.float64)
            X = X.T if m > n else X
            Xp = np.zeros((p, X.shape[1]))
            Xp[:X.shape[0]] = X
            sig = np.float32(dv["scalars"]["sigma"].item())
            s = float(np.float32(sig * sig))
            ref = s * (Xp @ Xp.T)
            bound = s * (np.abs(Xp) @ np.abs(Xp).T) * Xp.shape[1] * u + 2 * u * np.abs(ref)
            _check_rounded_product(A, ref, bound, f"matrix {i} {m}x{n} A")
        ref = a * np.eye(p) + b * A + c * (A @ A)
        bound = (abs(c) * (np.abs(A) @ np.abs(A)) * p + abs(b) * np.abs(A) + abs(a)) * u * 4
        B = dv["B"].float().cpu().numpy().astype(np.float64)
        lo = dv["B_lo"].float().cpu().numpy().astype(np.float64) if "B_lo" in dv else None
        _check_rounded_product(B, ref, bound, f"matrix {i} {m}x{n} B'", split_lo=lo)


# Four shape kinds (a split contraction with K = 2 m', unsplit K = 768, a tall
# matrix, a wide split one) repeated: 496 update tiles, more than one per
# compute unit, of different K and pitch in one grouped launch.
MIXED = [(100, 2900), (700, 1500), (1500, 300), (64, 5000)] * 8


def test_many_tiles_mixed_shapes():
    say(f"[parity] mixed shapes {len(MIXED)} matrices malter x2")
    W0 = [wl.weight(96, i, s) for i, s in enumerate(MIXED)]
    grads = [[wl.grad(96, t, i, s, "row_loguniform") for i, s in enumerate(MIXED)] for t in (1, 2)]
    hp = dict(lr=4e-3)
    g = run_gpu(MIXED, "malter", W0, grads, hp)
    o = run_oracle(MIXED, "malter", W0, grads, hp)
    worst = compare(g, o, "malter", label="mixed")
    say(f"[parity] mixed worst {worst}")


def test_c4_gpt2_large_sampled():
    # The benchmark's launch configuration: all 144 GPT-2 Large matrices in one
    # plan; the oracle checks one matrix of each shape from the first and last
    # blocks (the step is independent per matrix).
    w = wl.WORKLOADS[4]
    sample = [0, 1, 2, 3, 140, 141, 142, 143]
    say(f"[parity] C4 gpt2-large {len(w.shapes)} matrices {w.variant} x1, oracle on {sample}")
    W0, grads = _inputs(w, 1)
    g = run_gpu(list(w.shapes), w.variant, W0, grads, _hp(w), collect=sample)
    o = run_oracle(list(w.shapes), w.variant, W0, grads, _hp(w), collect=sample)
    worst = compare(g, o, w.variant, label="C4")
    say(f"[parity] C4 worst {worst}")


@pytest.mark.slow
def test_c4_gpt2_large_ten_steps_persistent_state():
    # The benchmark's timed configuration: ten consecutive steps of the full
    # 144-matrix plan with persistent state and fresh gradients per step; the
    # oracle follows eight matrices (one of each shape from the first and last
    # blocks) through all ten steps and every step is compared.
    w = wl.WORKLOADS[4]
    sample = [0, 1, 2, 3, 140, 141, 142, 143]
    say(f"[parity] C4 gpt2-large {len(w.shapes)} matrices {w.variant} x{w.steps}, oracle on {sample}")
    worst = run_sampled_against_oracle(w, w.steps, sample, _hp(w), label="C4x10")
    say(f"[parity] C4 x{w.steps} worst {worst}")


@pytest.mark.slow
def test_c5_stress_full_plan_one_step():
    # C5 as configured: one MALTER step over all 128 matrices in one grouped
    # plan (its own XCD-balanced tile lists); four matrices, two of each
    # shape from both ends of the list, are compared with the oracle.
    w = wl.WORKLOADS[5]
    sample = [0, 1, 126, 127]
    say(f"[parity] C5 stress {len(w.shapes)} matrices {w.variant} x1, oracle on {sample}")
    worst = run_sampled_against_oracle(w, 1, sample, _hp(w), label="C5 full")
    say(f"[parity] C5 full plan worst {worst}")


@pytest.mark.parametrize("ns_steps", [2, 4])
def test_even_newton_schulz_step_counts(ns_steps):
    # With an even iteration count the final O lands in the first X buffer
    # (the odd counts of every other test end in the second).
    shapes = [(768, 2304), (2304, 768), (100, 900), (20, 300)]
    say(f"[parity] ns_steps={ns_steps} {shapes} malter x2")
    W0 = [wl.weight(88, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(88, t, i, s, "row_loguniform") for i, s in enumerate(shapes)] for t in (1, 2)]
    hp = dict(lr=5e-3, ns_steps=ns_steps)
    g = run_gpu(shapes, "malter", W0, grads, hp)
    o = run_oracle(shapes, "malter", W0, grads, hp)
    worst = compare(g, o, "malter", label=f"ns{ns_steps}")
    say(f"[parity] ns_steps={ns_steps} worst {worst}")


@pytest.mark.parametrize("abc", [(1.5, -0.5, 0.0), (2.0, -1.5, 0.5)])
def test_other_newton_schulz_coefficients(abc):
    # The coefficients are hyper-parameters. c = 0 is the cubic iteration
    # X <- a X + b X X^T X: its polynomial phase has no product, B' = a I + b A.
    # A second quintic checks that nothing assumes Muon's numbers.
    a, b, c = abc
    shapes = [(300, 900), (900, 300), (768, 768), (100, 400)]
    say(f"[parity] ns coefficients {abc} {shapes} malt x2")
    W0 = [wl.weight(89, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(89, t, i, s, "normal") for i, s in enumerate(shapes)] for t in (1, 2)]
    hp = dict(lr=5e-3, ns_a=a, ns_b=b, ns_c=c)
    g = run_gpu(shapes, "malt", W0, grads, hp)
    o = run_oracle(shapes, "malt", W0, grads, hp)
    worst = compare(g, o, "malt", label=f"ns{abc}")
    say(f"[parity] ns coefficients {abc} worst {worst}")


@pytest.mark.slow
def test_c5_stress_subset_two_steps():
    # C5's two shapes at full size (4096 x 4096 and 4096 x 11008, Student-t
    # gradients), two MALTER steps so alpha departs from 1.  The plan holds the
    # subset only: the step is independent per matrix.
    w = wl.WORKLOADS[5]
    idx = [0, 1]
    shapes = [w.shapes[i] for i in idx]
    say(f"[parity] C5 subset {shapes} {w.variant} x2")
    W0, grads = _inputs(w, 2, indices=idx)
    g = run_gpu(shapes, w.variant, W0, grads, _hp(w))
    o = run_oracle(shapes, w.variant, W0, grads, _hp(w))
    worst = compare(g, o, w.variant, label="C5")
    assert abs(g[1].scal[1]["alpha"] - 1.0) > 1e-3
    say(f"[parity] C5 worst {worst}")


# Extreme aspect ratios: the split (m' <= 128) contraction with the longest
# allowed dimension, and a thin tall matrix.
EXTREME = [(1, 1 << 20), (1 << 20, 2), (3, 700000)]


def test_extreme_aspect_ratios():
    say(f"[parity] extreme aspect ratios {EXTREME} malter x2")
    W0 = [wl.weight(97, i, s) for i, s in enumerate(EXTREME)]
    grads = [[wl.grad(97, t, i, s, "row_loguniform") for i, s in enumerate(EXTREME)] for t in (1, 2)]
    hp = dict(lr=1e-2)
    g = run_gpu(EXTREME, "malter", W0, grads, hp)
    o = run_oracle(EXTREME, "malter", W0, grads, hp)
    worst = compare(g, o, "malter", label="extreme")
    say(f"[parity] extreme worst {worst}")


@pytest.mark.slow
@pytest.mark.parametrize("shape,k,variant", [((300, 500), 300, "malter"), ((32768, 32768), 32768, "malt"),
                                             ((1 << 20, 1792), 1792, "malter")])
def test_permutation_closed_form_up_to_max_size(shape, k, variant):
    # A scaled partial permutation keeps every stage entrywise (closed form in
    # tests/closed_forms.py, pinned to the oracle on the CPU), and bf16 holds
    # its pattern exactly: off-pattern entries must come out exactly zero.
    # Covers the largest accepted shapes: min dimension 32768, and the longest
    # dimension 2^20 with the padded matrix near 2^31 elements (tall path).
    import torch
    from closed_forms import permutation_step, random_permutation_pattern
    m, n = shape
    say(f"[parity] permutation closed form {shape} k={k} {variant}")
    rows, cols, g = random_permutation_pattern(m, n, k, seed=99)
    g32 = g.astype(np.float32)
    hp = dict(lr=1e-3, mu1=0.95, mu2=0.99, eps=1e-8)
    dev = torch.device("cuda:0")
    rt, ct = torch.from_numpy(rows).to(dev), torch.from_numpy(cols).to(dev)
    G = torch.zeros(m, n, device=dev)
    G[rt, ct] = torch.from_numpy(g32).to(dev)
    W = torch.zeros(m, n, device=dev)
    plan = lm.Plan([shape], variant)
    plan.step([W], [G], lm.make_hparams(**hp))
    torch.cuda.synchronize()
    l, r, Lv, Rv, dw = permutation_step(m, n, rows, cols, g32.astype(np.float64), variant, **hp)
    Mg, lg, rg, _ = plan.state_views(0)
    dvw = plan.debug_views(0)
    assert rel_fro(lg.double().cpu().numpy(), l) <= TOL_STATE
    assert rel_fro(rg.double().cpu().numpy(), r) <= TOL_STATE
    assert rel_fro(dvw["Lv"].double().cpu().numpy(), Lv) <= TOL_STATE
    assert rel_fro(dvw["Rv"].double().cpu().numpy(), Rv) <= TOL_STATE
    assert rel_fro(Mg[rt, ct].double().cpu().numpy(), 0.05 * g32.astype(np.float64)) <= TOL_STATE
    err = rel_fro(W[rt, ct].double().cpu().numpy(), dw)
    # Off the pattern (W started at zero, so W = dW): exactly zero.
    rng = np.random.default_rng(7)
    ri = torch.from_numpy(rng.integers(0, m, 50000)).to(dev)
    ci = torch.from_numpy(rng.integers(0, n, 50000)).to(dev)
    on = torch.zeros(m, dtype=torch.int64, device=dev) - 1
    on[rt] = ct
    off = on[ri] != ci
    assert int(off.sum().item()) > 0
    assert float(W[ri[off], ci[off]].abs().max().item()) == 0.0
    say(f"[parity] permutation {shape}: dW rel err on the pattern {err:.3e}")
    assert err <= TOL_NS
    if m * n <= 1 << 20:   # small case: the oracle itself agrees
        G0 = np.zeros((m, n), np.float32)
        G0[rows, cols] = g32
        o = run_oracle([shape], variant, [np.zeros((m, n), np.float32)], [[G0]], hp)
        assert rel_fro(W.double().cpu().numpy(), o[0]["inter"][0].dW) <= TOL_NS
    plan.close()
    del W, G
    torch.cuda.empty_cache()


SMALL = [(5, 5), (32, 4000), (4000, 32), (33, 600), (2, 3), (17, 70000), (31, 31)]


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_short_side_up_to_32_runs_in_fp32(variant):
    # Short side <= 32: Newton-Schulz in fp32 (X, A, B' never rounded), so with
    # rows scaled over three decades (a spread spectrum the quintic does not
    # flatten in five steps) the only bf16 rounding left is the final O's.
    # (33, 600) sits just past the boundary, on the matrix-core path.
    say(f"[parity] short sides {SMALL} {variant} x3, row scales over 1e-3..1")
    W0 = [wl.weight(89, i, s) for i, s in enumerate(SMALL)]
    grads = [[wl.grad(89, t, i, s, "row_loguniform") for i, s in enumerate(SMALL)] for t in (1, 2, 3)]
    hp = dict(lr=1e-2)
    g = run_gpu(SMALL, variant, W0, grads, hp)
    o = run_oracle(SMALL, variant, W0, grads, hp)
    worst = compare(g, o, variant, label="small")
    for t in range(3):
        for k, s in enumerate(SMALL):
            if min(s) <= 32:
                err = rel_fro(g[t].O[k], o[t]["inter"][k].O)
                assert err <= 4e-3, f"step {t + 1} {s}: O rel err {err:.3e} (fp32 path)"
    say(f"[parity] small worst {worst}")


# Low-rank-plus-noise gradients (rank r factors fixed per matrix, noise drawn
# per step `noise` below them): the regime of real gradients at small batch.
LOW_RANK = [((300, 900), "lowrank16_0.1", 16), ((768, 2304), "lowrank32_0.1", 32),
            ((1024, 1024), "lowrank8_0.2", 8), ((1536, 512), "lowrank64_0.05", 64)]


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_low_rank_gradients(variant):
    # Newton-Schulz maps every singular value above ~2e-3 of the top one close
    # to 1, so the noise directions of such a gradient end up carrying most of
    # ||O|| (67-89% here) although they hold a few percent of ||M~||.  bf16
    # rounding of X in every iteration perturbs that noise subspace, and the
    # quintic then amplifies the perturbation: a CPU emulation of the bf16
    # path puts the whole O at 1.6-6.8e-2 from fp64 on these inputs, but the
    # rank-r part of O at 0.8-1.1e-2.  Bars: the state at 1e-5, O projected on
    # the oracle's top-r left singular vectors of M~ at 2e-2, and the whole O
    # and dW at 1e-1.
    shapes = [s for s, _, _ in LOW_RANK]
    say(f"[parity] low-rank gradients {[(s, d) for s, d, _ in LOW_RANK]} {variant} x2")
    W0 = [wl.weight(81, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(81, t, i, s, d) for i, (s, d, _) in enumerate(LOW_RANK)] for t in (1, 2)]
    hp = dict(lr=5e-3)
    g = run_gpu(shapes, variant, W0, grads, hp)
    o = run_oracle(shapes, variant, W0, grads, hp)
    worst = compare(g, o, variant, tol_ns=1e-1, label="low-rank")
    for t in range(2):
        for k, (s, d, r) in enumerate(LOW_RANK):
            it = o[t]["inter"][k]
            U = np.linalg.svd(it.M_tilde, full_matrices=False)[0][:, :r]
            err = rel_fro(U.T @ g[t].O[k], U.T @ it.O)
            say(f"[parity] low-rank step {t + 1} {s} {d}: O {rel_fro(g[t].O[k], it.O):.3e}, rank-{r} part {err:.3e}")
            assert err <= TOL_NS, f"step {t + 1} {s}: rank-{r} part of O rel err {err:.3e}"
    say(f"[parity] low-rank worst {worst}")
