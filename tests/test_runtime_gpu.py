"""Runtime properties of libmalt on the GPU: determinism, checkpoint/resume,
independence of matrices, error paths and per-phase timing."""
import numpy as np
import pytest

from gpu_harness import run_gpu, say, to_dev
from paper_2608_05088_amd import libmalt as lm
from paper_2608_05088_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lm.lib()


SHAPES = [(768, 2304), (768, 768), (300, 1000), (1000, 300), (7, 33)]


def _inputs(steps, cid=96):
    W0 = [wl.weight(cid, i, s) for i, s in enumerate(SHAPES)]
    grads = [[wl.grad(cid, t, i, s, "student_t3") for i, s in enumerate(SHAPES)] for t in range(1, steps + 1)]
    return W0, grads


def test_bitwise_deterministic():
    say("[runtime] determinism")
    W0, grads = _inputs(2)
    a = run_gpu(SHAPES, "malter", W0, grads, dict(lr=6e-3))
    b = run_gpu(SHAPES, "malter", W0, grads, dict(lr=6e-3))
    for sa, sb in zip(a, b):
        for k in range(len(SHAPES)):
            assert np.array_equal(sa.W[k], sb.W[k])
            assert np.array_equal(sa.M[k], sb.M[k])
            assert np.array_equal(sa.l[k], sb.l[k]) and np.array_equal(sa.r[k], sb.r[k])
            assert sa.nu[k] == sb.nu[k]


def test_checkpoint_resume_is_bitwise():
    import torch
    say("[runtime] checkpoint/resume")
    W0, grads = _inputs(3)
    hp = lm.make_hparams(lr=6e-3)
    ref = run_gpu(SHAPES, "malter", W0, grads, dict(lr=6e-3))
    plan = lm.Plan(SHAPES, "malter")
    Wd = to_dev(W0)
    for Gs in grads[:2]:
        plan.step(Wd, to_dev(Gs), hp)
    torch.cuda.synchronize()
    saved_state = plan.state.clone()
    saved_W = [w.clone() for w in Wd]
    t = plan.t
    plan.close()
    plan2 = lm.Plan(SHAPES, "malter", state=saved_state, from_existing=True, step=t)
    assert plan2.t == 2
    plan2.step(saved_W, to_dev(grads[2]), hp)
    torch.cuda.synchronize()
    for k in range(len(SHAPES)):
        assert np.array_equal(saved_W[k].double().cpu().numpy(), ref[2].W[k])


def test_matrices_are_independent():
    say("[runtime] subset independence")
    W0, grads = _inputs(2)
    full = run_gpu(SHAPES, "malt", W0, grads, dict(lr=1e-2))
    sub_idx = [1, 3]
    sub = run_gpu([SHAPES[i] for i in sub_idx], "malt", [W0[i] for i in sub_idx],
                  [[g[i] for i in sub_idx] for g in grads], dict(lr=1e-2))
    for t in range(2):
        for k, i in enumerate(sub_idx):
            assert np.array_equal(sub[t].W[k], full[t].W[i])


def test_errors_leave_state_untouched():
    import torch
    say("[runtime] error paths")
    shapes = [(64, 96), (96, 64)]
    plan = lm.Plan(shapes, "malt")
    W = to_dev([wl.weight(97, i, s) for i, s in enumerate(shapes)])
    G = to_dev([wl.grad(97, 1, i, s) for i, s in enumerate(shapes)])
    before = plan.state.clone()
    with pytest.raises(lm.MaltError) as e:
        plan._c_shapes[0].rows = 65
        plan.step(W, G)
    assert e.value.status == lm.MALT_ERR_STATE_MISMATCH
    plan._c_shapes[0].rows = 64
    with pytest.raises(ValueError):
        plan.step([W[0], W[0]], G)            # matrix 1 gets a tensor of another shape
    with pytest.raises(lm.MaltError) as e:
        plan._step_ptrs([W[0], W[0]], G)      # in-place outputs overlap (the C library's check)
    assert e.value.status in (lm.MALT_ERR_ALIAS, lm.MALT_ERR_STATE_MISMATCH)
    with pytest.raises(lm.MaltError) as e:
        plan.step(W, G, lm.make_hparams(mu1=1.0))
    assert e.value.status == lm.MALT_ERR_INVALID_ARG
    with pytest.raises(lm.MaltError) as e:
        plan.step(W, G, lm.make_hparams(ns_steps=0))
    assert e.value.status == lm.MALT_ERR_INVALID_ARG
    with pytest.raises(lm.MaltError) as e:
        plan.step([W[0], G[1]], G)            # a param aliases a grad
    assert e.value.status == lm.MALT_ERR_ALIAS
    torch.cuda.synchronize()
    assert plan.t == 0
    assert torch.equal(plan.state, before)
    plan.step(W, G)
    torch.cuda.synchronize()
    assert plan.t == 1


def test_profile_counts_every_launch():
    import torch
    say("[runtime] profiling")
    shapes = [(256, 512), (512, 256)]
    plan = lm.Plan(shapes, "malt")
    W = to_dev([wl.weight(98, i, s) for i, s in enumerate(shapes)])
    plan.profile_enable(True)
    for t in (1, 2):
        plan.step(W, to_dev([wl.grad(98, t, i, s) for i, s in enumerate(shapes)]))
    torch.cuda.synchronize()
    prof = plan.profile_read()
    assert prof["ns_gram"]["launches"] == 10 and prof["ns_update"]["launches"] == 10
    assert prof["momentum_rowcol"]["launches"] == 2 and prof["backmap_write"]["launches"] == 2
    assert all(v["ms"] >= 0 for v in prof.values())
    assert prof["ns_update"]["flops"] == 5 * 2.0 * 2 * 256 * 256 * 512
    again = plan.profile_read()
    assert again["ns_gram"]["launches"] == 0


def test_binding_rejects_tensors_the_c_abi_cannot_check():
    import torch
    say("[runtime] binding tensor checks")
    shapes = [(64, 96), (96, 64)]
    plan = lm.Plan(shapes, "malt")
    W = to_dev([wl.weight(96, i, s) for i, s in enumerate(shapes)])
    G = to_dev([wl.grad(96, 1, i, s) for i, s in enumerate(shapes)])
    bad = [
        ([W[0].double(), W[1]], G),                      # dtype
        ([W[0].t().contiguous().t(), W[1]], G),          # non-contiguous (transposed view)
        (W, [G[0], G[1].reshape(64, 96)]),               # shape
        ([W[0].cpu(), W[1]], G),                         # device
    ]
    for params, grads in bad:
        with pytest.raises(ValueError):
            plan.step(params, grads)
    torch.cuda.synchronize()
    assert plan.t == 0
    plan.step(W, G)
    torch.cuda.synchronize()
    assert plan.t == 1


def test_non_finite_gradient_stays_in_its_matrix():
    """NaN/Inf propagate without checks, but only inside the matrix that has
    them: every other matrix of the grouped step is bitwise the same as in a
    step without the bad gradient."""
    import torch
    say("[runtime] NaN gradient confined to its matrix")
    shapes = [(256, 512), (512, 256), (300, 700), (5, 40)]
    W0 = [wl.weight(95, i, s) for i, s in enumerate(shapes)]
    G = [wl.grad(95, 1, i, s) for i, s in enumerate(shapes)]
    bad = [g.copy() for g in G]
    bad[2][7, 11] = np.nan
    outs = []
    for grads in (G, bad):
        plan = lm.Plan(shapes, "malter")
        W = to_dev(W0)
        plan.step(W, to_dev(grads))
        torch.cuda.synchronize()
        outs.append([w.cpu().numpy() for w in W])
        plan.close()
    for k in (0, 1, 3):
        assert np.array_equal(outs[0][k], outs[1][k])
    assert not np.all(np.isfinite(outs[1][2]))


def test_concurrent_plans_on_two_streams_match_a_single_plan():
    # Plans share no device state: two plans stepping at the same time on two
    # streams (default priority) give bitwise the results of one plan alone.
    import torch
    shapes = [(700, 1500), (1500, 300), (64, 5000), (20, 3000)]
    say(f"[runtime] two plans on two streams {shapes}")
    W0 = [wl.weight(94, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(94, t, i, s, "row_loguniform") for i, s in enumerate(shapes)] for t in (1, 2, 3)]
    hp = lm.make_hparams(lr=3e-3)

    ref = lm.Plan(shapes, "malter")
    Wr = to_dev(W0)
    for g in grads:
        ref.step(Wr, to_dev(g), hp)
    torch.cuda.synchronize()

    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    plans = [lm.Plan(shapes, "malter", stream=st) for st in streams]
    Ws = [to_dev(W0), to_dev(W0)]
    Gs = [[to_dev(g) for g in grads], [to_dev(g) for g in grads]]
    torch.cuda.synchronize()
    for t in range(len(grads)):
        for k in range(2):
            with torch.cuda.stream(streams[k]):
                plans[k].step(Ws[k], Gs[k][t], hp, stream=streams[k])
    torch.cuda.synchronize()
    for k in range(2):
        for i in range(len(shapes)):
            assert torch.equal(Ws[k][i], Wr[i]), f"plan {k}, matrix {i} differs from the single-plan run"
    for pl in plans + [ref]:
        pl.close()


def test_precond_condition_matches_the_state_and_the_oracle():
    """kappa(diag l), kappa(diag r) per matrix: exactly max/min of the state's
    l and r, within the state bar of the oracle's, +inf for a zero row or a
    plan that has not stepped; argument errors are refused on the host."""
    import ctypes
    import torch
    from gpu_harness import run_oracle
    shapes = [(300, 900), (1024, 256), (17, 5)]
    say(f"[runtime] preconditioner condition numbers {shapes}")
    W0 = [wl.weight(97, i, s) for i, s in enumerate(shapes)]
    grads = [[wl.grad(97, t, i, s, "row_loguniform") for i, s in enumerate(shapes)] for t in (1, 2, 3)]
    for Gs in grads:
        Gs[2][4, :] = 0.0   # l_4 of the third matrix stays 0
    plan = lm.Plan(shapes, "malt")
    assert np.all(np.isinf(plan.precond_condition().cpu().numpy()))   # l = r = 0 before any step
    Wd = to_dev(W0)
    for Gs in grads:
        plan.step(Wd, to_dev(Gs), lm.make_hparams(lr=1e-3))
    kap = plan.precond_condition().cpu().numpy()
    o = run_oracle(shapes, "malt", W0, grads, dict(lr=1e-3))
    for i in range(len(shapes)):
        _, l, r, _ = plan.state_views(i)
        for j, (v, vo) in enumerate(((l, o[-1]["l"][i]), (r, o[-1]["r"][i]))):
            v = v.double().cpu().numpy()
            assert kap[i, j] == (v.max() / v.min() if v.min() > 0 else np.inf)
            if vo.min() == 0:
                assert np.isinf(kap[i, j])
            else:
                assert abs(kap[i, j] / (vo.max() / vo.min()) - 1.0) <= 1e-5
    assert np.isinf(kap[2, 0]) and np.isfinite(kap[2, 1])
    # Row scales over three decades spread l (squared: six) and leave r flat.
    assert np.all(kap[:2, 0] > 1e4) and np.all(kap[:2, 1] < 10.0)
    say(f"[runtime] kappa {kap.tolist()}")
    out = torch.empty(8, dtype=torch.float64, device=plan.device)
    f = lm.lib().malt_precond_condition
    assert f(plan._h, None, None) == lm.MALT_ERR_INVALID_ARG
    assert f(plan._h, ctypes.c_void_p(out.data_ptr() + 4), None) == lm.MALT_ERR_ALIGNMENT
    assert f(plan._h, ctypes.c_void_p(plan.state.data_ptr()), None) == lm.MALT_ERR_ALIAS
    torch.cuda.synchronize()
    plan.close()
