"""The appendix's matrix quadratic regression: the problem generator and the
exact-whitening comparison, pinned on the CPU; libmalt runs on the GPU."""
import numpy as np
import pytest

from paper_2608_05088_amd.toy import make_problem, run_polar_muon, run_whitened


@pytest.mark.parametrize("kappa", [10.0, 1e2, 1e3, 1e4])
def test_problem_has_the_prescribed_hessian_condition(kappa):
    p = make_problem(kappa)
    # Hessian in vec(X) is (B^T B) kron (A^T A): its extreme eigenvalues, directly.
    H = np.kron(p.B.T @ p.B, p.A.T @ p.A)
    w = np.linalg.eigvalsh(H)
    assert w[-1] / w[0] == pytest.approx(kappa, rel=1e-8)
    assert p.hessian_cond() == pytest.approx(kappa, rel=1e-8)
    # C lies in the model's range: the least-squares optimum has f* = 0, and f(0) = ||C||^2 / 2 = 1/2.
    assert p.f(p.lstsq()) < 1e-20 * kappa
    assert p.f(np.zeros((5, 5))) == pytest.approx(0.5, rel=1e-12)


def test_gradient_matches_finite_differences():
    p = make_problem(100.0)
    X = np.random.default_rng(3).standard_normal((5, 5))
    G = p.grad(X)
    h = 1e-6
    for i, j in [(0, 0), (1, 3), (4, 2)]:
        E = np.zeros_like(X)
        E[i, j] = h
        assert (p.f(X + E) - p.f(X - E)) / (2 * h) == pytest.approx(G[i, j], rel=1e-6, abs=1e-9)


def test_whitened_muon_does_not_see_the_condition_number():
    # With P = (A^T A)^(-1/2) and Q = (B^T B)^(-1/2), Y = P^(-1) X Q^(-1) follows
    # Y <- Y - eta Orth(Y - Y*) with ||Y*|| = ||S||: the same gap sequence for every
    # kappa, since only R1 and R2's singular values change with it.
    g10 = run_whitened(make_problem(10.0), 400)
    g1e4 = run_whitened(make_problem(1e4), 400)
    for t in g10:
        assert g1e4[t] == pytest.approx(g10[t], rel=1e-7, abs=1e-12)
    assert g10[400] < 0.5 * g10[0]


def test_polar_muon_slows_as_the_condition_number_grows():
    # The appendix's Muon (exact polar factor, no momentum) on the same
    # problems: its gap after 1000 steps grows with kappa, while the whitened
    # run's does not (the comparison its figure makes).
    gaps = [run_polar_muon(make_problem(k), 1000)[1000] for k in (10.0, 1e2, 1e3, 1e4)]
    assert all(a < b for a, b in zip(gaps, gaps[1:]))
    w = [run_whitened(make_problem(k), 1000)[1000] for k in (10.0, 1e4)]
    assert w[1] == pytest.approx(w[0], rel=1e-7, abs=1e-12) and w[0] < gaps[0]
    # One step at eta_max (a 1-step schedule is all plateau): X1 = -eta Orth(G0),
    # with Orth(G0) = G0 (G0^T G0)^(-1/2) written out from the eigenvalues.
    p = make_problem(1e3)
    G0 = p.grad(np.zeros((5, 5)))
    w_, V = np.linalg.eigh(G0.T @ G0)
    X1 = -1e-3 * G0 @ (V / np.sqrt(w_)) @ V.T
    assert run_polar_muon(p, 1)[1] == pytest.approx(p.f(X1) - p.f(p.lstsq()), rel=1e-10)


@pytest.mark.gpu
def test_libmalt_runs_the_toy():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_05088_amd.toy import run_libmalt
    print("[toy] libmalt muon / malt, kappa 10 and 1e4, 1000 steps", flush=True)
    res = {}
    for kappa in (10.0, 1e4):
        p = make_problem(kappa)
        for name in ("muon", "malt"):
            g = run_libmalt(p, 1000, name)
            assert all(np.isfinite(v) for v in g.values())
            assert g[1000] < g[0]
            res[(kappa, name)] = g[1000]
    print(f"[toy] gaps after 1000 steps: {res}", flush=True)
    # At kappa = 10 both at least halve the gap (f(0) = 1/2) within the 1000 steps.
    assert res[(10.0, "muon")] < 0.25 and res[(10.0, "malt")] < 0.25
    # The whole trajectory follows the fp64 oracle's over the same 1000 steps:
    # the NS rounding does not steer the run elsewhere.
    from oracle import OracleHparams, oracle_init, oracle_step
    from paper_2608_05088_amd.schedules import wsd
    for (kappa, name), gap in res.items():
        p = make_problem(kappa)
        st, X, sched = oracle_init([(5, 5)], "malt"), np.zeros((5, 5)), wsd(100, 700, 200)
        for t in range(1, 1001):
            hp = OracleHparams(lr=1e-3 * sched(t), precond_identity=(name == "muon"))
            X = oracle_step([X], [p.grad(X)], st, hp)[0][0]
        print(f"[toy] kappa {kappa:g} {name}: gap {gap:.4e}, oracle {p.f(X):.4e}", flush=True)
        assert gap == pytest.approx(p.f(X), rel=0.1)


@pytest.mark.gpu
@pytest.mark.parametrize("kappa", [10.0, 1e3, 1e4])
def test_libmalt_toy_steps_match_the_oracle(kappa):
    """Three MALT steps on the 5 x 5 toy, the gradients taken along the GPU's
    own trajectory and fed to the oracle as well.  A short side of 5 takes the
    fp32 Newton-Schulz path, so only the final bf16 rounding of O separates
    the two: dW errors of 1.2-1.9e-3 at kappa = 10, 1e3 and 1e4.  (At
    kappa = 1e3 the preconditioned momentum has five singular values spread
    over 50x, where the quintic is far from converged on the small ones; a
    bf16 iteration magnifies its own rounding there.)"""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from gpu_harness import TOL_NS, TOL_STATE, run_oracle
    from oracle import rel_fro
    from paper_2608_05088_amd import libmalt as lm
    print(f"[toy] libmalt vs oracle, kappa {kappa:g}, 3 steps", flush=True)
    p = make_problem(kappa)
    dev = torch.device("cuda:0")
    X = torch.zeros((5, 5), dtype=torch.float32, device=dev)
    plan = lm.Plan([(5, 5)], "malt", device=dev)
    hp = dict(lr=1e-2)
    grads, dW = [], []
    for _ in range(3):
        G = torch.from_numpy(p.grad(X.double().cpu().numpy()).astype(np.float32)).to(dev)
        grads.append([G.cpu().numpy()])
        before = X.double().cpu().numpy()
        plan.step([X], [G], lm.make_hparams(**hp))
        torch.cuda.synchronize()
        dW.append(X.double().cpu().numpy() - before)
    o = run_oracle([(5, 5)], "malt", [np.zeros((5, 5), np.float32)], grads, hp)
    errs = [rel_fro(dW[t], o[t]["inter"][0].dW) for t in range(3)]
    print(f"[toy] kappa {kappa:g} dW errors {errs}", flush=True)
    M, l, r, _ = plan.state_views(0)
    assert rel_fro(M.double().cpu().numpy(), o[2]["M"][0]) <= TOL_STATE
    assert rel_fro(l.double().cpu().numpy(), o[2]["l"][0]) <= TOL_STATE
    assert rel_fro(r.double().cpu().numpy(), o[2]["r"][0]) <= TOL_STATE
    assert max(errs) <= TOL_NS
