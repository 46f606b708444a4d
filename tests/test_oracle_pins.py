"""Pins of the fp64 oracle against facts the paper and the mathematics fix.

CPU only.  Each test checks the oracle against something other than itself:
closed forms of the recurrences, the spectral-mapping form of Newton-Schulz
(SVD), invariances the method has (or provably lacks), the paper's printed
state-memory table, and brute-force loops on tiny inputs.  A plausible slip
anywhere in the oracle (a dropped term, a wrong sign or exponent, an index on
the wrong axis, a transposed operand) fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import (NS_A, NS_B, NS_C, NS_EPS, NS_STEPS, OracleHparams, newton_schulz,
                    oracle_init, oracle_step, polar_svd, rel_fro)
from paper_2608_05088_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _p(x):
    """Scalar quintic written from the published coefficients (golden file)."""
    q = _load("muon_ns_quintic.json")
    return q["a"] * x + q["b"] * x ** 3 + q["c"] * x ** 5


def _phi(x, k=5):
    for _ in range(k):
        x = _p(x)
    return x


def _rand(shape, seed=0, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


# --------------------------------------------------------------------------
# Reading pins: the coefficients the oracle uses are the published ones.
# --------------------------------------------------------------------------

def test_ns_reading_matches_published_quintic():
    q = _load("muon_ns_quintic.json")
    assert (NS_A, NS_B, NS_C, NS_STEPS, NS_EPS) == (q["a"], q["b"], q["c"], q["steps"], q["norm_eps"])


def test_default_hparams_match_paper_table():
    hp = OracleHparams()
    t = _load("hyperparameters.json")["malt"]
    assert (hp.mu1, hp.mu2, hp.eps) == (t["mu1"], t["mu2"], t["eps"])
    lr = _load("hyperparameters.json")["optimal_lr"]
    W = workloads.WORKLOADS
    assert W[1].lr == lr["small"]["malt"] and W[2].lr == lr["small"]["malt"]
    assert W[3].lr == lr["medium"]["malter"]
    assert W[4].lr == lr["large"]["malt"]
    assert W[5].lr == lr["large"]["malter"]
    for w in W.values():
        assert (w.mu1, w.mu2, w.eps) == (t["mu1"], t["mu2"], t["eps"])


# --------------------------------------------------------------------------
# P1: momentum and row/column EMAs, closed forms and the l/r mass identity.
# --------------------------------------------------------------------------

def test_p1_constant_gradient_closed_form():
    m, n = 5, 7
    G = _rand((m, n), 1, 1e-2)
    st = oracle_init([(m, n)])
    hp = OracleHparams()
    W = [np.zeros((m, n))]
    for t in range(1, 8):
        W, _ = oracle_step(W, [G], st, hp)
        np.testing.assert_allclose(st.M[0], (1 - hp.mu1 ** t) * G, rtol=1e-13, atol=0)
        np.testing.assert_allclose(st.l[0], (1 - hp.mu2 ** t) * np.einsum("ij,ij->i", G, G), rtol=1e-12)
        np.testing.assert_allclose(st.r[0], (1 - hp.mu2 ** t) * np.einsum("ij,ij->j", G, G), rtol=1e-12)


def test_p1_row_and_column_mass_agree():
    # ||l_t||_1 = ||r_t||_1: both are the EMA of ||G||_F^2 (used in the proof of Thm. 1).
    shapes = [(3, 9), (8, 2)]
    st = oracle_init(shapes)
    hp = OracleHparams()
    W = [np.zeros(s) for s in shapes]
    for t in range(1, 5):
        Gs = [_rand(s, 10 * t + i, 10 ** (-i)) for i, s in enumerate(shapes)]
        W, _ = oracle_step(W, Gs, st, hp)
        for i in range(len(shapes)):
            assert math.isclose(st.l[i].sum(), st.r[i].sum(), rel_tol=1e-13)


def test_p1_bruteforce_tiny_loops():
    # Pure-Python loops over a 3x4 matrix for two steps, element by element.
    m, n = 3, 4
    G1 = _rand((m, n), 3, 0.1)
    G2 = _rand((m, n), 4, 0.1)
    hp = OracleHparams(lr=0.5)
    st = oracle_init([(m, n)])
    W0 = _rand((m, n), 5)
    Ws, _ = oracle_step([W0], [G1], st, hp)
    Ws, inter = oracle_step(Ws, [G2], st, hp)
    mu1, mu2, eps = hp.mu1, hp.mu2, hp.eps
    M = [[0.0] * n for _ in range(m)]
    l = [0.0] * m
    r = [0.0] * n
    for G in (G1, G2):
        for i in range(m):
            for j in range(n):
                M[i][j] = mu1 * M[i][j] + (1 - mu1) * G[i][j]
        for i in range(m):
            l[i] = mu2 * l[i] + (1 - mu2) * sum(G[i][j] ** 2 for j in range(n))
        for j in range(n):
            r[j] = mu2 * r[j] + (1 - mu2) * sum(G[i][j] ** 2 for i in range(m))
    Lv = [(x + eps) ** -0.125 for x in l]
    Rv = [(x + eps) ** -0.125 for x in r]
    for i in range(m):
        for j in range(n):
            assert math.isclose(st.M[0][i, j], M[i][j], rel_tol=1e-14)
            assert math.isclose(inter[0].M_tilde[i, j], Lv[i] * M[i][j] * Rv[j], rel_tol=1e-13)
            assert math.isclose(inter[0].D[i, j], Lv[i] * inter[0].O[i, j] * Rv[j], rel_tol=1e-13)
    np.testing.assert_allclose(inter[0].Lv, Lv, rtol=1e-14)
    np.testing.assert_allclose(inter[0].Rv, Rv, rtol=1e-14)


# --------------------------------------------------------------------------
# P2: preconditioner bounds.
# --------------------------------------------------------------------------

def test_p2_preconditioner_bounds():
    m, n = 6, 5
    G = _rand((m, n), 7, 1e-3)
    G[2, :] = 0.0       # a row that has always been zero
    G[:, 4] = 0.0       # a column that has always been zero
    st = oracle_init([(m, n)])
    hp = OracleHparams()
    W = [np.zeros((m, n))]
    for _ in range(3):
        W, inter = oracle_step(W, [G], st, hp)
    cap = hp.eps ** -0.125                  # ||L|| <= eps^(-1/8) = 10
    assert math.isclose(cap, 10.0, rel_tol=1e-15)
    for v in (inter[0].Lv, inter[0].Rv):
        assert np.all(v > 0) and np.all(v <= cap * (1 + 1e-15))
    assert inter[0].Lv[2] == pytest.approx(10.0, rel=1e-15)
    assert inter[0].Rv[4] == pytest.approx(10.0, rel=1e-15)
    # Larger accumulated row norm => smaller factor (monotone decreasing map).
    order = np.argsort(st.l[0])
    assert np.all(np.diff(inter[0].Lv[order]) <= 0)


def test_p2_uniform_rows_give_scalar_preconditioner():
    m, n = 8, 8
    H = np.array([[1.0]])
    while H.shape[0] < m:
        H = np.block([[H, H], [H, -H]])
    st = oracle_init([(m, n)])
    _, inter = oracle_step([np.zeros((m, n))], [0.01 * H], st, OracleHparams())
    assert np.ptp(inter[0].Lv) < 1e-15 * inter[0].Lv[0]
    assert np.ptp(inter[0].Rv) < 1e-15 * inter[0].Rv[0]


# --------------------------------------------------------------------------
# P3 / P4: Newton-Schulz closed forms, spectral map, equivariance, band.
# --------------------------------------------------------------------------

def test_p3_rectangular_diagonal_maps_entrywise():
    m, n = 5, 9
    d = np.array([0.9, -0.3, 0.05, 2.0, -1.1])
    X = np.zeros((m, n))
    X[np.arange(m), np.arange(m)] = d
    Y = newton_schulz(X)
    nrm = math.sqrt(sum(x * x for x in d)) + NS_EPS
    expect = np.zeros((m, n))
    for i in range(m):
        expect[i, i] = _phi(d[i] / nrm)
    np.testing.assert_allclose(Y, expect, rtol=1e-13, atol=1e-15)
    # Tall orientation: the transpose maps the same way.
    np.testing.assert_allclose(newton_schulz(X.T), expect.T, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("m,n", [(16, 40), (40, 16), (24, 24), (1, 12), (12, 1)])
def test_p3_semi_orthogonal_is_scaled(m, n):
    k = min(m, n)
    Q, _ = np.linalg.qr(_rand((max(m, n), k), 11))
    Q = Q if m >= n else Q.T          # m x n with orthonormal short side
    Y = newton_schulz(Q)
    s = _phi(1.0 / (math.sqrt(k) + NS_EPS))
    np.testing.assert_allclose(Y, s * Q, rtol=1e-12, atol=1e-14)


def test_p3_vector_case_value():
    x = _rand((1, 33), 12)
    Y = newton_schulz(x)
    scale = _phi(1.0 / (1.0 + NS_EPS / np.linalg.norm(x)))
    np.testing.assert_allclose(Y, scale * x / np.linalg.norm(x), rtol=1e-12)
    assert _phi(1.0) == pytest.approx(0.6964364095, abs=1e-10)


@pytest.mark.parametrize("m,n", [(7, 11), (11, 7), (9, 9)])
def test_p3_spectral_mapping_via_svd(m, n):
    X = _rand((m, n), 13)
    U, S, Vt = np.linalg.svd(X, full_matrices=False)
    expect = (U * _phi(S / (np.linalg.norm(X) + NS_EPS))) @ Vt
    np.testing.assert_allclose(newton_schulz(X), expect, rtol=1e-11, atol=1e-13)


def test_p3_orthogonal_equivariance():
    m, n = 10, 14
    X = _rand((m, n), 14)
    U, _ = np.linalg.qr(_rand((m, m), 15))
    V, _ = np.linalg.qr(_rand((n, n), 16))
    np.testing.assert_allclose(newton_schulz(U @ X @ V), U @ newton_schulz(X) @ V, atol=1e-12)


def test_p4_singular_values_land_in_band():
    # Normalised singular values >= 2e-3 end inside [p(x_min), p(x_max)], the
    # local minimum / maximum values of the quintic on (0, inf).
    a, b, c = NS_A, NS_B, NS_C
    crit = np.sqrt(np.roots([5 * c, 3 * b, a]).real)          # p'(x) = 0 in x^2
    lo, hi = sorted(_p(x) for x in crit)
    assert lo == pytest.approx(0.6818, abs=1e-4) and hi == pytest.approx(1.2024, abs=1e-4)
    m, n = 48, 96
    sv = np.geomspace(2e-3, 1.0, m)
    sv = sv / np.linalg.norm(sv)
    U, _ = np.linalg.qr(_rand((m, m), 17))
    V, _ = np.linalg.qr(_rand((n, m), 18))
    X = (U * sv) @ V.T
    S_out = np.linalg.svd(newton_schulz(X), compute_uv=False)
    assert S_out.max() <= hi + 1e-9
    keep = np.sort(sv)[::-1] * (1.0 / (1.0 + NS_EPS)) >= 2e-3
    assert np.all(S_out[keep] >= lo - 1e-9)


# --------------------------------------------------------------------------
# P5: exact-Orth mode.
# --------------------------------------------------------------------------

def test_p5_svd_mode_is_semi_orthogonal():
    m, n = 6, 10
    X = _rand((m, 3), 19) @ _rand((3, n), 20)      # rank 3
    O = polar_svd(X)
    S = np.linalg.svd(O, compute_uv=False)
    np.testing.assert_allclose(np.sort(S)[::-1][:3], 1.0, atol=1e-12)
    np.testing.assert_allclose(S[3:], 0.0, atol=1e-12)
    assert np.linalg.norm(O) == pytest.approx(math.sqrt(3), rel=1e-12)
    Of = polar_svd(_rand((m, n), 21))
    np.testing.assert_allclose(Of @ Of.T, np.eye(m), atol=1e-12)


# --------------------------------------------------------------------------
# P6: reduction to Muon; failure of orthogonal equivariance.
# --------------------------------------------------------------------------

def _muon_steps(W, Gs, lr, mu1, ns_eps=NS_EPS):
    """Muon (Sec. 3.1 update) with the EMA momentum of the algorithms."""
    M = np.zeros_like(W)
    for G in Gs:
        M = mu1 * M + (1 - mu1) * G
        W = W - lr * newton_schulz(M, eps=ns_eps)
    return W


def test_p6_identity_preconditioner_is_muon():
    m, n = 12, 20
    hp = OracleHparams(precond_identity=True, lr=0.01)
    Gs = [_rand((m, n), 30 + t, 1e-2) for t in range(3)]
    W0 = _rand((m, n), 29, 0.02)
    st = oracle_init([(m, n)])
    W = [W0]
    for G in Gs:
        W, inter = oracle_step(W, [G], st, hp)
        assert inter[0].graft == pytest.approx(1.0, abs=1e-7)
    np.testing.assert_allclose(W[0], _muon_steps(W0, Gs, hp.lr, hp.mu1), rtol=0, atol=1e-9)


def test_p6_uniform_norm_gradients_reduce_to_muon():
    # Sign matrices have equal row norms and equal column norms: L, R are
    # scalars, so the step is Muon's up to the eps terms.  With the NS
    # normalisation eps set to 0 only the graft eps (1e-8) remains.
    m, n = 8, 16
    rng = np.random.default_rng(31)
    Gs = [0.01 * (t + 1) * np.sign(rng.standard_normal((m, n))) for t in range(3)]
    W0 = _rand((m, n), 32, 0.02)
    for ns_eps, tol in ((0.0, 1e-9), (NS_EPS, 1e-4)):
        hp = OracleHparams(lr=0.01, ns_eps=ns_eps)
        st = oracle_init([(m, n)])
        W = [W0]
        for G in Gs:
            W, _ = oracle_step(W, [G], st, hp)
        assert rel_fro(W[0] - W0, _muon_steps(W0, Gs, hp.lr, hp.mu1, ns_eps) - W0) < tol


def test_p6_not_orthogonally_equivariant():
    m, n = 8, 12
    G = 1e-2 * _rand((m, n), 33) * (10.0 ** np.linspace(-2, 0, m))[:, None]
    U, _ = np.linalg.qr(_rand((m, m), 34))
    hp = OracleHparams(lr=1.0)
    _, a = oracle_step([np.zeros((m, n))], [U @ G], oracle_init([(m, n)]), hp)
    _, b = oracle_step([np.zeros((m, n))], [G], oracle_init([(m, n)]), hp)
    assert rel_fro(a[0].dW, U @ b[0].dW) > 1e-2
    # ...whereas Muon (identity preconditioner) is equivariant.
    hp_i = OracleHparams(lr=1.0, precond_identity=True)
    _, a = oracle_step([np.zeros((m, n))], [U @ G], oracle_init([(m, n)]), hp_i)
    _, b = oracle_step([np.zeros((m, n))], [G], oracle_init([(m, n)]), hp_i)
    assert rel_fro(a[0].dW, U @ b[0].dW) < 1e-10


# --------------------------------------------------------------------------
# P7: graft identity.   P8: MALTER stepsize.   P9: scale invariance.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_p7_graft_identity(variant):
    m, n = 9, 15
    hp = OracleHparams(variant=variant, lr=3e-3)
    st = oracle_init([(m, n)], variant)
    W = [_rand((m, n), 40)]
    for t in range(3):
        W, inter = oracle_step(W, [_rand((m, n), 41 + t, 1e-2)], st, hp)
        it = inter[0]
        nD = np.linalg.norm(it.D)
        expect = hp.lr * it.alpha * np.linalg.norm(it.O) * nD / (nD + hp.eps)
        assert np.linalg.norm(it.dW) == pytest.approx(expect, rel=1e-12)


def test_p8_malter_alpha_first_step_is_one():
    for seed in range(3):
        m, n = 6 + seed, 11
        st = oracle_init([(m, n)], "malter")
        _, inter = oracle_step([np.zeros((m, n))], [_rand((m, n), 50 + seed, 10.0 ** -seed)], st,
                               OracleHparams(variant="malter"))
        assert inter[0].alpha == pytest.approx(1.0, abs=1e-6)


def test_p8_malter_alpha_constant_gradient_closed_form():
    mu2 = 0.99

    def closed(t):
        c = lambda tau: (1 - mu2 ** tau) ** -0.25
        return math.sqrt(1 - mu2 ** t) * c(t) / math.sqrt(
            (1 - mu2) * sum(mu2 ** (t - tau) * c(tau) ** 2 for tau in range(1, t + 1)))

    assert closed(2) == pytest.approx(0.9112378763, abs=1e-10)
    m, n = 7, 13
    G = _rand((m, n), 60, 1.0)         # large enough that eps terms are ~1e-9
    hp = OracleHparams(variant="malter", mu2=mu2)
    st = oracle_init([(m, n)], "malter")
    W = [np.zeros((m, n))]
    for t in range(1, 11):
        W, inter = oracle_step(W, [G], st, hp)
        assert inter[0].alpha == pytest.approx(closed(t), rel=1e-6)


def test_p8_malt_constant_gradient_steps_repeat():
    m, n = 7, 13
    G = _rand((m, n), 61, 0.5)
    st = oracle_init([(m, n)])
    W = [np.zeros((m, n))]
    hp = OracleHparams(ns_eps=0.0)     # NS is then exactly scale-invariant
    W, first = oracle_step(W, [G], st, hp)
    for _ in range(4):
        W, inter = oracle_step(W, [G], st, hp)
        assert rel_fro(inter[0].dW, first[0].dW) < 1e-6   # eps terms only


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_p9_scale_invariance(variant):
    m, n = 10, 6
    hp = OracleHparams(variant=variant, ns_eps=0.0)   # only the 1e-8 damping terms remain
    outs = []
    for s in (1.0, 7.0):
        st = oracle_init([(m, n)], variant)
        W = [np.zeros((m, n))]
        for t in range(3):
            W, inter = oracle_step(W, [s * _rand((m, n), 70 + t, 1e-1)], st, hp)
        outs.append(inter[0].dW)
    assert rel_fro(outs[1], outs[0]) < 1e-5   # 1e-8 / (1 - mu1^t) etc.


# --------------------------------------------------------------------------
# P10: transposition / permutation / sign-flip equivariance.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_p10_transpose_equivariance(variant):
    m, n = 9, 14
    hp = OracleHparams(variant=variant)
    sa = oracle_init([(m, n)], variant)
    sb = oracle_init([(n, m)], variant)
    Wa, Wb = [np.zeros((m, n))], [np.zeros((n, m))]
    for t in range(3):
        G = _rand((m, n), 80 + t, 1e-2)
        Wa, ia = oracle_step(Wa, [G], sa, hp)
        Wb, ib = oracle_step(Wb, [G.T.copy()], sb, hp)
        np.testing.assert_allclose(ib[0].dW, ia[0].dW.T, rtol=1e-10, atol=1e-16)
        np.testing.assert_allclose(sb.l[0], sa.r[0], rtol=1e-14)


def test_p10_permutation_and_sign_equivariance():
    m, n = 8, 11
    rng = np.random.default_rng(90)
    P = np.eye(m)[rng.permutation(m)]
    Q = np.eye(n)[:, rng.permutation(n)]
    S = np.diag(np.where(rng.random(m) < 0.5, -1.0, 1.0))
    T = np.diag(np.where(rng.random(n) < 0.5, -1.0, 1.0))
    hp = OracleHparams(variant="malter")
    G = _rand((m, n), 91, 1e-2) * (10.0 ** np.linspace(-1, 0, n))[None, :]
    _, a = oracle_step([np.zeros((m, n))], [G], oracle_init([(m, n)], "malter"), hp)
    for left, right in ((P, Q), (S, T)):
        _, b = oracle_step([np.zeros((m, n))], [left @ G @ right], oracle_init([(m, n)], "malter"), hp)
        np.testing.assert_allclose(b[0].dW, left @ a[0].dW @ right, rtol=1e-10, atol=1e-16)


# --------------------------------------------------------------------------
# P11: state size reproduces the paper's memory table.
# --------------------------------------------------------------------------

def test_p11_state_memory_matches_paper_table():
    g = _load("state_memory_gpt2_medium.json")
    mb = g["optimizer_state_mb"]
    shapes = workloads.gpt2_matrix_shapes(24, 1024)
    assert list(shapes) == list(workloads.WORKLOADS[3].shapes)
    mn = sum(m * n for m, n in shapes)
    # MALT state mn+m+n vs Muon's mn: the paper's 1554.88 - 1553.38 MB gap.
    malt_vals = oracle_init(shapes, "malt").num_state_values()
    malter_vals = oracle_init(shapes, "malter").num_state_values()
    to_mb = lambda vals: vals * g["bytes_per_value"] / 2 ** 20
    assert round(to_mb(malt_vals - mn), 2) == round(mb["malt"] - mb["muon"], 2)
    assert round(to_mb(malter_vals - mn), 2) == round(mb["malter"] - mb["muon"], 2)
    # AdamW's 2mn vs Muon's mn: the 2705.38 - 1553.38 MB gap.
    assert round(to_mb(mn), 2) == round(mb["adamw"] - mb["muon"], 2)
    assert malter_vals - malt_vals == len(shapes)


# --------------------------------------------------------------------------
# P12: degenerate inputs.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_p12_zero_gradient_gives_zero_update(variant):
    shapes = [(4, 6), (1, 5), (5, 1)]
    st = oracle_init(shapes, variant)
    W0 = [_rand(s, 95 + i) for i, s in enumerate(shapes)]
    W, inter = oracle_step(W0, [np.zeros(s) for s in shapes], st, OracleHparams(variant=variant))
    for i in range(len(shapes)):
        assert np.all(np.isfinite(W[i]))
        np.testing.assert_array_equal(W[i], W0[i])
        assert inter[i].graft == 0.0
        if variant == "malter":
            assert inter[i].alpha == 0.0


def test_p12_vector_shapes_step():
    for shape in ((1, 17), (17, 1)):
        st = oracle_init([shape])
        G = _rand(shape, 97, 1e-2)
        _, inter = oracle_step([np.zeros(shape)], [G], st, OracleHparams())
        O = inter[0].O
        Mt = inter[0].M_tilde
        np.testing.assert_allclose(O, _phi(np.linalg.norm(Mt) / (np.linalg.norm(Mt) + NS_EPS))
                                   * Mt / np.linalg.norm(Mt), rtol=1e-12)


# P13: a scaled partial permutation keeps every stage entrywise, so the whole
# step is a closed form (tests/closed_forms.py, written from the update rule):
# the oracle must reproduce it, zero entries included.
@pytest.mark.parametrize("shape,k,variant", [((60, 90), 50, "malt"), ((90, 40), 40, "malter"), ((64, 64), 64, "malt")])
def test_p13_permutation_closed_form(shape, k, variant):
    from closed_forms import permutation_step, random_permutation_pattern
    m, n = shape
    rows, cols, g = random_permutation_pattern(m, n, k, seed=13)
    G = np.zeros((m, n), np.float32)
    G[rows, cols] = g.astype(np.float32)
    gg = G[rows, cols].astype(np.float64)
    st = oracle_init([shape], variant)
    hp = OracleHparams(variant=variant, lr=1e-3)
    W, inter = oracle_step([np.zeros((m, n))], [G], st, hp)
    l, r, Lv, Rv, dw = permutation_step(m, n, rows, cols, gg, variant, lr=1e-3)
    assert rel_fro(st.l[0], l) < 1e-12 and rel_fro(st.r[0], r) < 1e-12
    assert rel_fro(inter[0].Lv, Lv) < 1e-12 and rel_fro(inter[0].Rv, Rv) < 1e-12
    expect = np.zeros((m, n))
    expect[rows, cols] = dw
    assert rel_fro(W[0], expect) < 1e-9


# --------------------------------------------------------------------------
# P14: decoupled weight decay.  The algorithms omit it; the hyper-parameter
# table sets 0.1 and the paper cites decoupled weight decay (AdamW).  The
# oracle's reading is pinned to torch's AdamW, a library implementation of
# that rule: a multiplicative (1 - eta*lambda) shrink, applied before the
# optimizer's own update and independent of it.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_p14_zero_gradient_step_is_adamw_decay(variant):
    import torch
    shapes = [(5, 7), (7, 3)]
    lr, lam = 3e-2, 0.1
    W0 = [_rand(s, 140 + i) for i, s in enumerate(shapes)]
    W, _ = oracle_step(W0, [np.zeros(s) for s in shapes], oracle_init(shapes, variant),
                       OracleHparams(variant=variant, lr=lr, weight_decay=lam))
    ps = [torch.tensor(w, dtype=torch.float64, requires_grad=True) for w in W0]
    opt = torch.optim.AdamW(ps, lr=lr, weight_decay=lam)
    for p in ps:
        p.grad = torch.zeros_like(p)
    opt.step()
    for w, p in zip(W, ps):
        np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-15, atol=0)


@pytest.mark.parametrize("variant", ["malt", "malter"])
def test_p14_decay_precedes_and_separates_from_the_update(variant):
    shapes = [(6, 9), (9, 4)]
    lr, lam = 2e-2, 0.1
    W0 = [_rand(s, 150 + i) for i, s in enumerate(shapes)]
    G = [[_rand(s, 160 + 10 * t + i, 1e-2) for i, s in enumerate(shapes)] for t in range(3)]
    runs = {}
    for wd in (0.0, lam):
        st = oracle_init(shapes, variant)
        W, steps = [w.copy() for w in W0], []
        for t in range(3):
            Wn, _ = oracle_step(W, G[t], st, OracleHparams(variant=variant, lr=lr, weight_decay=wd))
            steps.append([wn - w for wn, w in zip(Wn, W)])
            W = Wn
        runs[wd] = (W, steps)
    # The direction does not depend on W, so with decay each step adds exactly
    # -eta*lambda*W_prev to the undecayed step; W_prev is the decayed iterate.
    W_prev = [w.copy() for w in W0]
    for t in range(3):
        for i in range(len(shapes)):
            np.testing.assert_allclose(runs[lam][1][t][i] - runs[0.0][1][t][i], -lr * lam * W_prev[i],
                                       rtol=1e-9, atol=1e-15)
        W_prev = [w + d for w, d in zip(W_prev, runs[lam][1][t])]
