"""Pins of the float64 oracle against things other than itself.

Each test checks the oracle against what the paper or the mathematics fixes:
hand-derived worked examples (tests/golden), brute-force inversion of the
explicitly accumulated factor, closed forms, exact rational arithmetic,
library routines, and the paper's lemmas as invariants.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from tests.golden import load as load_golden

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _f(M):
    return np.array([[float(v) for v in r] for r in M], dtype=np.float64)


def _spd(rng, d, scale=1.0):
    Q = rng.standard_normal((d, d))
    return scale * (np.eye(d) + Q @ Q.T / d)


# ---------------------------------------------------------------- golden fixtures

@pytest.mark.parametrize("name", ["sm_exact_2x2.txt", "sm_exact_stab_2x2.txt", "sm_paper_eq6_2x2.txt"])
def test_golden_sm_step(name):
    g = load_golden(name)
    variant = O.EXACT if g["variant"] == "exact" else O.PAPER_EQ6
    p = O.Params(gamma=float(g["gamma"]), zeta=float(g["zeta"]), eps=float(g["eps"]),
                 variant=variant)
    P1, st = O.update_factor(_f(g["P0"]), np.array([float(v) for v in g["x"]]), p)
    np.testing.assert_allclose(P1, _f(g["P1"]), rtol=0, atol=1e-14)
    assert st.stab == bool(g["stab"])
    assert st.s == pytest.approx(float(g["s"]), abs=1e-14)


def test_golden_precond_rescale():
    g = load_golden("precond_rescale_2x2.txt")
    Linv, Rinv, G = _f(g["Linv"]), _f(g["Rinv"]), _f(g["G"])
    dW_hat = O.precondition(Linv, G, Rinv)
    np.testing.assert_array_equal(dW_hat, _f(g["dW_hat"]))
    dW, nG, nD, sc = O.rescale(G, dW_hat)
    assert nG == pytest.approx(float(g["norm_G"]), abs=1e-15)
    assert nD * nD == pytest.approx(float(g["norm_dW_hat_sq"]), rel=1e-15)
    assert sc * sc == pytest.approx(float(g["scale_sq"]), rel=1e-15)
    np.testing.assert_allclose(dW, math.sqrt(2) / 5 * _f(g["dW_hat"]), rtol=1e-15)


def test_golden_norms():
    g = load_golden("norm_2x2.txt")
    P = _f(g["P"])
    assert O.factor_norm(P, O.NORM_INF) == float(g["norm_inf"])
    assert O.factor_norm(P, O.NORM_MAXABS) == float(g["norm_maxabs"])


# ---------------------------------------------------------------- library routines

@pytest.mark.parametrize("d", [1, 3, 17, 64])
def test_norm_matches_numpy_linalg(d):
    rng = np.random.default_rng(d)
    P = rng.standard_normal((d, d))
    assert O.factor_norm(P, O.NORM_INF) == pytest.approx(np.linalg.norm(P, np.inf), rel=1e-15)
    assert O.factor_norm(P, O.NORM_MAXABS) == pytest.approx(np.linalg.norm(P.ravel(), np.inf), rel=0)


# ---------------------------------------------------------------- brute force (exact variant)

def _brute_force_run(d, steps, gamma, zeta, eps, seed, norm_kind=O.NORM_INF, xscale=1.0):
    """Accumulate M_t = gamma * M_hat_{t-1} + (1 - gamma) x x^T explicitly and
    invert it with numpy; the stabiliser decision is taken on inv(M) itself."""
    rng = np.random.default_rng(seed)
    M = np.eye(d)
    P = np.eye(d)
    p = O.Params(gamma=gamma, zeta=zeta, eps=eps, norm_kind=norm_kind, variant=O.EXACT)
    fired = 0
    for t in range(steps):
        x = rng.standard_normal(d) * xscale / math.sqrt(d)
        Minv = np.linalg.inv(M)
        nrm = (np.linalg.norm(Minv, np.inf) if norm_kind == O.NORM_INF
               else np.linalg.norm(Minv.ravel(), np.inf))
        if math.isfinite(eps) and abs(nrm - eps) <= 1e-9 * max(1.0, eps):
            pytest.skip("near-tie of the stabiliser threshold in brute force")
        if nrm > eps:
            M_hat = np.linalg.inv(zeta * Minv + (1 - zeta) * np.eye(d))
            fired += 1
        else:
            M_hat = M
        M = gamma * M_hat + (1 - gamma) * np.outer(x, x)
        P, st = O.update_factor(P, x, p)
        assert st.stab == (nrm > eps)
        ref = np.linalg.inv(M)
        rel = np.linalg.norm(P - ref) / np.linalg.norm(ref)
        cond = np.linalg.cond(M)
        assert rel <= 1e-12 * cond, (t, rel, cond)
        assert np.linalg.norm(P @ M - np.eye(d)) <= 1e-11 * cond
    return fired


@pytest.mark.parametrize("d", [1, 2, 5, 16, 64])
def test_exact_matches_inverse_of_accumulated_factor(d):
    _brute_force_run(d, 50, 0.9, 0.5, math.inf, seed=10 + d)


@pytest.mark.parametrize("d,eps,norm_kind", [(4, 3.0, O.NORM_INF), (16, 5.0, O.NORM_INF),
                                             (16, 2.5, O.NORM_MAXABS), (64, 8.0, O.NORM_INF)])
def test_exact_with_stabiliser_matches_brute_force(d, eps, norm_kind):
    fired = _brute_force_run(d, 50, 0.9, 0.5, eps, seed=100 + d, norm_kind=norm_kind)
    assert fired > 0, "stabiliser never fired: the test would not pin it"


def test_closed_form_repeated_vector():
    """Repeated x from P_0 = I: M_t = gamma^t I + (1 - gamma^t) x x^T, whose
    inverse is gamma^-t (I - (1 - gamma^t) x x^T / (gamma^t + (1 - gamma^t) |x|^2))."""
    rng = np.random.default_rng(7)
    d, gamma = 12, 0.9
    x = rng.standard_normal(d)
    P = np.eye(d)
    p = O.Params(gamma=gamma, eps=math.inf)
    for t in range(1, 31):
        P, _ = O.update_factor(P, x, p)
        gt = gamma ** t
        ref = (np.eye(d) - (1 - gt) * np.outer(x, x) / (gt + (1 - gt) * (x @ x))) / gt
        assert np.linalg.norm(P - ref) / np.linalg.norm(ref) < 1e-13


def test_scalar_case():
    """d = 1: the factor is a number, p_t = 1 / (gamma / p_{t-1} + (1 - gamma) x^2)."""
    rng = np.random.default_rng(3)
    p = O.Params(gamma=0.8, eps=math.inf)
    P = np.array([[1.0]])
    q = 1.0
    for _ in range(40):
        x = rng.standard_normal(1)
        P, _ = O.update_factor(P, x, p)
        q = 1.0 / (0.8 / q + 0.2 * x[0] ** 2)
        assert P[0, 0] == pytest.approx(q, rel=1e-14)


def test_zero_vector():
    rng = np.random.default_rng(5)
    P = _spd(rng, 6)
    x = np.zeros(6)
    P1, _ = O.update_factor(P, x, O.Params(gamma=0.9, eps=math.inf, variant=O.EXACT))
    np.testing.assert_allclose(P1, P / 0.9, rtol=1e-15)
    P2, _ = O.update_factor(P, x, O.Params(gamma=0.9, eps=math.inf, variant=O.PAPER_EQ6))
    np.testing.assert_allclose(P2, 0.9 * P, rtol=1e-15)


def _frac_inv(M):
    """Gauss-Jordan inverse over the rationals."""
    n = len(M)
    A = [list(r) + [Fraction(int(i == j)) for j in range(n)] for i, r in enumerate(M)]
    for c in range(n):
        piv = next(r for r in range(c, n) if A[r][c] != 0)
        A[c], A[piv] = A[piv], A[c]
        inv = 1 / A[c][c]
        A[c] = [v * inv for v in A[c]]
        for r in range(n):
            if r != c and A[r][c] != 0:
                f = A[r][c]
                A[r] = [vr - f * vc for vr, vc in zip(A[r], A[c])]
    return [r[n:] for r in A]


@pytest.mark.parametrize("n", [2, 3])
def test_exact_rational_accumulation(n):
    """Exact rational run: explicit accumulation + rational inverse vs the oracle."""
    rng = np.random.default_rng(n)
    gamma = Fraction(3, 4)
    M = [[Fraction(int(i == j)) for j in range(n)] for i in range(n)]
    P = np.eye(n)
    p = O.Params(gamma=float(gamma), eps=math.inf)
    for _ in range(6):
        xi = [int(v) for v in rng.integers(-3, 4, size=n)]
        M = [[gamma * M[i][j] + (1 - gamma) * xi[i] * xi[j] for j in range(n)] for i in range(n)]
        P, _ = O.update_factor(P, np.array(xi, dtype=np.float64), p)
        ref = np.array([[float(v) for v in r] for r in _frac_inv(M)])
        np.testing.assert_allclose(P, ref, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- invariants (Lemma 1, symmetry)

@pytest.mark.parametrize("variant", [O.EXACT, O.PAPER_EQ6])
def test_factors_stay_spd_and_symmetric(variant):
    rng = np.random.default_rng(11)
    d = 24
    P = np.eye(d)
    p = O.Params(gamma=0.9, zeta=0.5, eps=20.0, variant=variant)
    for _ in range(50):
        x = rng.standard_normal(d) / math.sqrt(d)
        P, _ = O.update_factor(P, x, p)
        np.testing.assert_allclose(P, P.T, rtol=0, atol=1e-12 * np.abs(P).max())
        np.linalg.cholesky(0.5 * (P + P.T))  # raises if not positive definite


# ---------------------------------------------------------------- stabiliser (Eq. 11)

def test_stabiliser_blend_matches_eq11_expansion():
    """(zeta A + (1-zeta) I) G (zeta B + (1-zeta) I)
       = zeta^2 A G B + zeta (1-zeta) (A G + G B) + (1-zeta)^2 G   (Eq. 11)."""
    rng = np.random.default_rng(21)
    d_in, d_out, zeta = 5, 7, 0.3
    A, B = _spd(rng, d_in), _spd(rng, d_out)
    G = rng.standard_normal((d_in, d_out))
    A_hat, fa = O.stabilize(A, O.factor_norm(A), 0.0, zeta)
    B_hat, fb = O.stabilize(B, O.factor_norm(B), 0.0, zeta)
    assert fa and fb
    lhs = O.precondition(A_hat, G, B_hat)
    rhs = zeta ** 2 * A @ G @ B + zeta * (1 - zeta) * (A @ G + G @ B) + (1 - zeta) ** 2 * G
    np.testing.assert_allclose(lhs, rhs, rtol=1e-13, atol=1e-13)


def test_stabiliser_thresholds():
    rng = np.random.default_rng(22)
    P = _spd(rng, 6)
    nu = O.factor_norm(P)
    Pi, f = O.stabilize(P, nu, math.inf, 0.5)
    assert not f and Pi is P
    P0, f = O.stabilize(P, nu, 0.0, 0.5)
    assert f
    P1, f = O.stabilize(P, nu, 0.0, 1.0)          # zeta = 1 is a no-op blend
    assert f
    np.testing.assert_array_equal(P1, P)
    _, f = O.stabilize(P, nu, nu, 0.5)            # strict '>'
    assert not f
    # stabilised update with x = 0: P_1 = P_hat / gamma
    P2, st = O.update_factor(P, np.zeros(6), O.Params(gamma=0.9, zeta=0.25, eps=0.0))
    assert st.stab
    np.testing.assert_allclose(0.9 * P2, 0.25 * P + 0.75 * np.eye(6), rtol=1e-14)


# ---------------------------------------------------------------- precondition / rescale

def test_precondition_matches_kronecker_form():
    """vec(L G R) = (R^T kron L) vec(G) with column-major vec; non-symmetric
    L and R so that a transposed operand or a swapped side fails."""
    rng = np.random.default_rng(31)
    L, R = rng.standard_normal((3, 3)), rng.standard_normal((4, 4))
    G = rng.standard_normal((3, 4))
    lhs = O.precondition(L, G, R).ravel(order="F")
    rhs = np.kron(R.T, L) @ G.ravel(order="F")
    np.testing.assert_allclose(lhs, rhs, rtol=1e-13, atol=1e-13)


def test_identity_and_scalar_factors_give_gradient():
    rng = np.random.default_rng(32)
    G = rng.standard_normal((6, 9))
    np.testing.assert_array_equal(O.precondition(np.eye(6), G, np.eye(9)), G)
    dW, *_ = O.rescale(G, O.precondition(3.0 * np.eye(6), G, 0.125 * np.eye(9)))
    np.testing.assert_allclose(dW, G, rtol=1e-15)


def test_rescale_norm_and_descent():
    """The rescaled update keeps the gradient norm (rescale line) and is a
    descent direction for SPD factors (Lemma 3)."""
    rng = np.random.default_rng(33)
    for _ in range(10):
        L, R = _spd(rng, 8), _spd(rng, 5)
        G = rng.standard_normal((8, 5))
        dW, nG, nD, sc = O.rescale(G, O.precondition(L, G, R))
        assert np.linalg.norm(dW) == pytest.approx(np.linalg.norm(G), rel=1e-14)
        assert float(np.sum(G * dW)) > 0
    dW, _, nD, sc = O.rescale(G, np.zeros_like(G))
    assert nD == 0 and sc == 0 and not dW.any()


# ---------------------------------------------------------------- layer-level wiring

def test_layer_pairs_a_with_left_and_g_with_right():
    rng = np.random.default_rng(41)
    d_in, d_out = 3, 5
    a, g = rng.standard_normal(d_in), rng.standard_normal(d_out)
    G = rng.standard_normal((d_in, d_out))
    p = O.Params(gamma=0.9, eps=math.inf)
    Li, Ri, dW, st = O.layer_step(np.eye(d_in), np.eye(d_out), a, g, G, p)
    ML = 0.9 * np.eye(d_in) + 0.1 * np.outer(a, a)
    MR = 0.9 * np.eye(d_out) + 0.1 * np.outer(g, g)
    np.testing.assert_allclose(Li, np.linalg.inv(ML), rtol=1e-13)
    np.testing.assert_allclose(Ri, np.linalg.inv(MR), rtol=1e-13)
    ref = np.linalg.inv(ML) @ G @ np.linalg.inv(MR)
    ref *= np.linalg.norm(G) / np.linalg.norm(ref)
    np.testing.assert_allclose(dW, ref, rtol=1e-13, atol=1e-15)


def test_first_order_layer_passes_gradient():
    rng = np.random.default_rng(42)
    G = rng.standard_normal((4, 6))
    Li, Ri, dW, st = O.layer_step(2 * np.eye(4), np.eye(6), np.ones(4), np.ones(6), G,
                                  O.Params(), second_order=False)
    np.testing.assert_array_equal(dW, G)
    np.testing.assert_array_equal(Li, 2 * np.eye(4))


def test_guard_nonfinite():
    G = np.ones((3, 3))
    a = np.array([1.0, np.nan, 0.0])
    p = O.Params(gamma=0.9, eps=math.inf, guard_nonfinite=True)
    Li, Ri, dW, st = O.layer_step(np.eye(3), np.eye(3), a, np.ones(3), G, p)
    assert st.L.skipped and st.nonfinite & O.NONFINITE_L
    np.testing.assert_array_equal(Li, np.eye(3))
    assert np.isfinite(dW).all()
    p.guard_nonfinite = False
    Li, Ri, dW, st = O.layer_step(np.eye(3), np.eye(3), a, np.ones(3), G, p)
    assert np.isnan(Li).any()


# ------------------------------------------------------------------ rank-1 means
def test_rank1_means_exact_rationals():
    """Integer rows: the mean is computed exactly (Fraction arithmetic by hand)."""
    rows = np.array([[3, -1, 7], [5, 2, -7], [-2, 2, 0], [6, 1, 4]], dtype=np.float64)
    want = [Fraction(3 + 5 - 2 + 6, 4), Fraction(-1 + 2 + 2 + 1, 4), Fraction(7 - 7 + 0 + 4, 4)]
    got = O.rank1_means(rows)
    assert [Fraction(x) for x in got] == want


def test_rank1_means_identical_rows_make_the_approximation_exact():
    """Algorithm 1 approximates the covariance (1/b) A^T A by a a^T; for b identical
    samples the two are equal, and the mean is the sample itself."""
    rng = np.random.default_rng(3)
    x = rng.integers(-1000, 1000, size=9) / 64.0   # few mantissa bits: every partial sum is exact
    rows = np.tile(x, (16, 1))
    a = O.rank1_means(rows)
    np.testing.assert_array_equal(a, x)
    cov = rows.T @ rows / rows.shape[0]
    np.testing.assert_allclose(np.outer(a, a), cov, rtol=1e-14, atol=1e-14)


def test_rank1_means_invariances():
    rng = np.random.default_rng(4)
    R = rng.standard_normal((37, 11))
    a = O.rank1_means(R)
    # duplicating every sample leaves the mean unchanged; row order does not matter
    np.testing.assert_allclose(O.rank1_means(np.vstack([R, R])), a, rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(O.rank1_means(R[::-1]), a, rtol=1e-14, atol=1e-15)
    # one sample: the mean is that sample; a shifted copy shifts the mean
    np.testing.assert_array_equal(O.rank1_means(R[:1]), R[0])
    np.testing.assert_allclose(O.rank1_means(R + 2.5), a + 2.5, rtol=1e-14, atol=1e-14)
    # samples that cancel in adjacent pairs have mean zero (each pair sums exactly)
    pairs = np.empty((2 * R.shape[0], R.shape[1]))
    pairs[0::2], pairs[1::2] = R, -R
    np.testing.assert_array_equal(O.rank1_means(pairs), np.zeros(11))


def test_layer_step_rows_uses_row_means():
    rng = np.random.default_rng(5)
    d_in, d_out, b = 6, 4, 10
    A = rng.standard_normal((b, d_in))
    Go = rng.standard_normal((b, d_out)) * 1e-3
    G = rng.standard_normal((d_in, d_out)) * 1e-3
    p = O.Params(gamma=0.9, eps=math.inf)
    Li, Ri, dW, st, a, g = O.layer_step_rows(np.eye(d_in), np.eye(d_out), A, Go, G, p)
    a2 = A.sum(axis=0) / b
    g2 = Go.sum(axis=0) / b
    np.testing.assert_allclose(a, a2, rtol=1e-14)
    np.testing.assert_allclose(g, g2, rtol=1e-14)
    Lj, Rj, dWj, _ = O.layer_step(np.eye(d_in), np.eye(d_out), a2, g2, G, p)
    np.testing.assert_allclose(Li, Lj, rtol=1e-12)
    np.testing.assert_allclose(dW, dWj, rtol=1e-12)
    with pytest.raises(ValueError):
        O.rank1_means(np.zeros((0, 3)))


# ---------------------------------------------------------------- the grouped step

def test_oracle_step_grouped_against_brute_force():
    """oracle_step over a list (Algorithm 1, "for each layer"): a mixed
    second_order list, a stabiliser override on one factor of one layer, and
    the update / precondition halves run separately, each layer checked
    against the explicit inverse of its explicitly accumulated factors (and a
    first-order layer against its gradient), over two steps."""
    rng = np.random.default_rng(2306)
    gamma, zeta = 0.9, 0.5
    p = O.Params(gamma=gamma, zeta=zeta, eps=math.inf)
    shapes = [(5, 3), (4, 6), (3, 7)]
    so = [True, False, True]
    layers = []
    M = []   # explicit factors (inverses of the inverse factors)
    for (i, o), s in zip(shapes, so):
        P0L, P0R = np.eye(i), np.linalg.inv(_spd(rng, o, 0.5))
        layers.append(dict(Linv=P0L, Rinv=P0R, second_order=s))
        M.append([np.linalg.inv(P0L), np.linalg.inv(P0R)])
    for step in range(2):
        for L, (i, o) in zip(layers, shapes):
            L["a"], L["g"] = rng.standard_normal(i), rng.standard_normal(o) * 0.3
            L["G"] = rng.standard_normal((i, o))
        # only layer 2's right factor is blended on step 0
        ov = [(None, None), (None, None), (None, step == 0)]
        half = O.oracle_step(layers, p, update=True, precond=False, stab_overrides=ov)
        mid = [dict(L, Linv=h["Linv"], Rinv=h["Rinv"]) for L, h in zip(layers, half)]
        pre = O.oracle_step(mid, p, update=False, precond=True)
        full = O.oracle_step(layers, p, stab_overrides=ov)
        for k, ((i, o), L) in enumerate(zip(shapes, layers)):
            assert half[k]["dW"] is None
            np.testing.assert_array_equal(pre[k]["dW"], full[k]["dW"])
            if not so[k]:
                np.testing.assert_array_equal(full[k]["dW"], L["G"])
                np.testing.assert_array_equal(full[k]["Linv"], L["Linv"])
                np.testing.assert_array_equal(full[k]["Rinv"], L["Rinv"])
                continue
            new = []
            for side, x in ((0, L["a"]), (1, L["g"])):
                Mh = M[k][side]
                if ov[k][side]:
                    Mh = np.linalg.inv(zeta * np.linalg.inv(Mh) + (1 - zeta) * np.eye(len(x)))
                M[k][side] = gamma * Mh + (1 - gamma) * np.outer(x, x)
                new.append(np.linalg.inv(M[k][side]))
            assert full[k]["stats"].R.stab == bool(ov[k][1])
            np.testing.assert_allclose(full[k]["Linv"], new[0], rtol=0, atol=1e-12)
            np.testing.assert_allclose(full[k]["Rinv"], new[1], rtol=0, atol=1e-12)
            dW_hat = new[0] @ L["G"] @ new[1]
            ref = np.linalg.norm(L["G"]) / np.linalg.norm(dW_hat) * dW_hat
            np.testing.assert_allclose(full[k]["dW"], ref, rtol=0, atol=1e-12)
        for L, f in zip(layers, full):
            L["Linv"], L["Rinv"] = f["Linv"], f["Rinv"]
