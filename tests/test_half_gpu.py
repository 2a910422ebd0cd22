"""GPU parity of the half-precision (bf16) factor path against the half
oracle (oracle/half.py), through the C ABI, and against the fp32 path.

Bars (derived in the design notes from the arithmetic):
* dW after one step from the same stored factors: relative Frobenius error
  <= TOL_HALF_STEP.  The only source above fp32 rounding is the bf16 rounding
  of Y = G Rinv, which the kernel decides on an fp32 accumulation and the
  oracle on the exact value: an element near a rounding midpoint may land on
  the other neighbour, one bf16 ulp away.
* Stored factors after one step: each element must be the bf16 rounding of a
  value within delta of the oracle's unrounded update P, where delta bounds
  the fp32 evaluation error of the update: a few fp32 ulps of the magnitudes
  it combines (the previous factor, the rank-1 term, I when the stabiliser
  blends) plus the error of u = P_hat x accumulated over d terms, carried
  into k u u^T.  Where the terms cancel, delta exceeds an ulp of P; elsewhere
  this leaves the nearest bf16 value, or the other neighbour of a value
  within delta of the midpoint.
* After up to 50 independently accumulated steps: relative Frobenius error
  <= TOL_HALF_FREE on factors and dW.  Two bf16 trajectories that once take
  a different rounding decision drift apart at the scale of the quantisation
  itself (the next update spreads the one-ulp difference over the factor,
  where it flips further roundings): about 2^-9 relative per step, adding up
  like a random walk, sqrt(50) 2^-9 = 1.4e-2 after 50 steps.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from oracle.half import layer_step_half, round_bf16
from paper_2306_01685_amd import Params, harness as H, SM_PAPER_EQ6
from tests.parity import TOL_HALF_FREE, TOL_HALF_STEP, oparams, rel, spd

pytestmark = pytest.mark.gpu

NEAR_MID_ULPS = 16   # fp32 ulps of the update's term magnitude

# multiples of 64 (the bf16 path's requirement) that span several 256 x 128
# tiles with ragged edges in both tile dimensions
SHAPES = [(64, 64), (320, 192), (64, 448), (576, 320), (256, 128), (128, 704)]


def _bf16_spd(seed, d):
    return W.round_to_bf16(spd(seed, d))


def _inputs(seed, d_in, d_out, grad_dtype):
    rng = np.random.default_rng(seed)
    a = (rng.standard_normal(d_in) / math.sqrt(d_in)).astype(np.float32)
    g = (rng.standard_normal(d_out) / math.sqrt(d_out)).astype(np.float32)
    G = (rng.standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
    if grad_dtype == "bf16":
        G = W.round_to_bf16(G)
    return a, g, G


def _setup(shapes, grad_dtype, seed, factor_dtype="bf16"):
    layers = H.allocate_layers(shapes, grad_dtype, factor_dtype=factor_dtype)
    host = []
    for i, (L, (d_in, d_out)) in enumerate(zip(layers, shapes)):
        Li, Ri = _bf16_spd(seed * 7 + i, d_in), _bf16_spd(seed * 11 + i, d_out)
        a, g, G = _inputs(seed + i, d_in, d_out, grad_dtype)
        H.set_factors(L, Li, Ri)
        H.set_inputs(L, a, g, G)
        host.append((Li.astype(np.float64), Ri.astype(np.float64), a, g, G))
    return layers, host


def _ulp(v):
    """bf16 spacing at |v| (normal range)."""
    e = np.floor(np.log2(np.maximum(np.abs(v), 2.0 ** -126)))
    return 2.0 ** (e - 7)


def update_error_bound(Q, x, op, stab):
    """delta of the docstring above for one factor update from the stored Q
    (the oracle's update, with the stabiliser decision `stab`)."""
    d = Q.shape[0]
    P_hat = op.zeta * Q + (1.0 - op.zeta) * np.eye(d) if stab else Q
    x = np.asarray(x, np.float64)
    _, u, _, k = O.sm_update(P_hat, x, op.gamma, op.variant)
    a = np.abs(P_hat) @ np.abs(x)                   # magnitude summed into u
    g = max(op.gamma, 1.0 / op.gamma)
    terms = g * (np.abs(P_hat) + np.eye(d) + abs(k) * np.outer(np.abs(u), np.abs(u)))
    u_err = math.sqrt(d) * a                        # (in fp32 ulps) error of u
    cross = g * abs(k) * (np.outer(u_err, np.abs(u)) + np.outer(np.abs(u), u_err))
    return NEAR_MID_ULPS * 2.0 ** -24 * (terms + cross)


def check_stored(gpu, P_exact, delta, what):
    """Stored bf16 factor vs the oracle's unrounded update: every element is
    the bf16 rounding of a value within delta of P_exact.  Returns the fraction
    of elements that differ from round_bf16(P_exact)."""
    gv = gpu.astype(np.float64)
    err = np.abs(gv - P_exact)
    allowed = 0.5 * _ulp(np.abs(P_exact) + delta) + delta
    bad = err > allowed
    if bad.any():
        j = np.argmax(err / allowed)
        raise AssertionError((what, "stored value off", int(bad.sum()), float(P_exact.flat[j]), float(gv.flat[j]),
                              float(delta.flat[j]), float(_ulp(P_exact.flat[j]))))
    return float(np.mean(gv != round_bf16(P_exact)))


@pytest.mark.parametrize("grad_dtype,variant,eps", [("fp32", 0, math.inf), ("bf16", 0, math.inf),
                                                    ("bf16", 0, 0.0), ("fp32", SM_PAPER_EQ6, 0.0)])
def test_half_single_step(grad_dtype, variant, eps):
    layers, host = _setup(SHAPES, grad_dtype, seed=300 + variant)
    plan = H.make_plan(layers)
    p = Params(eps=eps, variant=variant)
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    op = oparams(p)
    flips = []
    for i, (L, (Li, Ri, a, g, G)) in enumerate(zip(layers, host)):
        PL, PR, dW, st = layer_step_half(Li, Ri, a, g, G, op)
        e = rel(H.get_dW(L), dW)
        print(i, L["d_in"], L["d_out"], "dW rel err", e)
        assert e <= TOL_HALF_STEP, (i, L["d_in"], L["d_out"], e)
        s = H.get_stats(L)
        assert s["norm_G"] == pytest.approx(st.norm_G, rel=1e-5)
        assert s["scale"] == pytest.approx(st.scale, rel=1e-3)
        assert bool(s["stab_L"]) == st.L.stab and bool(s["stab_R"]) == st.R.stab
        assert s["nu_L"] == pytest.approx(st.L.nu, rel=1e-5)
        Lg, Rg = H.get_factors(L)
        flips.append((check_stored(Lg, PL, update_error_bound(Li, a, op, st.L.stab), ("L", i)),
                      check_stored(Rg, PR, update_error_bound(Ri, g, op, st.R.stab), ("R", i))))
        print("   factor flip fraction", flips[-1])
    assert max(max(f) for f in flips) < 1e-2


def test_half_precondition_after_update_and_sync():
    """update_factors then two preconditionings use the fresh (unrounded)
    factors; after sync_factors the preconditioning uses the stored bf16 ones."""
    layers, host = _setup(SHAPES[:4], "bf16", seed=350)
    plan = H.make_plan(layers)
    p = Params(eps=math.inf)
    op = oparams(p)
    plan.update_factors(p)
    exp = []
    for Li, Ri, a, g, G in host:
        PL, PR, _, _ = layer_step_half(Li, Ri, a, g, G, op, precond=False)
        exp.append((PL, PR))
    for _ in range(2):
        plan.precondition(p)
        torch.cuda.synchronize()
        for L, (PL, PR), (_, _, a, g, G) in zip(layers, exp, host):
            _, _, dW, _ = layer_step_half(PL, PR, a, g, G, op, update=False)
            assert rel(H.get_dW(L), dW) <= TOL_HALF_STEP
    plan.sync_factors()
    plan.precondition(p)
    torch.cuda.synchronize()
    for L, (PL, PR), (_, _, a, g, G) in zip(layers, exp, host):
        Lg, Rg = H.get_factors(L)
        _, _, dW, _ = layer_step_half(Lg.astype(np.float64), Rg.astype(np.float64), a, g, G, op,
                                      update=False)
        assert rel(H.get_dW(L), dW) <= TOL_HALF_STEP


def test_half_mixed_plan():
    """bf16-factor, fp32-factor and first-order layers in one plan."""
    shapes = [(320, 192), (130, 250), (50, 70), (64, 448)]
    kinds = ["bf16", "fp32", "first", "bf16"]
    layers = []
    for (d_in, d_out), k in zip(shapes, kinds):
        layers += H.allocate_layers([(d_in, d_out)], "fp32", second_order=[k != "first"],
                                    factor_dtype="bf16" if k == "bf16" else "fp32")
    host = []
    for i, (L, (d_in, d_out), k) in enumerate(zip(layers, shapes, kinds)):
        a, g, G = _inputs(400 + i, d_in, d_out, "fp32")
        if k == "first":
            H.set_inputs(L, G=G)
            host.append((None, None, a, g, G))
            continue
        Li, Ri = _bf16_spd(410 + i, d_in), _bf16_spd(420 + i, d_out)
        H.set_factors(L, Li, Ri)
        H.set_inputs(L, a, g, G)
        host.append((Li.astype(np.float64), Ri.astype(np.float64), a, g, G))
    plan = H.make_plan(layers)
    p = Params(eps=1.0)
    op = oparams(p)
    plan.step(p)
    torch.cuda.synchronize()
    for L, k, (Li, Ri, a, g, G) in zip(layers, kinds, host):
        if k == "first":
            assert np.array_equal(H.get_dW(L), G)
        elif k == "bf16":
            _, _, dW, _ = layer_step_half(Li, Ri, a, g, G, op)
            assert rel(H.get_dW(L), dW) <= TOL_HALF_STEP
        else:
            _, _, dW, _ = O.layer_step(Li, Ri, a, g, G, op)
            assert rel(H.get_dW(L), dW) <= 1e-4


def _run_steps(layers, plan, host, p, steps, seed, oracle=True):
    """Steps the plan with fresh seeded (a, g, G) each step; the half oracle
    follows when asked.  Returns the oracle's final (PL, PR, dW) per layer."""
    op = oparams(p)
    state = [(Li, Ri) for Li, Ri, *_ in host]
    last = [None] * len(layers)
    for t in range(steps):
        for i, L in enumerate(layers):
            a, g, G = _inputs(seed + 1000 * t + i, L["d_in"], L["d_out"],
                              "bf16" if L["G"].dtype == torch.bfloat16 else "fp32")
            H.set_inputs(L, a, g, G)
            if oracle:
                PL, PR, dW, _ = layer_step_half(state[i][0], state[i][1], a, g, G, op)
                state[i] = (PL, PR)
                last[i] = dW
        plan.step(p)
    torch.cuda.synchronize()
    return state, last


def test_half_free_run_50_steps():
    layers, host = _setup(SHAPES, "bf16", seed=500)
    plan = H.make_plan(layers)
    p = Params(eps=100.0)
    state, last = _run_steps(layers, plan, host, p, 50, seed=510)
    plan.sync_factors()
    torch.cuda.synchronize()
    for i, L in enumerate(layers):
        Lg, Rg = H.get_factors(L)
        eL, eR = rel(Lg, round_bf16(state[i][0])), rel(Rg, round_bf16(state[i][1]))
        eD = rel(H.get_dW(L), last[i])
        print(i, L["d_in"], L["d_out"], "50-step errors L R dW", eL, eR, eD)
        assert max(eL, eR, eD) <= TOL_HALF_FREE, (i, eL, eR, eD)


def test_half_against_fp32_path():
    """Same inputs through the fp32-factor and the bf16-factor path: they
    differ by the bf16 quantisation (a few 2^-9 relative per step), not more."""
    shapes = SHAPES[1:4]
    lh, host = _setup(shapes, "fp32", seed=600, factor_dtype="bf16")
    lf, _ = _setup(shapes, "fp32", seed=600, factor_dtype="fp32")
    ph, pf = H.make_plan(lh), H.make_plan(lf)
    p = Params(eps=100.0)
    errs = []
    for t in range(20):
        for i, (a_, b_) in enumerate(zip(lh, lf)):
            a, g, G = _inputs(610 + 1000 * t + i, a_["d_in"], a_["d_out"], "fp32")
            H.set_inputs(a_, a, g, G)
            H.set_inputs(b_, a, g, G)
        ph.step(p)
        pf.step(p)
        torch.cuda.synchronize()
        errs.append(max(rel(H.get_dW(x), H.get_dW(y)) for x, y in zip(lh, lf)))
    print("bf16 vs fp32 factors, dW rel diff per step", errs)
    assert 1e-5 < errs[0] < 4 * 2.0 ** -9
    assert max(errs) < 5e-2


def test_half_bert_large_shapes_one_step():
    """The BERT-Large layer shapes with bf16 factors, in one grouped plan, one
    step against the half oracle."""
    shapes = [(1024, 1024), (1024, 4096), (4096, 1024)]
    layers, host = _setup(shapes, "bf16", seed=700)
    plan = H.make_plan(layers)
    p = Params(eps=100.0)
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    op = oparams(p)
    for i, (L, (Li, Ri, a, g, G)) in enumerate(zip(layers, host)):
        PL, PR, dW, st = layer_step_half(Li, Ri, a, g, G, op)
        e = rel(H.get_dW(L), dW)
        print(shapes[i], "dW rel err", e)
        assert e <= TOL_HALF_STEP
        Lg, Rg = H.get_factors(L)
        f = (check_stored(Lg, PL, update_error_bound(Li, a, op, st.L.stab), ("L", i)),
             check_stored(Rg, PR, update_error_bound(Ri, g, op, st.R.stab), ("R", i)))
        print("   flip fraction", f)


# ------------------------------------------------------------------ against full precision

def _trajectory(seed, d, steps=5, gamma=0.9):
    """A factor after a few float64 updates from I: not bf16-representable."""
    rng = np.random.default_rng(seed)
    P = np.eye(d)
    p = O.Params(gamma=gamma, eps=math.inf)
    for _ in range(steps):
        P, _ = O.update_factor(P, rng.standard_normal(d) / math.sqrt(d), p)
    return P


def first_order_update_error(P, E, x, gamma):
    """Frobenius bound, to first order in E, on the change of the exact
    Sherman-Morrison update P' = (P - k P x x^T P) / gamma,
    k = (1 - gamma) / (gamma + (1 - gamma) x^T P x), when its input P moves
    by E: dP' = (E - k (E x u^T + u x^T E) + k^2 (x^T E x) u u^T) / gamma with
    u = P x (dk = -k^2 d(x^T P x))."""
    u = P @ x
    k = (1.0 - gamma) / (gamma + (1.0 - gamma) * float(x @ u))
    Ex = E @ x
    return (np.linalg.norm(E) + 2 * abs(k) * np.linalg.norm(Ex) * np.linalg.norm(u)
            + k * k * abs(float(x @ Ex)) * float(u @ u)) / gamma


@pytest.mark.parametrize("grad_dtype", ["fp32", "bf16"])
def test_half_step_against_full_precision(grad_dtype):
    """One bf16-factor step from stored factors Q = bf16(P) against the
    fp32-reading oracle (Algorithm 1 in float64, nothing rounded).

    Factors: the stored result against the update of the unquantised P, within
    Lemma 2's bound (eps = max |Q - P|, m = the largest entry of P and x) plus
    the rounding of the result to bf16; and, in Frobenius norm, within the
    first-order change of the update under E = Q - P plus that rounding
    (10 % margin for the higher-order terms and the fp32 evaluation).

    dW: against the oracle's step from the same stored Q.  The kernel rounds
    Y = G_h Rinv' to bf16 (and an fp32 G to G_h), each a relative error of at
    most 2^-9 per element; through dW_hat = Linv' Y_h that is a relative error
    of at most kappa(Linv') ((kappa(Rinv') + 1) 2^-9 (fp32 G) or 2^-9 (bf16 G)),
    doubled by the normalisation of the rescale, plus 2^-9 for ||G_h|| in
    place of ||G|| (fp32 G)."""
    from oracle.half import lemma2_bound
    shapes = [(192, 256), (512, 128), (1024, 1024)]
    p = Params(eps=math.inf)
    op = oparams(p)
    layers = H.allocate_layers(shapes, grad_dtype, factor_dtype="bf16")
    host = []
    for i, (L, (d_in, d_out)) in enumerate(zip(layers, shapes)):
        PL, PR = _trajectory(40 + i, d_in), _trajectory(50 + i, d_out)
        QL, QR = round_bf16(PL), round_bf16(PR)
        a, g, G = _inputs(60 + i, d_in, d_out, grad_dtype)
        H.set_factors(L, QL, QR)
        H.set_inputs(L, a, g, G)
        host.append((PL, PR, QL, QR, a, g, G))
    plan = H.make_plan(layers)
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    u9 = 2.0 ** -9
    for i, (L, (PL, PR, QL, QR, a, g, G)) in enumerate(zip(layers, host)):
        stored = H.get_factors(L)
        updated = []
        for P, Q, x, S in ((PL, QL, a, stored[0]), (PR, QR, g, stored[1])):
            x = np.asarray(x, np.float64)
            P_full, _ = O.update_factor(P, x, op)
            Pq, _ = O.update_factor(Q, x, op)
            updated.append(Pq)
            S = S.astype(np.float64)
            eps_q = float(np.max(np.abs(Q - P)))
            m = float(max(np.max(np.abs(P)), np.max(np.abs(x))))
            err = float(np.max(np.abs(S - P_full)))
            bound = lemma2_bound(op.gamma, m, P.shape[0], eps_q) + u9 * float(np.max(np.abs(P_full)))
            assert eps_q > 0.0 and err <= bound, (i, err, bound)
            fo = 1.1 * first_order_update_error(P, Q - P, x, op.gamma) + u9 * np.linalg.norm(P_full)
            ef = float(np.linalg.norm(S - P_full))
            print(shapes[i], grad_dtype, "factor: max err", err, "Lemma 2 bound", bound,
                  "Frobenius err", ef, "first-order bound", fo)
            assert ef <= fo, (i, ef, fo)
        _, _, dW_ref, _ = O.layer_step(QL, QR, a, g, G, op)
        kL, kR = np.linalg.cond(updated[0]), np.linalg.cond(updated[1])
        if grad_dtype == "bf16":
            tol = 2 * kL * u9 + 1e-5
        else:
            tol = 2 * kL * (kR + 1) * u9 + u9 + 1e-5
        e = rel(H.get_dW(L), dW_ref)
        print(shapes[i], grad_dtype, "dW err", e, "bound", tol, "kappa", kL, kR)
        assert e <= tol, (i, e, tol)
