"""GPU parity of the HIP path against the float64 oracle (through the C ABI).

Bars: relative Frobenius error <= 1e-4 after one step from the same state,
<= 1e-3 after up to 50 independently accumulated steps; stabiliser decisions
agree outside a relative 1e-4 band around eps (where fp32 and fp64 may
legitimately differ, the oracle adopts the GPU's decision).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from paper_2306_01685_amd import Params, harness as H, SM_PAPER_EQ6, NORM_MAXABS
from tests.parity import TOL_FREE, TOL_STEP, FreeRun, check_close, oparams, rel, spd

pytestmark = pytest.mark.gpu

RAGGED = [(1, 1), (3, 5), (37, 100), (100, 37), (128, 128), (130, 250), (256, 384), (64, 1000)]


def _random_inputs(seed, d_in, d_out, grad_dtype):
    rng = np.random.default_rng(seed)
    a = (rng.standard_normal(d_in) / math.sqrt(d_in)).astype(np.float32)
    g = (rng.standard_normal(d_out) / math.sqrt(d_out)).astype(np.float32)
    G = (rng.standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
    if grad_dtype == "bf16":
        G = W.round_to_bf16(G)
    return a, g, G


def _setup(shapes, grad_dtype, seed, second_order=None):
    layers = H.allocate_layers(shapes, grad_dtype, second_order=second_order)
    host = []
    for i, (L, (d_in, d_out)) in enumerate(zip(layers, shapes)):
        a, g, G = _random_inputs(seed + i, d_in, d_out, grad_dtype)
        if L["second_order"]:
            Li, Ri = spd(seed * 7 + i, d_in), spd(seed * 11 + i, d_out)
            H.set_factors(L, Li, Ri)
            H.set_inputs(L, a, g, G)
        else:
            Li = Ri = None
            H.set_inputs(L, G=G)
        host.append((Li, Ri, a, g, G))
    return layers, host


@pytest.mark.parametrize("grad_dtype", ["fp32", "bf16"])
def test_precondition_single_step(grad_dtype):
    layers, host = _setup(RAGGED, grad_dtype, seed=100)
    plan = H.make_plan(layers)
    p = Params(eps=math.inf)
    plan.precondition(p)
    torch.cuda.synchronize()
    for i, (L, (Li, Ri, a, g, G)) in enumerate(zip(layers, host)):
        _, _, dW, st = O.layer_step(Li, Ri, a, g, G, oparams(p), update=False)
        check_close(H.get_dW(L), dW, TOL_STEP, i, L["d_in"], L["d_out"])
        s = H.get_stats(L)
        assert s["norm_G"] == pytest.approx(st.norm_G, rel=1e-5)
        assert s["norm_dW_hat"] == pytest.approx(st.norm_dW_hat, rel=1e-4)
        assert s["scale"] == pytest.approx(st.scale, rel=1e-4)


def test_precondition_without_rescale():
    layers, host = _setup(RAGGED[:5], "fp32", seed=150)
    plan = H.make_plan(layers)
    p = Params(eps=math.inf, rescale=False)
    plan.precondition(p)
    torch.cuda.synchronize()
    for L, (Li, Ri, a, g, G) in zip(layers, host):
        ref = O.precondition(Li, G, Ri)
        check_close(H.get_dW(L), ref, TOL_STEP, L["d_in"], L["d_out"])
        assert H.get_stats(L)["scale"] == 1.0


@pytest.mark.parametrize("variant,norm_kind,eps", [(0, 0, math.inf), (0, 0, 0.0), (1, 0, math.inf),
                                                   (0, 1, 0.0), (1, 1, 0.0)])
def test_update_factors_single_step(variant, norm_kind, eps):
    layers, host = _setup(RAGGED, "fp32", seed=200 + variant)
    plan = H.make_plan(layers)
    p = Params(eps=eps, variant=variant, norm_kind=norm_kind, zeta=0.3)
    op = oparams(p)
    plan.update_factors(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    for i, (L, (Li, Ri, a, g, G)) in enumerate(zip(layers, host)):
        Lo, sL = O.update_factor(Li, a, op)
        Ro, sR = O.update_factor(Ri, g, op)
        Lg, Rg = H.get_factors(L)
        check_close(Lg, Lo, TOL_STEP, i, "L")
        check_close(Rg, Ro, TOL_STEP, i, "R")
        np.testing.assert_array_equal(Lg, Lg.T)   # bitwise symmetric
        np.testing.assert_array_equal(Rg, Rg.T)
        s = H.get_stats(L)
        assert s["stab_L"] == int(sL.stab) and s["stab_R"] == int(sR.stab)
        assert s["nu_L"] == pytest.approx(sL.nu, rel=1e-5)
        assert s["s_L"] == pytest.approx(sL.s, rel=1e-4, abs=1e-6)
        assert s["skip_L"] == 0 and s["skip_R"] == 0


@pytest.mark.parametrize("eps", [math.inf, 4.0])
def test_cfg1_free_running(eps):
    w = W.SINGLE_64
    fr = FreeRun(w, Params(gamma=w.gamma, eps=eps), sample=[0], explicit=True)
    for t in range(w.steps):
        out = fr.step(precond_oracle=True)
        tol = TOL_STEP if t == 0 else TOL_FREE
        fr.check_factors(tol)
        fr.check_dW(out, tol)
    fired = fr.check_flags()
    if math.isfinite(eps):
        assert fired > 0


def test_first_order_layers_pass_gradient():
    shapes = [(64, 96), (37, 100), (128, 256), (100, 37)]
    for dt in ("fp32", "bf16"):
        layers, host = _setup(shapes, dt, seed=300, second_order=[1, 0, 1, 0])
        plan = H.make_plan(layers)
        plan.step(Params(eps=math.inf))
        torch.cuda.synchronize()
        for L, (Li, Ri, a, g, G) in zip(layers, host):
            if not L["second_order"]:
                np.testing.assert_array_equal(H.get_dW(L), G)
            else:
                _, _, dW, _ = O.layer_step(Li, Ri, a, g, G, oparams(Params(eps=math.inf)))
                check_close(H.get_dW(L), dW, TOL_STEP, dt, L["d_in"], L["d_out"])


def test_guard_nonfinite():
    shapes = [(64, 64), (40, 80)]
    layers, host = _setup(shapes, "fp32", seed=400)
    a_bad = host[0][2].copy()
    a_bad[3] = np.nan
    H.set_inputs(layers[0], a=a_bad)
    L0_before = H.get_factors(layers[0])[0]
    plan = H.make_plan(layers)
    plan.step(Params(eps=math.inf, guard_nonfinite=True))
    plan.sync_factors()
    torch.cuda.synchronize()
    s = H.get_stats(layers[0])
    assert s["skip_L"] == 1 and s["skip_R"] == 0
    np.testing.assert_array_equal(H.get_factors(layers[0])[0], L0_before)
    assert np.isfinite(H.get_dW(layers[0])).all()
    Li, Ri, a, g, G = host[1]
    Lo, _ = O.update_factor(Li, a, oparams(Params(eps=math.inf)))
    assert rel(H.get_factors(layers[1])[0], Lo) <= TOL_STEP
    # without the guard the NaN propagates into the factor
    plan.step(Params(eps=math.inf, guard_nonfinite=False))
    plan.sync_factors()
    torch.cuda.synchronize()
    assert np.isnan(H.get_factors(layers[0])[0]).any()
    assert H.get_stats(layers[0])["skip_L"] == 1


def test_stages_in_order_equal_step():
    """Launching the stages one by one (mkor_run_stage 0 .. NUM_STAGES - 1, as
    bench.py does for per-kernel times) is mkor_step: the same bits, over
    several steps, on the split, fp32 MFMA and first-order paths."""
    from paper_2306_01685_amd import NUM_STAGES
    shapes = [(128, 256), (256, 128), (37, 100), (64, 64)]
    second = [1, 1, 1, 0]
    A, _ = _setup(shapes, "bf16", seed=500, second_order=second)
    B, _ = _setup(shapes, "bf16", seed=500, second_order=second)
    pa, pb = H.make_plan(A), H.make_plan(B)
    p = Params(eps=3.0)
    for t in range(5):
        for i, (LA, LB) in enumerate(zip(A, B)):
            a, g, G = _random_inputs(900 + 10 * t + i, LA["d_in"], LA["d_out"], "bf16")
            for L in (LA, LB):
                if L["second_order"]:
                    H.set_inputs(L, a, g, G)
                else:
                    H.set_inputs(L, G=G)
        pa.step(p)
        for st in range(NUM_STAGES):
            pb.run_stage(p, st)
        torch.cuda.synchronize()
        for x, y in zip(A, B):
            assert torch.equal(x["dW"], y["dW"]), t
    pa.sync_factors()
    pb.sync_factors()
    torch.cuda.synchronize()
    for x, y in zip(A, B):
        if x["second_order"]:
            assert torch.equal(x["Linv"], y["Linv"]) and torch.equal(x["Rinv"], y["Rinv"])


def test_lazy_write_back_cadence():
    """On the split path Rinv (the first GEMM's factor here) is written back
    every other step and Linv every step: after two steps the Rinv buffer
    still holds the initial factor and the Linv buffer P_1; after three, Rinv
    holds P_2 (both pending terms, evaluated in order) and Linv P_2."""
    layers, host = _setup([(128, 192)], "fp32", seed=420)
    Li, Ri, a, g, G = host[0]
    L = layers[0]
    plan = H.make_plan(layers)
    p = Params(eps=math.inf)
    op = oparams(p)
    L1, _ = O.update_factor(Li, a, op)
    R1, _ = O.update_factor(Ri, g, op)
    L2, _ = O.update_factor(L1, a, op)
    R2, _ = O.update_factor(R1, g, op)
    plan.step(p)
    plan.step(p)
    torch.cuda.synchronize()
    Lg, Rg = H.get_factors(L)
    np.testing.assert_array_equal(Rg, Ri.astype(np.float32))
    assert rel(Lg, L1) <= TOL_STEP
    plan.step(p)
    torch.cuda.synchronize()
    Lg, Rg = H.get_factors(L)
    assert rel(Lg, L2) <= TOL_STEP and rel(Rg, R2) <= TOL_STEP


def test_guard_nonfinite_keeps_lazy_pending_term():
    """The split path writes the first GEMM's factor (Rinv here) back only
    every other step; an update skipped while the previous one is still
    pending keeps that one: after a good step and a skipped one the factor is
    the good step's."""
    layers, host = _setup([(64, 64)], "fp32", seed=410)
    Li, Ri, a, g, G = host[0]
    plan = H.make_plan(layers)
    p = Params(eps=math.inf, guard_nonfinite=True)
    plan.step(p)
    g_bad = g.copy()
    g_bad[5] = np.nan
    H.set_inputs(layers[0], g=g_bad)
    plan.step(p)
    torch.cuda.synchronize()
    s = H.get_stats(layers[0])
    assert s["skip_R"] == 1 and s["skip_L"] == 0
    assert np.isfinite(H.get_dW(layers[0])).all()
    plan.sync_factors()
    torch.cuda.synchronize()
    Ro, _ = O.update_factor(Ri, g, oparams(p))
    assert rel(H.get_factors(layers[0])[1], Ro) <= TOL_STEP


def _run_steps(shapes, steps, seed, dt="bf16", layers=None, start=0, sync_every=False, gemm_path=None,
               sync_at=None):
    if layers is None:
        layers = H.allocate_layers(shapes, dt, gemm_path=gemm_path)
    plan = H.make_plan(layers)
    p = Params(eps=3.0)
    for t in range(start, start + steps):
        for i, L in enumerate(layers):
            a, g, G = _random_inputs(seed + 1000 * t + i, L["d_in"], L["d_out"], dt)
            H.set_inputs(L, a, g, G)
        plan.step(p)
        if sync_every or t + 1 == sync_at:
            plan.sync_factors()
    plan.sync_factors()
    torch.cuda.synchronize()
    return layers


def test_determinism_and_checkpoint_resume():
    shapes = [(128, 256), (37, 100), (256, 128)]
    A = _run_steps(shapes, 10, seed=7)
    B = _run_steps(shapes, 10, seed=7)
    for x, y in zip(A, B):
        for k in ("Linv", "Rinv", "dW"):
            assert torch.equal(x[k], y[k]), k
    # 5 steps, save the state (a sync: the buffers then hold the factors and
    # nothing is pending), fresh buffers and plan, 5 more steps: the same bits
    # as syncing after step 5 and going on in the same plan.  Without that
    # sync the factors are the same bits too; dW, whose split-path epilogue
    # applies one or two pending terms algebraically, differs by rounding.
    C = _run_steps(shapes, 5, seed=7)
    saved = [(H.get_factors(L)) for L in C]
    D = H.allocate_layers(shapes, "bf16")
    for L, (Li, Ri) in zip(D, saved):
        H.set_factors(L, Li, Ri)
    D = _run_steps(shapes, 5, seed=7, layers=D, start=5)
    E = _run_steps(shapes, 10, seed=7, sync_at=5)
    for x, y, z in zip(A, D, E):
        for k in ("Linv", "Rinv", "dW"):
            assert torch.equal(z[k], y[k]), k
        for k in ("Linv", "Rinv"):
            assert torch.equal(x[k], y[k]), k
        assert rel(x["dW"].cpu().numpy(), y["dW"].cpu().numpy()) <= 1e-6


def test_pending_term_matches_write_back_every_step():
    """Keeping each update pending (applied in the fp32 GEMM's loads and
    written by the next pass) gives the same bits as writing it back after
    every step.  On the split path the pending term enters the epilogue
    algebraically, and the first GEMM's factor carries two terms every other
    step (the pass writes it back only then, evaluating them one after the
    other): the factors still agree bit for bit, dW to rounding."""
    shapes = [(128, 256), (37, 100), (256, 128), (64, 64)]
    A = _run_steps(shapes, 8, seed=11, dt="fp32", gemm_path="fp32")
    B = _run_steps(shapes, 8, seed=11, dt="fp32", sync_every=True, gemm_path="fp32")
    for x, y in zip(A, B):
        for k in ("Linv", "Rinv", "dW"):
            assert torch.equal(x[k], y[k]), k
    shapes = [(128, 256), (256, 128), (64, 64)]
    A = _run_steps(shapes, 8, seed=11, dt="fp32", gemm_path="split")
    B = _run_steps(shapes, 8, seed=11, dt="fp32", sync_every=True, gemm_path="split")
    for x, y in zip(A, B):
        for k in ("Linv", "Rinv"):
            assert torch.equal(x[k], y[k]), k
        assert rel(x["dW"].cpu().numpy(), y["dW"].cpu().numpy()) <= 1e-6


def test_buffers_lag_until_sync():
    """After a step the buffers hold the factors before that step's update;
    sync_factors writes the updated ones, and a second sync changes nothing."""
    layers, host = _setup([(64, 96), (37, 100)], "fp32", seed=700)
    before = [H.get_factors(L) for L in layers]
    plan = H.make_plan(layers)
    p = Params(eps=math.inf)
    plan.step(p)
    torch.cuda.synchronize()
    for L, (Lb, Rb) in zip(layers, before):
        Lg, Rg = H.get_factors(L)
        np.testing.assert_array_equal(Lg, Lb)
        np.testing.assert_array_equal(Rg, Rb)
    plan.sync_factors()
    torch.cuda.synchronize()
    synced = [H.get_factors(L) for L in layers]
    for L, (Li, Ri, a, g, G), (Lg, Rg) in zip(layers, host, synced):
        Lo, Ro, _, _ = O.layer_step(Li, Ri, a, g, G, oparams(p))
        check_close(Lg, Lo, TOL_STEP, "L")
        check_close(Rg, Ro, TOL_STEP, "R")
    plan.sync_factors()
    torch.cuda.synchronize()
    for L, (Lg, Rg) in zip(layers, synced):
        np.testing.assert_array_equal(H.get_factors(L)[0], Lg)
        np.testing.assert_array_equal(H.get_factors(L)[1], Rg)


def test_plan_reuse_two_plans_same_buffers():
    """Two plans over disjoint layer lists on one stream give independent results."""
    layers1, host1 = _setup([(64, 128)], "fp32", seed=500)
    layers2, host2 = _setup([(128, 64)], "fp32", seed=600)
    p1, p2 = H.make_plan(layers1), H.make_plan(layers2)
    p1.step(Params(eps=math.inf))
    p2.step(Params(eps=math.inf))
    torch.cuda.synchronize()
    for layers, host in ((layers1, host1), (layers2, host2)):
        Li, Ri, a, g, G = host[0]
        Lo, Ro, dW, _ = O.layer_step(Li, Ri, a, g, G, oparams(Params(eps=math.inf)))
        check_close(H.get_dW(layers[0]), dW, TOL_STEP)


def test_layer_results_do_not_depend_on_the_plan():
    """A layer's dW and factors are the same bits whether it is stepped alone
    or among other layers (every reduction is per layer, in a fixed order;
    tile scheduling and table positions change with the plan's contents):
    three layers on the split path, the fp32 MFMA path and bf16 factors, each
    alone and together with 20 filler layers, over three steps."""
    spec = [((128, 192), "bf16", {}), ((37, 100), "fp32", {}), ((64, 64), "fp32", dict(factor_dtype="bf16"))]
    rng = np.random.default_rng(31)
    fill = [(int(rng.integers(1, 300)), int(rng.integers(1, 300))) for _ in range(20)]

    def run(which, with_fill):
        layers = []
        for k in which:
            shape, gdt, kw = spec[k]
            L = H.allocate_layers([shape], gdt, **kw)[0]
            Li, Ri = spd(70 + 2 * k, shape[0], 0.3), spd(71 + 2 * k, shape[1], 0.3)
            if kw.get("factor_dtype") == "bf16":
                Li, Ri = W.round_to_bf16(Li), W.round_to_bf16(Ri)
            H.set_factors(L, Li, Ri)
            layers.append((k, L))
        extra = H.allocate_layers(fill, "fp32") if with_fill else []
        plan = H.make_plan([L for _, L in layers[:1]] + extra + [L for _, L in layers[1:]])
        p = Params(gamma=0.9, zeta=0.5, eps=2.0)
        for t in range(3):
            for k, L in layers:
                a, g, G = _random_inputs(500 + 10 * t + k, L["d_in"], L["d_out"], spec[k][1])
                H.set_inputs(L, a, g, G)
            for j, E in enumerate(extra):
                a, g, G = _random_inputs(900 + 50 * t + j, E["d_in"], E["d_out"], "fp32")
                H.set_inputs(E, a, g, G)
            plan.step(p)
        plan.sync_factors()
        torch.cuda.synchronize()
        return {k: (L["dW"].clone(), L["Linv"].clone(), L["Rinv"].clone()) for k, L in layers}

    together = run([0, 1, 2], True)
    for k in range(3):
        alone = run([k], False)[k]
        for name, x, y in zip(("dW", "Linv", "Rinv"), alone, together[k]):
            assert torch.equal(x, y), (k, name)
