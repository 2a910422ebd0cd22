"""GPU parity of the preconditioning of fp32 factors on the three-way bf16
split (MKOR_GEMM_SPLIT) against the float64 oracle, and its accuracy beside
the fp32 MFMA path (MKOR_GEMM_FP32) on the same inputs.

Bars: relative Frobenius error <= 1e-4 after one step from the same state (as
for every path); the split's error is also held to the fp32 MFMA path's order
(at most 3x it, or 2e-6), since it is meant as an fp32-accurate product.
Without a pending term the split's dW is held to 2e-6 Frobenius and 4e-6
element-wise (TOL_SPLIT_ELEM: the largest of some 10^5 element errors runs
2-3x the Frobenius figure on these shapes).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from paper_2306_01685_amd import MkorError, Params, harness as H
from tests.parity import TOL_STEP, check_close, oparams, rel, relmax, spd

pytestmark = pytest.mark.gpu

# multiples of 64, ragged against the 256 x 256 tiles; with a bf16 G the layers
# with d_in > d_out take the other association ((Linv G) Rinv, dW stored
# transposed from the second GEMM)
SHAPES = [(64, 64), (128, 192), (192, 320), (320, 64), (256, 512), (576, 320)]
TOL_SPLIT_ELEM = 4e-6


def _inputs(seed, d_in, d_out, grad_dtype, scale=1.0):
    rng = np.random.default_rng(seed)
    a = (rng.standard_normal(d_in) / math.sqrt(d_in)).astype(np.float32)
    g = (rng.standard_normal(d_out) / math.sqrt(d_out)).astype(np.float32)
    G = (rng.standard_normal((d_in, d_out)) * 1e-3 * scale).astype(np.float32)
    if grad_dtype == "bf16":
        G = W.round_to_bf16(G)
    return a, g, G


def _run(path, grad_dtype, seed, p, update=True, fscale=1.0, gscale=1.0):
    layers = H.allocate_layers(SHAPES, grad_dtype, gemm_path=path)
    host = []
    for i, (L, (d_in, d_out)) in enumerate(zip(layers, SHAPES)):
        Li = (spd(seed * 7 + i, d_in) * np.float32(fscale)).astype(np.float32)
        Ri = (spd(seed * 11 + i, d_out) * np.float32(fscale)).astype(np.float32)
        a, g, G = _inputs(seed + i, d_in, d_out, grad_dtype, gscale)
        H.set_factors(L, Li, Ri)
        H.set_inputs(L, a, g, G)
        host.append((Li, Ri, a, g, G))
    plan = H.make_plan(layers)
    if update:
        plan.step(p)
    else:
        plan.precondition(p)
    torch.cuda.synchronize()
    return layers, host


@pytest.mark.parametrize("grad_dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("eps", [math.inf, 0.0])
def test_split_single_step(grad_dtype, eps):
    p = Params(eps=eps)
    op = oparams(p)
    split, host = _run("split", grad_dtype, 30, p)
    fp32, _ = _run("fp32", grad_dtype, 30, p)
    for i, (Ls, Lf, (Li, Ri, a, g, G)) in enumerate(zip(split, fp32, host)):
        Lo, Ro, dW, st = O.layer_step(Li, Ri, a, g, G, op)
        es, ef = rel(H.get_dW(Ls), dW), rel(H.get_dW(Lf), dW)
        ms, mf = relmax(H.get_dW(Ls), dW), relmax(H.get_dW(Lf), dW)
        print(SHAPES[i], grad_dtype, eps, "dW error split", es, ms, "fp32 MFMA", ef, mf)
        assert es <= TOL_STEP and ms <= TOL_STEP, (i, es, ms)
        assert es <= max(3 * ef, 2e-6), (i, es, ef)
        assert ms <= max(3 * mf, TOL_SPLIT_ELEM), (i, ms, mf)
        s = H.get_stats(Ls)
        assert s["norm_G"] == pytest.approx(st.norm_G, rel=1e-5)
        assert s["norm_dW_hat"] == pytest.approx(st.norm_dW_hat, rel=1e-5)
        assert bool(s["stab_L"]) == st.L.stab and bool(s["stab_R"]) == st.R.stab
    # the factor update does not depend on the GEMM path
    for Ls, Lf in zip(split, fp32):
        for k in ("Linv", "Rinv"):
            assert torch.equal(Ls[k], Lf[k]), k


@pytest.mark.parametrize("grad_dtype", ["fp32", "bf16"])
def test_split_precondition_only(grad_dtype):
    """No pending term (the epilogue's plain path), with and without rescale."""
    for rescale in (True, False):
        p = Params(eps=math.inf, rescale=rescale)
        layers, host = _run("split", grad_dtype, 60, p, update=False)
        for i, (L, (Li, Ri, a, g, G)) in enumerate(zip(layers, host)):
            _, _, dW, _ = O.layer_step(Li, Ri, a, g, G, oparams(p), update=False)
            e, m = rel(H.get_dW(L), dW), relmax(H.get_dW(L), dW)
            print(SHAPES[i], grad_dtype, rescale, "dW error", e, m)
            assert e <= 2e-6 and m <= TOL_SPLIT_ELEM, (i, rescale, e, m)


def test_split_small_and_large_magnitudes():
    """The split is exact for operand magnitudes in [2^-110, 3.396e38): factors
    scaled by 1e-6 and 1e6 (and G with them; every partial product stays a
    normal fp32 number) keep the fp32-level error."""
    for fscale, gscale in ((1e-6, 1e-6), (1e6, 1e3)):
        p = Params(eps=math.inf, rescale=False)
        layers, host = _run("split", "fp32", 90, p, update=False, fscale=fscale, gscale=gscale)
        for i, (L, (Li, Ri, a, g, G)) in enumerate(zip(layers, host)):
            ref = O.precondition(Li, G, Ri)
            e, m = rel(H.get_dW(L), ref), relmax(H.get_dW(L), ref)
            print(SHAPES[i], fscale, "dW error", e, m)
            assert e <= 2e-6 and m <= TOL_SPLIT_ELEM, (fscale, i, e, m)


def test_split_after_sync_and_over_steps():
    """Several steps (pending terms carried), a sync in between, then a
    precondition-only step: dW of every step against the oracle.  With a bf16
    G, (320, 64) and (576, 320) take the other association, whose lazily
    written Linv carries two pending terms on every other step, so both forms
    of the first GEMM's epilogue are checked, before and after the sync
    shifts the write-back cadence."""
    p = Params(eps=3.0)
    op = oparams(p)
    shapes = SHAPES[:3] + [SHAPES[3], SHAPES[5]]
    layers = H.allocate_layers(shapes, "bf16", gemm_path="split")
    state = []
    for i, (L, (d_in, d_out)) in enumerate(zip(layers, shapes)):
        Li, Ri = spd(500 + i, d_in), spd(600 + i, d_out)
        H.set_factors(L, Li, Ri)
        state.append([Li.astype(np.float64), Ri.astype(np.float64)])
    plan = H.make_plan(layers)
    for t in range(9):
        update = t != 8
        outs = []
        for i, L in enumerate(layers):
            a, g, G = _inputs(700 + 10 * t + i, L["d_in"], L["d_out"], "bf16")
            H.set_inputs(L, a, g, G)
            Lo, Ro, dW, _ = O.layer_step(state[i][0], state[i][1], a, g, G, op, update=update)
            state[i] = [Lo, Ro]
            outs.append(dW)
        if update:
            plan.step(p)
        else:
            plan.precondition(p)
        if t == 2:
            plan.sync_factors()
        torch.cuda.synchronize()
        for i, L in enumerate(layers):
            check_close(H.get_dW(L), outs[i], TOL_STEP, t, i)


def test_split_shape_rule():
    with pytest.raises(MkorError):
        H.make_plan(H.allocate_layers([(64, 96)], "fp32", gemm_path="split"))
    # AUTO takes the fp32 MFMA path for that shape
    H.make_plan(H.allocate_layers([(64, 96)], "fp32", gemm_path="auto"))
