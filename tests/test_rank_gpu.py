"""GPU parity of the rank-r update (the paper's extension to higher ranks)
against the rank-r oracle (oracle/rank.py), through the C ABI.

Bars as for the rank-1 path: relative Frobenius error <= 1e-4 after one step
from the same state, <= 1e-3 after 50 independently accumulated steps;
stabiliser decisions agree (eps is set far from the norms here).  A rank-r
update is written into the factor buffers within the step, so the buffers are
compared without mkor_sync_factors (which must then change nothing).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
from oracle.rank import layer_step_rank
from paper_2306_01685_amd import MkorError, Params, SM_PAPER_EQ6, harness as H
from tests.parity import TOL_FREE, TOL_STEP, check_close, oparams, spd

pytestmark = pytest.mark.gpu

SHAPES = [(1, 5), (37, 100), (64, 64), (130, 250), (256, 384)]


def _vectors(seed, d, r):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((r, d)) / math.sqrt(d)).astype(np.float32)


def _setup(shapes, rank, seed):
    layers = H.allocate_layers(shapes, "fp32", rank=rank)
    host = []
    for i, (L, (d_in, d_out)) in enumerate(zip(layers, shapes)):
        Li, Ri = spd(seed * 7 + i, d_in), spd(seed * 11 + i, d_out)
        A, Gv = _vectors(seed + 100 * i, d_in, rank), _vectors(seed + 100 * i + 1, d_out, rank)
        G = (np.random.default_rng(seed + 100 * i + 2).standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
        H.set_factors(L, Li, Ri)
        H.set_inputs(L, A if rank > 1 else A[0], Gv if rank > 1 else Gv[0], G)
        host.append((Li.astype(np.float64), Ri.astype(np.float64), A.T.astype(np.float64),
                     Gv.T.astype(np.float64), G))
    return layers, host


@pytest.mark.parametrize("rank", [2, 3, 4])
@pytest.mark.parametrize("eps", [math.inf, 0.0])
def test_rank_single_step(rank, eps):
    layers, host = _setup(SHAPES, rank, seed=800 + rank)
    plan = H.make_plan(layers)
    p = Params(eps=eps)
    plan.step(p)
    torch.cuda.synchronize()
    op = oparams(p)
    before = [H.get_factors(L) for L in layers]
    for i, (L, (Li, Ri, A, Gv, G)) in enumerate(zip(layers, host)):
        Lo, Ro, dW, st = layer_step_rank(Li, Ri, A, Gv, G, op)
        Lg, Rg = before[i]
        eL, eR, eD = (check_close(x, y, TOL_STEP, i, k) for x, y, k in
                      ((Lg, Lo, "L"), (Rg, Ro, "R"), (H.get_dW(L), dW, "dW")))
        print(rank, eps, L["d_in"], L["d_out"], "errors L R dW", eL, eR, eD)
        s = H.get_stats(L)
        assert bool(s["stab_L"]) == st.L.stab and bool(s["stab_R"]) == st.R.stab
        assert s["nu_L"] == pytest.approx(st.L.nu, rel=1e-5)
        assert s["s_R"] == pytest.approx(st.R.s, rel=1e-4, abs=1e-7)
        assert not s["skip_L"] and not s["skip_R"]
    # the update is already in the buffers: syncing changes nothing
    plan.sync_factors()
    torch.cuda.synchronize()
    for L, (Lg, Rg) in zip(layers, before):
        La, Ra = H.get_factors(L)
        assert np.array_equal(La, Lg) and np.array_equal(Ra, Rg)


def test_rank_free_run_50_steps():
    shapes = [(64, 64), (130, 250), (256, 384)]
    rank = 4
    layers, host = _setup(shapes, rank, seed=900)
    plan = H.make_plan(layers)
    p = Params(eps=100.0)
    op = oparams(p)
    state = [(Li, Ri) for Li, Ri, *_ in host]
    for t in range(50):
        outs = []
        for i, L in enumerate(layers):
            d_in, d_out = shapes[i]
            A, Gv = _vectors(1000 * t + 10 * i, d_in, rank), _vectors(1000 * t + 10 * i + 1, d_out, rank)
            G = (np.random.default_rng(1000 * t + 10 * i + 2).standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
            H.set_inputs(L, A, Gv, G)
            Lo, Ro, dW, _ = layer_step_rank(state[i][0], state[i][1], A.T, Gv.T, G, op)
            state[i] = (Lo, Ro)
            outs.append(dW)
        plan.step(p)
    torch.cuda.synchronize()
    for i, L in enumerate(layers):
        Lg, Rg = H.get_factors(L)
        eL, eR, eD = (check_close(x, y, TOL_FREE, i, k) for x, y, k in
                      ((Lg, state[i][0], "L"), (Rg, state[i][1], "R"), (H.get_dW(L), outs[i], "dW")))
        print(shapes[i], "50-step errors L R dW", eL, eR, eD)


def test_rank_mixed_plan_and_variant_check():
    """rank-4, rank-1 and first-order layers in one plan; the printed variant
    is refused for a plan with rank-r layers."""
    l4 = H.allocate_layers([(96, 160)], "fp32", rank=4)[0]
    l1 = H.allocate_layers([(130, 250)], "bf16")[0]
    lf = H.allocate_layers([(50, 70)], "fp32", second_order=[False])[0]
    A, Gv = _vectors(1, 96, 4), _vectors(2, 160, 4)
    G4 = (np.random.default_rng(3).standard_normal((96, 160)) * 1e-3).astype(np.float32)
    Li4, Ri4 = spd(4, 96), spd(5, 160)
    H.set_factors(l4, Li4, Ri4)
    H.set_inputs(l4, A, Gv, G4)
    a1, g1 = _vectors(6, 130, 1)[0], _vectors(7, 250, 1)[0]
    import workloads as W
    G1 = W.round_to_bf16((np.random.default_rng(8).standard_normal((130, 250)) * 1e-3).astype(np.float32))
    Li1, Ri1 = spd(9, 130), spd(10, 250)
    H.set_factors(l1, Li1, Ri1)
    H.set_inputs(l1, a1, g1, G1)
    Gf = np.random.default_rng(11).standard_normal((50, 70)).astype(np.float32)
    H.set_inputs(lf, G=Gf)
    plan = H.make_plan([l4, l1, lf])
    with pytest.raises(MkorError):
        plan.step(Params(variant=SM_PAPER_EQ6))
    p = Params(eps=math.inf)
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    op = oparams(p)
    Lo, Ro, dW, _ = layer_step_rank(Li4, Ri4, A.T, Gv.T, G4, op)
    check_close(H.get_dW(l4), dW, TOL_STEP, "rank 4 dW")
    check_close(H.get_factors(l4)[0], Lo, TOL_STEP, "rank 4 L")
    Lo1, Ro1, dW1, _ = O.layer_step(Li1, Ri1, a1, g1, G1, op)
    check_close(H.get_dW(l1), dW1, TOL_STEP, "rank 1 dW")
    check_close(H.get_factors(l1)[1], Ro1, TOL_STEP, "rank 1 R")
    assert np.array_equal(H.get_dW(lf), Gf)
