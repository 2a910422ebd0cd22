"""mkor_step_noalloc, the entry point that allocates no device memory (its
workspace is a fixed device array of the library), against the plan-based
entry points on the same inputs: a fresh plan's mkor_step followed by
mkor_sync_factors.  Two calls in a row, the second over a smaller layer list,
so the second runs on what the first left in the array.  The float64 oracle
checks the fp32-factor layers of both calls as well.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
from paper_2306_01685_amd import Params, binding as B, harness as H
from tests.parity import TOL_STEP, oparams, rel, spd

pytestmark = pytest.mark.gpu

# (d_in, d_out, G dtype, factor dtype, second order): the split path in both
# associations (bf16 G, d_in <= d_out and d_in > d_out), the fp32 MFMA path on
# a ragged shape, bf16 factors, a first-order layer
FIRST = [(128, 256, "bf16", "fp32", 1), (320, 64, "bf16", "fp32", 1), (37, 100, "fp32", "fp32", 1),
         (192, 128, "fp32", "bf16", 1), (64, 96, "fp32", "fp32", 0)]
SECOND = [(64, 64, "fp32", "fp32", 1), (96, 40, "bf16", "fp32", 1)]


def _bf16_exact(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).float().numpy()


def _inputs(specs, seed):
    """Seeded host inputs per layer: factors (SPD, bitwise symmetric), a, g, G."""
    rng = np.random.default_rng(seed)
    out = []
    for k, (d_in, d_out, gdt, fdt, so) in enumerate(specs):
        L0, R0 = spd(seed * 100 + 2 * k, d_in), spd(seed * 100 + 2 * k + 1, d_out)
        if fdt == "bf16":
            L0, R0 = _bf16_exact(L0), _bf16_exact(R0)
        a = (rng.standard_normal(d_in) / math.sqrt(32)).astype(np.float32)
        g = (rng.standard_normal(d_out) * 1e-3 / math.sqrt(32)).astype(np.float32)
        G = (rng.standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
        if gdt == "bf16":
            G = _bf16_exact(G)
        out.append((L0, R0, a, g, G))
    return out


def _layers(specs, host):
    layers = []
    for (d_in, d_out, gdt, fdt, so), (L0, R0, a, g, G) in zip(specs, host):
        L = H.allocate_layers([(d_in, d_out)], gdt, factor_dtype=fdt, second_order=[so])[0]
        if so:
            H.set_factors(L, L0, R0)
            H.set_inputs(L, a, g, G)
        else:
            H.set_inputs(L, G=G)
        layers.append(L)
    return layers


def _check_call(specs, seed, p):
    host = _inputs(specs, seed)
    mine, ref = _layers(specs, host), _layers(specs, host)
    torch.cuda.synchronize()
    B.step_noalloc(mine, p)
    plan = H.make_plan(ref)
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    op = oparams(p)
    worst_ref = worst_oracle = 0.0
    for k, ((d_in, d_out, gdt, fdt, so), (L0, R0, a, g, G)) in enumerate(zip(specs, host)):
        got_dW, ref_dW = H.get_dW(mine[k]), H.get_dW(ref[k])
        e = rel(got_dW, ref_dW)
        worst_ref = max(worst_ref, e)
        assert e <= TOL_STEP, (k, "dW vs plan", e)
        if not so:
            assert np.array_equal(got_dW, G), (k, "first-order dW = G")
            continue
        (gL, gR), (rL, rR) = H.get_factors(mine[k]), H.get_factors(ref[k])
        for name, x, y in (("Linv", gL, rL), ("Rinv", gR, rR)):
            e = rel(x, y)
            worst_ref = max(worst_ref, e)
            assert e <= TOL_STEP, (k, name, "vs plan", e)
        if fdt == "fp32":
            Lo, Ro, dWo, _ = O.layer_step(L0, R0, a, g, G, op)
            for name, x, y in (("Linv", gL, Lo), ("Rinv", gR, Ro), ("dW", got_dW, dWo)):
                e = rel(x, y)
                worst_oracle = max(worst_oracle, e)
                assert e <= TOL_STEP, (k, name, "vs oracle", e)
    del plan
    return worst_ref, worst_oracle


def test_noalloc_matches_plan_two_calls():
    p = Params(gamma=0.9, zeta=0.5, eps=math.inf)
    print("no-alloc call 1: layers", FIRST, flush=True)
    w1 = _check_call(FIRST, 11, p)
    print("no-alloc call 2 (smaller): layers", SECOND, flush=True)
    w2 = _check_call(SECOND, 12, p)
    print("worst rel error (vs plan, vs oracle): call 1", w1, "call 2", w2, flush=True)


def test_noalloc_stabiliser_and_rejects_oversize():
    # the stabiliser blend (eps = 0 fires on every factor), then a list that
    # needs more than the array holds: rejected on the host, nothing launched
    p = Params(gamma=0.9, zeta=0.5, eps=0.0)
    print("no-alloc, stabiliser on: layers", SECOND, flush=True)
    _check_call(SECOND, 13, p)
    big = H.allocate_layers([(4096, 4096)], "fp32")
    with pytest.raises(B.MkorError) as ei:
        B.step_noalloc(big, p)
    assert ei.value.status == B.MKOR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
