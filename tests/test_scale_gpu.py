"""A plan over thousands of layers (Algorithm 1, "for each layer", as one
grouped launch per kernel): 3000 small layers of random ragged shapes, a few
64-aligned ones on the split GEMMs, a sixth first-order, fp32 and bf16
gradients, checked one by one against the float64 oracle after one step, so
that every descriptor table, tile queue and partial-sum slot is exercised
far past the sizes of the model layer sets."""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from paper_2306_01685_amd import Params, harness as H
from tests.parity import TOL_STEP, check_close, oparams, spd

pytestmark = pytest.mark.gpu

N = 3000


def _specs(rng):
    out = []
    for _ in range(N):
        if rng.random() < 0.05:
            d_in, d_out = int(rng.choice([64, 128])), int(rng.choice([64, 128]))
        else:
            d_in, d_out = int(rng.integers(1, 49)), int(rng.integers(1, 49))
        out.append(dict(shape=(d_in, d_out), so=bool(rng.random() > 1 / 6),
                        gdt="bf16" if rng.random() < 0.5 else "fp32"))
    return out


def test_three_thousand_layers_one_step():
    rng = np.random.default_rng(3000)
    specs = _specs(rng)
    layers = [None] * N
    for gdt in ("fp32", "bf16"):
        idx = [k for k, sp in enumerate(specs) if sp["gdt"] == gdt]
        got = H.allocate_layers([specs[k]["shape"] for k in idx], gdt, stats=False,
                                second_order=[specs[k]["so"] for k in idx])
        for k, L in zip(idx, got):
            layers[k] = L
    host = []
    for k, (L, sp) in enumerate(zip(layers, specs)):
        d_in, d_out = sp["shape"]
        G = (rng.standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
        if sp["gdt"] == "bf16":
            G = W.round_to_bf16(G)
        if not sp["so"]:
            H.set_inputs(L, G=G)
            host.append((None, None, None, None, G))
            continue
        Li, Ri = spd(10 * k + 1, d_in, 0.3), spd(10 * k + 2, d_out, 0.3)
        a = (rng.standard_normal(d_in) / math.sqrt(d_in)).astype(np.float32)
        g = (rng.standard_normal(d_out) / math.sqrt(d_out)).astype(np.float32)
        H.set_factors(L, Li, Ri)
        H.set_inputs(L, a, g, G)
        host.append((Li, Ri, a, g, G))
    plan = H.make_plan(layers)
    p = Params(gamma=0.9, zeta=0.5, eps=math.inf)
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    op = oparams(p)
    worst = 0.0
    for k, (L, sp, (Li, Ri, a, g, G)) in enumerate(zip(layers, specs, host)):
        if not sp["so"]:
            np.testing.assert_array_equal(H.get_dW(L), G)
            continue
        Lo, Ro, dW, _ = O.layer_step(Li, Ri, a, g, G, op)
        Lg, Rg = H.get_factors(L)
        worst = max(worst, check_close(H.get_dW(L), dW, TOL_STEP, k, sp, "dW"),
                    check_close(Lg, Lo, TOL_STEP, k, sp, "L"), check_close(Rg, Ro, TOL_STEP, k, sp, "R"))
    print(N, "layers: worst relative error", worst)
