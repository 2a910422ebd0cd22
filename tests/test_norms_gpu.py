"""The rescale's two norms at full size, for every layer of a grouped step
(Algorithm 1's rescale line, "Rescaling Gradients"): the recorded ||G||_F
equals the float64 norm of G, and ||dW||_F equals ||G||_F.  Both hold by
definition at any size, so every layer of the set is checked, on every GEMM
path, over three steps (the lazily written factors carry one and two pending
terms).

The bars are rounding alone: the recorded norm and the scale are fp32 (up to
2^-24 = 6e-8 relative each), and each thread sums at most a few hundred
squares in fp32 before the partials meet in fixed-order trees and in float64
(drift of a few 1e-8).  Measured worst over these sets: 1.1e-7.  A single fp32
chain over all of a thread's K range or all of a block's rows (thousands of
positive terms) drifts low by 1.6e-6 to 2.3e-6 relative here: a scale error
that reaches every element of dW, and eight times these bars.
"""
import math

import pytest
import torch

import workloads as W
from paper_2306_01685_amd import Params, harness as H

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL_NORM_G = 2e-7   # |recorded ||G|| / ||G||_fp64 - 1|
TOL_RATIO = 2e-7    # | ||dW|| / ||G|| - 1 |

CASES = [(W.BERT_LARGE, dict(gemm_path="auto")), (W.BERT_LARGE, dict(gemm_path="fp32")),
         (W.BERT_LARGE, dict(factor_dtype="bf16")), (W.GPT2_XL, dict(gemm_path="auto")),
         (W.GPT2_XL, dict(gemm_path="fp32"))]


def _fill(layers, w, gen):
    for L in layers:
        d_in, d_out = L["d_in"], L["d_out"]
        if "a" in L:
            L["a"].normal_(0.0, 1.0 / math.sqrt(d_in), generator=gen)
            L["g"].normal_(0.0, 1.0 / math.sqrt(d_out), generator=gen)
        t = torch.empty((d_in, d_out), dtype=torch.float32, device="cuda")
        t.normal_(0.0, w.G_std, generator=gen)
        L["G"].copy_(t)   # rounded to nearest for a bf16 G


@pytest.mark.parametrize("w,kw", CASES, ids=[f"{w.name}-{next(iter(k.values()))}" for w, k in CASES])
def test_rescale_norms_every_layer(w, kw):
    layers = H.allocate_layers(w.shapes, w.grad_dtype, **kw)
    plan = H.make_plan(layers)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(9000 + w.cid)
    p = Params(gamma=w.gamma, zeta=0.5, eps=100.0)
    worst_g = worst_r = 0.0
    for t in range(3):
        _fill(layers, w, gen)
        plan.step(p)
        torch.cuda.synchronize()
        so = [L for L in layers if L["second_order"]]
        nG = torch.stack([L["G"].double().norm() for L in so]).cpu().tolist()
        nW = torch.stack([L["dW"].double().norm() for L in so]).cpu().tolist()
        for k, L in enumerate(so):
            st = H.get_stats(L)
            eg = abs(st["norm_G"] / nG[k] - 1.0)
            er = abs(nW[k] / nG[k] - 1.0)
            worst_g, worst_r = max(worst_g, eg), max(worst_r, er)
            assert eg <= TOL_NORM_G, (w.name, kw, t, k, (L["d_in"], L["d_out"]), "norm_G", eg)
            assert er <= TOL_RATIO, (w.name, kw, t, k, (L["d_in"], L["d_out"]), "||dW||/||G||", er)
    print(w.name, kw, "worst |norm_G - ||G|||/||G||", worst_g, "worst | ||dW||/||G|| - 1 |", worst_r)
