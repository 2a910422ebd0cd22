"""The method's degenerate cases on every path, against the oracle:

* a = g = 0 (or all-zero token rows): u = 0 and s = 0, so the update is
  P_hat / gamma (Eq. 6/7 with a zero vector; Algorithm 1 still rescales);
* G = 0: dW_hat = 0, so ||dW_hat|| = 0 and the rescale gives dW = 0, not NaN
  (the rescale reading); with the rescale off dW = dW_hat = 0 as well;
* eps = 0 with zeta = 1: the stabiliser fires (norm > 0) but its blend
  zeta P + (1 - zeta) I is P itself, so the factors follow the plain update.

Paths: fp32 MFMA at a ragged size, the split in both associations, bf16
factors, a rank-2 layer (zero vectors), means from all-zero token rows.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from oracle.half import layer_step_half, round_bf16
from oracle.rank import layer_step_rank
from paper_2306_01685_amd import Params, harness as H
from tests.parity import TOL_FREE, TOL_HALF_FREE, TOL_HALF_STEP, TOL_STEP, oparams, rel, spd

pytestmark = pytest.mark.gpu

SPECS = [dict(shape=(37, 100), gdt="fp32", path="fp32"), dict(shape=(128, 192), gdt="bf16", path="split"),
         dict(shape=(320, 64), gdt="bf16", path="split"), dict(shape=(128, 64), gdt="fp32", half=True),
         dict(shape=(64, 96), gdt="fp32", rank=2), dict(shape=(64, 100), gdt="bf16", rows=33)]


def _bf16(x):
    return W.round_to_bf16(np.asarray(x, np.float32))


def _alloc(sp):
    half, rank, rows = sp.get("half", False), sp.get("rank", 1), sp.get("rows", 0)
    return H.allocate_layers([sp["shape"]], sp["gdt"], factor_dtype="bf16" if half else "fp32", rank=rank,
                             rows=rows, act_dtype="bf16", gemm_path=None if half else sp.get("path"))[0]


def _oracle(sp, st, a, g, G, op):
    if sp.get("half"):
        return layer_step_half(st[0], st[1], a, g, G, op)
    if sp.get("rank", 1) > 1:
        return layer_step_rank(st[0], st[1], a.T, g.T, G, op)
    return O.layer_step(st[0], st[1], a, g, G, op)


def _inputs(rng, sp, zero_vec, zero_G):
    d_in, d_out = sp["shape"]
    r, rows = sp.get("rank", 1), sp.get("rows", 0)
    G = np.zeros((d_in, d_out), np.float32) if zero_G else (rng.standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
    if sp["gdt"] == "bf16":
        G = _bf16(G)
    if rows:
        A = np.zeros((rows, d_in), np.float32) if zero_vec else _bf16(rng.standard_normal((rows, d_in)))
        Go = np.zeros((rows, d_out), np.float32) if zero_vec else _bf16(rng.standard_normal((rows, d_out)) * 1e-3)
        return dict(G=G, A=A, Gout=Go, a=O.rank1_means(A), g=O.rank1_means(Go))
    sa = (r, d_in) if r > 1 else (d_in,)
    sg = (r, d_out) if r > 1 else (d_out,)
    if zero_vec:
        return dict(G=G, a=np.zeros(sa, np.float32), g=np.zeros(sg, np.float32))
    return dict(G=G, a=(rng.standard_normal(sa) / math.sqrt(d_in)).astype(np.float32),
                g=(rng.standard_normal(sg) / math.sqrt(d_out)).astype(np.float32))


def test_degenerate_cases_every_path():
    rng = np.random.default_rng(404)
    layers = [_alloc(sp) for sp in SPECS]
    state = []
    for k, (L, sp) in enumerate(zip(layers, SPECS)):
        d_in, d_out = sp["shape"]
        Li, Ri = spd(500 + 2 * k, d_in, 0.3), spd(501 + 2 * k, d_out, 0.3)
        if sp.get("half"):
            Li, Ri = _bf16(Li), _bf16(Ri)
        H.set_factors(L, Li, Ri)
        state.append([Li.astype(np.float64), Ri.astype(np.float64)])
    plan = H.make_plan(layers)
    # (zero vectors, zero G, params): each call's case
    cases = [(True, False, Params(gamma=0.9, zeta=0.5, eps=math.inf)),
             (False, True, Params(gamma=0.9, zeta=0.5, eps=math.inf)),
             (False, True, Params(gamma=0.9, zeta=0.5, eps=math.inf, rescale=False)),
             (False, False, Params(gamma=0.8, zeta=1.0, eps=0.0)),
             (True, True, Params(gamma=0.7, zeta=0.5, eps=0.0))]
    for t, (zv, zg, p) in enumerate(cases):
        op = oparams(p)
        xs = [_inputs(rng, sp, zv, zg) for sp in SPECS]
        for L, sp, x in zip(layers, SPECS, xs):
            H.set_inputs(L, G=x["G"])
            if sp.get("rows"):
                H.set_rows(L, x["A"], x["Gout"])
            else:
                H.set_inputs(L, x["a"], x["g"])
        plan.step(p)
        torch.cuda.synchronize()
        for k, (L, sp, x) in enumerate(zip(layers, SPECS, xs)):
            Lo, Ro, dW, ost = _oracle(sp, state[k], x["a"], x["g"], x["G"], op)
            state[k] = [Lo, Ro]
            got = H.get_dW(L)
            assert np.isfinite(got).all(), (t, k)
            st = H.get_stats(L)
            assert bool(st["stab_L"]) == ost.L.stab and bool(st["stab_R"]) == ost.R.stab, (t, k)
            assert not st["skip_L"] and not st["skip_R"] and not st["nonfinite_scale"], (t, k)
            if zg:
                assert not got.any(), (t, k, "dW must be exactly 0 when G = 0")
                if p.rescale:
                    assert st["scale"] == 0.0
                continue
            half = sp.get("half", False)
            tol = (TOL_HALF_STEP if half else TOL_STEP) if t == 0 else (TOL_HALF_FREE if half else TOL_FREE)
            e = rel(got, dW)
            assert e <= tol, (t, k, e)
    plan.sync_factors()
    torch.cuda.synchronize()
    for k, (L, sp) in enumerate(zip(layers, SPECS)):
        Lg, Rg = H.get_factors(L)
        Lo, Ro = state[k]
        if sp.get("half"):
            Lo, Ro = round_bf16(Lo), round_bf16(Ro)
        tol = TOL_HALF_FREE if sp.get("half") else TOL_FREE
        assert rel(Lg, Lo) <= tol and rel(Rg, Ro) <= tol, (k, rel(Lg, Lo), rel(Rg, Ro))


def test_zero_vectors_give_p_over_gamma():
    """One step with a = g = 0 from stored factors: the factors become
    P / gamma, up to the two fp32 roundings of c1 = 1 / gamma and of the
    product (2e-7), on the split path and the fp32 MFMA path."""
    for path in ("split", "fp32"):
        L = H.allocate_layers([(128, 192)], "fp32", gemm_path=path)[0]
        Li, Ri = spd(11, 128, 0.3), spd(12, 192, 0.3)
        H.set_factors(L, Li, Ri)
        H.set_inputs(L, np.zeros(128, np.float32), np.zeros(192, np.float32),
                     (np.random.default_rng(1).standard_normal((128, 192)) * 1e-3).astype(np.float32))
        plan = H.make_plan([L])
        plan.step(Params(gamma=0.9, eps=math.inf))
        plan.sync_factors()
        torch.cuda.synchronize()
        Lg, Rg = H.get_factors(L)
        assert rel(Lg, Li.astype(np.float64) / 0.9) <= 2e-7 and rel(Rg, Ri.astype(np.float64) / 0.9) <= 2e-7, path
