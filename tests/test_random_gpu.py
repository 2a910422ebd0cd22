"""Randomised parity: seeded random plans that mix what the other GPU tests
take one at a time, each followed by the oracle for three calls (step,
precondition only, step).

Per plan: 1 to 4 layers with random sizes (1 to 300 on the fp32 MFMA path;
multiples of 64 up to 320 on the split path and for bf16 factors), fp32 or
bf16 G, fp32 or bf16 factors, rank 1 to 3, means handed in or formed from
token rows (fp32 or bf16 rows), first-order layers; random gamma, zeta, eps
(off, 0, or near the factors' norms, so the stabiliser fires on some factors
and not others), norm kind, SM variant (the printed formula only in plans
without rank-r layers) and rescale on or off.  Bars as everywhere: the
one-step bar after the first call, the free-running bar after it (the bf16
factor bars for bf16-factor layers); first-order layers give dW = G bit for
bit; stabiliser decisions agree outside the near-tie band.
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
from tests.parity import TOL_FREE, TOL_HALF_FREE, TOL_HALF_STEP, TOL_STEP, near_tie, oparams, rel, relmax, spd

pytestmark = pytest.mark.gpu

N_PLANS = 120
M64 = [64, 128, 192, 256, 320]


def _spec(rng):
    so = rng.random() > 0.15
    half = so and rng.random() < 0.25
    path = "fp32" if half else rng.choice(["fp32", "split", "auto"])
    aligned = half or path in ("split", "auto") and rng.random() < 0.8
    if aligned:
        path = path if not half else None
        d_in, d_out = int(rng.choice(M64)), int(rng.choice(M64))
    else:
        path = "fp32" if path == "split" else path
        d_in, d_out = int(rng.integers(1, 301)), int(rng.integers(1, 301))
    rank = int(rng.integers(2, 4)) if (so and not half and rng.random() < 0.25) else 1
    rows = int(rng.choice([1, 33, 200])) if (so and rank == 1 and rng.random() < 0.25) else 0
    return dict(d_in=d_in, d_out=d_out, so=so, half=half, path=path, rank=rank, rows=rows,
                gdt="bf16" if rng.random() < 0.5 else "fp32", adt="bf16" if rng.random() < 0.5 else "fp32")


def _bf16(x):
    return W.round_to_bf16(np.asarray(x, np.float32))


def _alloc(sp):
    return H.allocate_layers([(sp["d_in"], sp["d_out"])], sp["gdt"], second_order=[sp["so"]],
                             factor_dtype="bf16" if sp["half"] else "fp32", rank=sp["rank"],
                             rows=sp["rows"], act_dtype=sp["adt"], gemm_path=sp["path"])[0]


def _inputs(rng, sp):
    d_in, d_out, r = sp["d_in"], sp["d_out"], sp["rank"]
    G = (rng.standard_normal((d_in, d_out)) * 1e-3).astype(np.float32)
    if sp["gdt"] == "bf16":
        G = _bf16(G)
    if sp["rows"]:
        A = rng.standard_normal((sp["rows"], d_in)).astype(np.float32)
        Gout = (rng.standard_normal((sp["rows"], d_out)) * 1e-3).astype(np.float32)
        if sp["adt"] == "bf16":
            A, Gout = _bf16(A), _bf16(Gout)
        a = O.rank1_means(A)
        g = O.rank1_means(Gout)
        return dict(G=G, A=A, Gout=Gout, a=a, g=g)
    shape_a = (r, d_in) if r > 1 else (d_in,)
    shape_g = (r, d_out) if r > 1 else (d_out,)
    a = (rng.standard_normal(shape_a) / math.sqrt(d_in)).astype(np.float32)
    g = (rng.standard_normal(shape_g) / math.sqrt(d_out)).astype(np.float32)
    return dict(G=G, a=a, g=g)


def _feed(L, sp, x, update):
    if not sp["so"]:
        H.set_inputs(L, G=x["G"])
    elif sp["rows"]:
        H.set_inputs(L, G=x["G"])
        if update:
            H.set_rows(L, x["A"], x["Gout"])
    else:
        H.set_inputs(L, x["a"], x["g"], x["G"])


def _oracle(sp, st, x, op, flags, update):
    """The layer's oracle call; adopts the GPU's stabiliser decision only in
    the near-tie band, and fails on any other disagreement."""
    a, g, G = x["a"], x["g"], x["G"]

    def run(ov):
        if sp["half"]:
            return layer_step_half(st[0], st[1], a, g, G, op, ov, update=update)
        if sp["rank"] > 1:
            return layer_step_rank(st[0], st[1], a.T, g.T, G, op, ov, update=update)
        return O.layer_step(st[0], st[1], a, g, G, op, stab_override=ov, update=update)

    Ln, Rn, dW, ost = run((None, None))
    if update:
        ov = tuple(flags[s] if (fs.stab != flags[s] and near_tie(fs.nu, op.eps)) else None
                   for s, fs in (("L", ost.L), ("R", ost.R)))
        if ov != (None, None):
            Ln, Rn, dW, ost = run(ov)
        for s, fs in (("L", ost.L), ("R", ost.R)):
            assert fs.stab == flags[s] or near_tie(fs.nu, op.eps), (s, fs.nu, op.eps, fs.stab, flags[s])
    return [Ln, Rn], dW, ost


@pytest.mark.parametrize("seed", range(N_PLANS))
def test_random_plan(seed):
    rng = np.random.default_rng([2306, seed])
    specs = [_spec(rng) for _ in range(int(rng.integers(1, 5)))]
    has_rank = any(sp["rank"] > 1 for sp in specs)
    layers = [_alloc(sp) for sp in specs]
    state = []
    for k, (L, sp) in enumerate(zip(layers, specs)):
        if not sp["so"]:
            state.append(None)
            continue
        Li, Ri = spd(1000 * seed + 2 * k, sp["d_in"], 0.3), spd(1000 * seed + 2 * k + 1, sp["d_out"], 0.3)
        if sp["half"]:
            Li, Ri = _bf16(Li), _bf16(Ri)
        H.set_factors(L, Li, Ri)
        state.append([Li.astype(np.float64), Ri.astype(np.float64)])
    # eps: off, always, or inside the range of the factors' norms (about 1.3 to 2 here)
    eps = [math.inf, 0.0, float(rng.uniform(1.2, 2.5))][int(rng.integers(0, 3))]
    p = Params(gamma=float(rng.uniform(0.5, 0.99)), zeta=float(rng.uniform(0.1, 0.9)), eps=eps,
               norm_kind=int(rng.integers(0, 2)), variant=0 if has_rank or rng.random() < 0.75 else 1,
               rescale=bool(rng.random() < 0.8))
    op = oparams(p)
    plan = H.make_plan(layers)
    desc = [(sp["d_in"], sp["d_out"], "so" if sp["so"] else "fo", "bf16f" if sp["half"] else sp["path"],
             f"r{sp['rank']}", f"rows{sp['rows']}", sp["gdt"]) for sp in specs]
    print("plan", seed, desc, p, flush=True)
    worst = 0.0
    for t, update in enumerate((True, False, True)):
        xs = [_inputs(rng, sp) for sp in specs]
        for L, sp, x in zip(layers, specs, xs):
            _feed(L, sp, x, update)
        (plan.step if update else plan.precondition)(p)
        torch.cuda.synchronize()
        for k, (L, sp, x) in enumerate(zip(layers, specs, xs)):
            if not sp["so"]:
                assert np.array_equal(H.get_dW(L), x["G"]), (seed, t, k)
                continue
            stt = H.get_stats(L)
            flags = {"L": bool(stt["stab_L"]), "R": bool(stt["stab_R"])}
            state[k], dW, _ = _oracle(sp, state[k], x, op, flags, update)
            tol = (TOL_HALF_STEP if sp["half"] else TOL_STEP) if t == 0 else (TOL_HALF_FREE if sp["half"] else TOL_FREE)
            got = H.get_dW(L)
            e = rel(got, dW)
            worst = max(worst, e)
            assert e <= tol, (seed, t, k, desc[k], e)
            if not sp["half"]:   # element-wise too (bf16: one-ulp rounding flips are legitimate)
                m = relmax(got, dW)
                assert m <= tol, (seed, t, k, desc[k], "element-wise", m)
    plan.sync_factors()
    torch.cuda.synchronize()
    for k, (L, sp) in enumerate(zip(layers, specs)):
        if not sp["so"]:
            continue
        Lg, Rg = H.get_factors(L)
        Lo, Ro = state[k]
        if sp["half"]:
            Lo, Ro = round_bf16(Lo), round_bf16(Ro)
        tol = TOL_HALF_FREE if sp["half"] else TOL_FREE
        assert rel(Lg, Lo) <= tol and rel(Rg, Ro) <= tol, (seed, k, desc[k], rel(Lg, Lo), rel(Rg, Ro))
    print("plan", seed, "worst dW error", worst)


def _f32(x):
    return float(np.float32(x))   # the ABI takes fp32 hyper-parameters


@pytest.mark.parametrize("seed", range(N_PLANS // 2))
def test_random_plan_switch_and_optimizer(seed):
    """Random plans as above with the backend optimizer fused (SGD or LAMB,
    random hyper-parameters) and MKOR-H switches between the calls: a random
    subset of the second-order layers runs the first-order branch for the
    second call (a step or a precondition only), and another random subset for
    the third.  The oracle follows each layer's branch; W, m (and v), and dW
    when stored, are checked after every call."""
    from oracle.optimizer import lamb_step, sgd_step
    from paper_2306_01685_amd import OPT_LAMB, OPT_SGD, OptParams

    rng = np.random.default_rng([2307, seed])
    specs = [_spec(rng) for _ in range(int(rng.integers(1, 5)))]
    lamb = bool(rng.random() < 0.5)
    layers = [H.allocate_layers([(sp["d_in"], sp["d_out"])], sp["gdt"], second_order=[sp["so"]],
                                factor_dtype="bf16" if sp["half"] else "fp32", rank=sp["rank"], rows=sp["rows"],
                                act_dtype=sp["adt"], gemm_path=sp["path"], optimizer="lamb" if lamb else "sgd")[0]
              for sp in specs]
    state, opt = [], []
    for k, (L, sp) in enumerate(zip(layers, specs)):
        shape = (sp["d_in"], sp["d_out"])
        W0 = (rng.standard_normal(shape) * 0.02).astype(np.float32)
        m0 = (rng.standard_normal(shape) * 1e-4).astype(np.float32)
        v0 = np.abs(rng.standard_normal(shape) * 1e-7).astype(np.float32)
        L["W"].copy_(torch.from_numpy(W0))
        L["opt_m"].copy_(torch.from_numpy(m0))
        if lamb:
            L["opt_v"].copy_(torch.from_numpy(v0))
        opt.append([W0.astype(np.float64), m0.astype(np.float64), v0.astype(np.float64)])
        if not sp["so"]:
            state.append(None)
            continue
        Li, Ri = spd(3000 * seed + 2 * k, sp["d_in"], 0.3), spd(3000 * seed + 2 * k + 1, sp["d_out"], 0.3)
        if sp["half"]:
            Li, Ri = _bf16(Li), _bf16(Ri)
        H.set_factors(L, Li, Ri)
        state.append([Li.astype(np.float64), Ri.astype(np.float64)])
    has_rank = any(sp["rank"] > 1 for sp in specs)
    eps = [math.inf, 0.0, float(rng.uniform(1.2, 2.5))][int(rng.integers(0, 3))]
    p = Params(gamma=float(rng.uniform(0.5, 0.99)), zeta=float(rng.uniform(0.1, 0.9)), eps=eps,
               norm_kind=int(rng.integers(0, 2)), variant=0 if has_rank or rng.random() < 0.75 else 1)
    op = oparams(p)
    hp = dict(lr=float(rng.uniform(1e-4, 1e-2)), momentum=float(rng.uniform(0.5, 0.95)),
              beta1=float(rng.uniform(0.8, 0.95)), beta2=float(rng.uniform(0.99, 0.9999)), eps=1e-6,
              weight_decay=float(rng.choice([0.0, 0.01])))
    plan = H.make_plan(layers)
    print("plan", seed, "lamb" if lamb else "sgd", [(sp["d_in"], sp["d_out"], sp["so"], sp["half"], sp["path"],
                                                     sp["rank"], sp["rows"], sp["gdt"]) for sp in specs], p, hp,
          flush=True)
    mode = [bool(sp["so"]) for sp in specs]
    for t, update in enumerate((True, bool(rng.random() < 0.5), True)):
        if t > 0:
            mode = [bool(sp["so"]) and bool(rng.random() < 0.5) for sp in specs]
            plan.set_second_order([int(m) for m in mode])
        store = bool(rng.random() < 0.7)
        o = OptParams(kind=OPT_LAMB if lamb else OPT_SGD, step=t + 1, store_dw=store, **hp)
        xs = [_inputs(rng, sp) for sp in specs]
        for L, sp, x in zip(layers, specs, xs):
            _feed(L, sp, x, update)
        (plan.step_opt if update else plan.precondition_opt)(p, o)
        torch.cuda.synchronize()
        for k, (L, sp, x) in enumerate(zip(layers, specs, xs)):
            if mode[k]:
                stt = H.get_stats(L)
                flags = {"L": bool(stt["stab_L"]), "R": bool(stt["stab_R"])}
                state[k], dW, _ = _oracle(sp, state[k], x, op, flags, update)
                dtol = (TOL_HALF_STEP if sp["half"] else TOL_STEP) if t == 0 else (
                    TOL_HALF_FREE if sp["half"] else TOL_FREE)
            else:
                dW, dtol = x["G"].astype(np.float64), 0.0
            if store:
                e = rel(H.get_dW(L), dW)
                assert e <= dtol, (seed, t, k, "dW", e)
            Wo, mo, vo = opt[k]
            if lamb:
                Wo, mo, vo, _ = lamb_step(Wo, mo, vo, dW, t + 1, _f32(hp["lr"]), _f32(hp["beta1"]),
                                          _f32(hp["beta2"]), _f32(hp["eps"]), _f32(hp["weight_decay"]))
            else:
                Wo, mo = sgd_step(Wo, mo, dW, _f32(hp["lr"]), _f32(hp["momentum"]), _f32(hp["weight_decay"]))
            opt[k] = [Wo, mo, vo]
            # bars: the layer's dW bar (at least the one-step bar, for the rounding of the
            # update itself); twice that for v, which accumulates g^2
            wtol = max(dtol, TOL_STEP)
            checks = [("W", L["W"], Wo, wtol), ("m", L["opt_m"], mo, wtol)]
            if lamb:
                checks.append(("v", L["opt_v"], vo, 2 * wtol))
            for name, got, want, tol in checks:
                e = rel(got.cpu().numpy(), want)
                assert e <= tol, (seed, t, k, name, e)
    plan.sync_factors()
    torch.cuda.synchronize()
    for k, (L, sp) in enumerate(zip(layers, specs)):
        if not sp["so"]:
            continue
        Lg, Rg = H.get_factors(L)
        Lo, Ro = state[k]
        if sp["half"]:
            Lo, Ro = round_bf16(Lo), round_bf16(Ro)
        tol = TOL_HALF_FREE if sp["half"] else TOL_FREE
        assert rel(Lg, Lo) <= tol and rel(Rg, Ro) <= tol, (seed, k, rel(Lg, Lo), rel(Rg, Ro))
