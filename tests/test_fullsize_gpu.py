"""Parity at the full workload sizes, in the launch configuration the bench
times (every layer of the set in one grouped launch per kernel).

The oracle follows a sample of layers (one of each shape, or two blocks)
step by step; the other layers run alongside with seeded inputs.  Checks at
step 1 (against the one-step bar), and at steps 49 and 50 (the free-running
bar): the factor check at step 1 writes the pending terms back, after which a
lazily written factor carries two pending terms on odd steps and one on even
steps, so steps 49 and 50 cover both forms of the preconditioning.  Where the full float64
preconditioning would be too slow (the 8192 x 8192 layer), the check uses
sampled rows of dW_hat (row i of Linv G Rinv depends only on row i of Linv)
plus the rescale property ||dW||_F = ||G||_F.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from paper_2306_01685_amd import OPT_LAMB, OptParams, Params, harness as H
from tests.parity import TOL_FREE, TOL_HALF_FREE, TOL_HALF_STEP, TOL_STEP, FreeRun, oparams, rel

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _free_run(w, steps, eps, sample, check_steps, gemm_path=None):
    fr = FreeRun(w, Params(gamma=w.gamma, zeta=0.5, eps=eps), sample=sample, gemm_path=gemm_path)
    worst = {}
    for t in range(steps):
        check = (t + 1) in check_steps
        out = fr.step(precond_oracle=check)
        if check:
            tol = TOL_STEP if t == 0 else TOL_FREE
            worst[t + 1] = (fr.check_factors(tol), fr.check_dW(out, tol))
    fired = fr.check_flags()
    return fr, worst, fired


def test_bert_base_72_layers_50_steps():
    fr, worst, fired = _free_run(W.BERT_BASE, 50, 100.0, sample=[0, 4, 5], check_steps={1, 49, 50})
    print("bert-base worst errors", worst, "stabiliser fired", fired)
    assert fired > 0


@pytest.mark.parametrize("gemm_path", ["auto", "fp32"])
def test_bert_large_144_layers_50_steps(gemm_path):
    """auto: the split path (every shape is a multiple of 64), as timed by the
    bench; fp32: the fp32 MFMA path."""
    fr, worst, fired = _free_run(W.BERT_LARGE, 50, 100.0, sample=[0, 4, 5, 138], check_steps={1, 49, 50},
                                 gemm_path=gemm_path)
    print("bert-large", gemm_path, "worst errors", worst, "stabiliser fired", fired)
    assert fired > 0


@pytest.mark.parametrize("gemm_path", ["auto", "fp32"])
def test_gpt2_xl_192_layers_two_blocks_50_steps(gemm_path):
    """GPT-2-XL set: all 192 layers stepped 50 times; the oracle follows two
    blocks (8 layers, every shape twice: 1600x4800, 1600x1600, 1600x6400,
    6400x1600).  eps = 100 fires within the run."""
    fr, worst, fired = _free_run(W.GPT2_XL, 50, 100.0, sample=list(range(8)), check_steps={1, 49, 50},
                                 gemm_path=gemm_path)
    print("gpt2-xl", gemm_path, "worst errors", worst, "stabiliser fired", fired)
    assert fired > 0


def test_gpt2_xl_explicit_student_t_means_one_step():
    """One step of the GPT-2-XL set with the rank-1 means of one block formed
    explicitly from 32768 Student-t(4) activation rows and 32768 N(0, 1e-6)
    gradient rows (the other tests draw the mean's distribution directly)."""
    w = W.GPT2_XL
    fr = FreeRun(w, Params(gamma=w.gamma, zeta=0.5, eps=100.0), sample=[0, 1, 2, 3], explicit=True)
    out = fr.step(precond_oracle=True)
    e = (fr.check_factors(TOL_STEP), fr.check_dW(out, TOL_STEP))
    print("gpt2-xl explicit Student-t means, step 1 worst errors (factors, dW)", e)


def test_bert_large_bf16_factors_20_steps():
    """The bench's half-precision leg: all 144 layers with bf16 factors in one
    grouped launch per kernel, 20 steps; the half-precision oracle follows a
    1024 x 1024 and a 4096 x 1024 layer (stored factors against the bf16
    rounding of its factors)."""
    w = W.BERT_LARGE
    fr = FreeRun(w, Params(gamma=w.gamma, zeta=0.5, eps=100.0), sample=[0, 5], half=True)
    worst = {}
    for t in range(20):
        check = (t + 1) in (1, 19, 20)
        out = fr.step(precond_oracle=check)
        if check:
            tf, td = (1e-3, TOL_HALF_STEP) if t == 0 else (TOL_HALF_FREE, TOL_HALF_FREE)
            worst[t + 1] = (fr.check_factors(tf), fr.check_dW(out, td))
    fr.check_flags()
    print("bert-large bf16 factors worst errors", worst)


def test_bert_large_update_every_10_steps():
    """The bench's schedule_f10 leg on the default path: factors updated on
    steps 1 and 11, the steps between precondition with the stale factors
    (pending terms held across them); dW of update and precondition-only steps
    against the oracle, factors at the end."""
    w = W.BERT_LARGE
    fr = FreeRun(w, Params(gamma=w.gamma, zeta=0.5, eps=100.0), sample=[0, 4, 5])
    worst = {}
    for t in range(13):
        update = t % 10 == 0
        check = t in (0, 1, 9, 10, 12)
        out = fr.step(precond_oracle=check, update=update)
        if check:
            worst[t + 1] = fr.check_dW(out, TOL_STEP if t <= 1 else TOL_FREE)
    worst["factors"] = fr.check_factors(TOL_FREE)
    print("bert-large update every 10 worst errors", worst)


def test_bert_large_fused_lamb_3_steps():
    """The bench's fused-optimizer leg: all 144 layers with weights and LAMB
    moments, three mkor_step_opt calls; dW, weights and moments of two sampled
    layers against the oracle."""
    w = W.BERT_LARGE
    fr = FreeRun(w, Params(gamma=w.gamma, zeta=0.5, eps=100.0), sample=[0, 5], optimizer="lamb")
    worst = []
    for t in range(3):
        out = fr.step(precond_oracle=True, opt=OptParams(kind=OPT_LAMB, step=t + 1, lr=1e-3, store_dw=True))
        worst.append((fr.check_dW(out, TOL_STEP), fr.check_optimizer(TOL_STEP)))
    print("bert-large fused LAMB worst errors (dW, W/m/v)", worst)


def test_bert_large_mixed_first_order_layers():
    """Algorithm 1's else-branch at scale: the BERT-Large set with every layer
    i = 3 (mod 5) planned first-order (each of the six positions of a block,
    so every shape, is first-order in some block), all 144 layers in one
    grouped launch per kernel, three steps.  Every first-order layer gets dW = G bit for bit; one second-order
    layer of each shape follows the oracle (dW each step, factors at the end).
    """
    w = W.BERT_LARGE
    so = [i % 5 != 3 for i in range(w.n_layers)]
    assert {i % 6 for i in range(w.n_layers) if not so[i]} == set(range(6))
    sample = [0, 4, 5]   # 1024 x 1024, 1024 x 4096, 4096 x 1024, all second-order
    assert all(so[i] for i in sample)
    layers = H.allocate_layers(w.shapes, w.grad_dtype, second_order=so)
    plan = H.make_plan(layers)
    p = Params(gamma=w.gamma, zeta=0.5, eps=100.0)
    op = oparams(p)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4321)
    state = {i: [np.eye(w.shapes[i][0]), np.eye(w.shapes[i][1])] for i in sample}
    worst = 0.0
    for t in range(3):
        host = {}
        for i, L in enumerate(layers):
            if i in sample:
                a, g = W.rank1_vectors(w, i, t)
                G = W.gradient(w, i, t)
                H.set_inputs(L, a, g, G)
                host[i] = (a, g, G)
                continue
            if so[i]:
                L["a"].normal_(0.0, 1.0 / math.sqrt(w.rows), generator=gen)
                L["g"].normal_(0.0, w.grad_row_std / math.sqrt(w.rows), generator=gen)
            tmp = torch.empty(L["G"].shape, dtype=torch.float32, device="cuda")
            tmp.normal_(0.0, w.G_std, generator=gen)
            L["G"].copy_(tmp)
        plan.step(p)
        torch.cuda.synchronize()
        for i, L in enumerate(layers):
            if not so[i]:
                assert torch.equal(L["dW"], L["G"].float()), (t, i)
        for i, (a, g, G) in host.items():
            Lo, Ro, dW, _ = O.layer_step(state[i][0], state[i][1], a, g, G, op)
            state[i] = [Lo, Ro]
            e = rel(H.get_dW(layers[i]), dW)
            worst = max(worst, e)
            assert e <= (TOL_STEP if t == 0 else TOL_FREE), (t, i, e)
    plan.sync_factors()
    torch.cuda.synchronize()
    for i in sample:
        Lg, Rg = H.get_factors(layers[i])
        assert rel(Lg, state[i][0]) <= TOL_FREE and rel(Rg, state[i][1]) <= TOL_FREE, i
    print("bert-large with first-order layers: worst dW error", worst)


def _sampled_rows_check(L, Lo, Ro, G, rows, tol):
    dW = H.get_dW(L)
    st = H.get_stats(L)
    # rescale property on the GPU output itself
    nG = float(np.linalg.norm(G.astype(np.float64)))
    assert float(np.linalg.norm(dW.astype(np.float64))) == pytest.approx(nG, rel=1e-5)
    assert st["norm_G"] == pytest.approx(nG, rel=1e-5)
    ref_rows = O.precondition(Lo[rows], G, Ro)
    got_rows = dW[rows].astype(np.float64) / st["scale"]
    e = rel(got_rows, ref_rows)
    assert e <= tol, e
    return e


def test_single_8192_layer_20_steps():
    """8192 x 8192, perturbed SPD init, gamma = 0.95, 20 steps; eps = 2 fires
    around step 13."""
    w = W.SINGLE_8192
    fr = FreeRun(w, Params(gamma=w.gamma, zeta=0.5, eps=2.0), sample=[0])
    rows = np.random.default_rng(5).choice(8192, size=96, replace=False)
    G_last = None
    for t in range(w.steps):
        fr.step(precond_oracle=False)
        G_last = W.gradient(w, 0, t)
        if t == 0:
            fr.check_factors(TOL_STEP)
            _sampled_rows_check(fr.layers[0], *fr.state[0], G_last, rows, TOL_STEP)
    fr.check_factors(TOL_FREE)
    e = _sampled_rows_check(fr.layers[0], *fr.state[0], G_last, rows, TOL_FREE)
    fired = fr.check_flags()
    print("8192 layer: sampled-row dW error", e, "stabiliser fired", fired)
    assert fired > 0


def _identity_update_k(x, gamma):
    """From P = I the oracle's update is (1/gamma)(I - k x x^T) with
    k = (1 - gamma) / (gamma + (1 - gamma) x^T x) (the SM step with P_hat = I,
    u = x, s = x^T x); returns k."""
    x = np.asarray(x, np.float64)
    return (1.0 - gamma) / (gamma + (1.0 - gamma) * float(x @ x))


@pytest.mark.parametrize("path", ["auto", "fp32", "bf16f"])
def test_max_dim_layer_one_step(path):
    """The largest layer the ABI accepts, MKOR_MAX_DIM x MKOR_MAX_DIM (32768):
    each fp32 factor is 4 GiB and the kernels form their largest offsets.  bf16
    G, factors from the identity, one step on the split path (auto), the fp32
    MFMA path, or with bf16 factors.  From the identity the oracle's update has
    a closed form, checked against the oracle itself at d = 64 first; then every
    element of both factors is compared with it (1024 rows at a time; with bf16
    factors, with its bf16 rounding), and the rescale property ||dW|| = ||G||.
    fp32 factors: sampled rows of dW_hat through Linv[i, :] G Rinv =
    (G[i, :] - kL a_i (a^T G)) Rinv.  (With bf16 factors a row of dW_hat needs
    all of the bf16-rounded Y = G Rinv, out of the CPU's reach at this size.)"""
    import paper_2306_01685_amd as M
    from oracle.half import round_bf16

    gamma = 0.9
    p = Params(gamma=gamma, zeta=0.5, eps=100.0)
    op = oparams(p)
    x64 = np.random.default_rng(64).standard_normal(64) / 8.0
    P1, st1 = O.update_factor(np.eye(64), x64, op)
    k64 = _identity_update_k(x64, gamma)
    assert not st1.stab
    assert rel(P1, (np.eye(64) - k64 * np.outer(x64, x64)) / gamma) <= 1e-14

    d = M.MAX_DIM
    half = path == "bf16f"
    L = H.allocate_layers([(d, d)], "bf16", factor_dtype="bf16" if half else "fp32",
                          gemm_path=None if half else path)[0]
    rng = np.random.default_rng(32768)
    a = (rng.standard_normal(d) / math.sqrt(d)).astype(np.float32)
    g = (rng.standard_normal(d) / math.sqrt(d)).astype(np.float32)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    tmp = torch.empty((d, d), dtype=torch.float32, device="cuda")
    tmp.normal_(0.0, 1e-3, generator=gen)
    L["G"].copy_(tmp)
    del tmp
    torch.cuda.empty_cache()
    H.set_inputs(L, a, g)
    plan = H.make_plan([L])
    plan.step(p)
    plan.sync_factors()
    torch.cuda.synchronize()
    st = H.get_stats(L)
    assert not st["stab_L"] and not st["stab_R"]

    kL, kR = _identity_update_k(a, gamma), _identity_update_k(g, gamma)
    a64, g64 = a.astype(np.float64), g.astype(np.float64)
    worst_f = 0.0
    aG = np.zeros(d)        # a^T G, accumulated over row blocks of G
    nG2 = 0.0
    CH = 1024
    for r0 in range(0, d, CH):
        r1 = r0 + CH
        for key, x, k in (("Linv", a64, kL), ("Rinv", g64, kR)):
            got = L[key][r0:r1].float().cpu().numpy().astype(np.float64)
            want = -k * np.outer(x[r0:r1], x)
            want[np.arange(CH), np.arange(r0, r1)] += 1.0
            want /= gamma
            if half:
                want = round_bf16(want)
            e = rel(got, want)
            worst_f = max(worst_f, e)
            assert e <= (1e-3 if half else TOL_STEP), (key, r0, e)
        Gb = L["G"][r0:r1].float().cpu().numpy().astype(np.float64)
        aG += a64[r0:r1] @ Gb
        nG2 += float((Gb * Gb).sum())
    nG = math.sqrt(nG2)
    assert st["norm_G"] == pytest.approx(nG, rel=2e-7)
    nW = float(torch.linalg.vector_norm(L["dW"], dtype=torch.float64))
    assert nW == pytest.approx(nG, rel=2e-7)
    if half:
        print("max-dim layer, bf16 factors: worst factor block error", worst_f)
        return
    rows = np.concatenate([[0, d - 1], np.random.default_rng(9).choice(d, size=14, replace=False)])
    Grows = L["G"][torch.from_numpy(rows).cuda()].float().cpu().numpy().astype(np.float64)
    v = (Grows - kL * np.outer(a64[rows], aG)) / gamma                   # rows of Linv G
    ref = (v - kR * np.outer(v @ g64, g64)) / gamma                      # rows of Linv G Rinv
    got = L["dW"][torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64) / st["scale"]
    e = rel(got, ref)
    assert e <= TOL_STEP, e
    print("max-dim layer", path, ": worst factor block error", worst_f, "sampled dW_hat rows error", e)
