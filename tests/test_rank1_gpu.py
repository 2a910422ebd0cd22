"""GPU parity of the rank-1 means (Algorithm 1, its first two lines) and of a
step driven by token rows, through the C ABI, against the float64 oracle.

The library sums in float64 and rounds once, so a and g must equal the float64
mean rounded to fp32 up to float64 summation-order effects (checked elementwise
at 2 fp32 ulps); steps driven by rows meet the usual 1e-4 / 1e-3 bars.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from paper_2306_01685_amd import Params, harness as H
from tests.parity import TOL_FREE, TOL_STEP, check_close, oparams

pytestmark = pytest.mark.gpu

SHAPES = [(1, 1), (3, 5), (64, 100), (100, 37), (256, 257), (1000, 64)]
ROWS = [1, 3, 1000, 1025, 2048]


def _mean_check(got, rows):
    want = O.rank1_means(rows).astype(np.float32)
    np.testing.assert_array_max_ulp(got, want, maxulp=2)


@pytest.mark.parametrize("dt", ["fp32", "bf16"])
@pytest.mark.parametrize("rows", ROWS)
def test_means_ragged(dt, rows):
    w = W.custom(SHAPES, rows=rows, cid=300 + rows)
    layers = H.allocate_layers(SHAPES, "fp32", rows=rows, act_dtype=dt)
    host = []
    for i, L in enumerate(layers):
        A, Go = W.token_rows(w, i, 0, dtype=dt)
        H.set_rows(L, A, Go)
        H.set_inputs(L, G=W.gradient(w, i, 0))
        host.append((A, Go))
    plan = H.make_plan(layers)
    plan.run_stage(Params(), 0)   # the means stage alone
    torch.cuda.synchronize()
    for L, (A, Go) in zip(layers, host):
        a, g = H.get_means(L)
        _mean_check(a, A)
        _mean_check(g, Go)


def test_step_from_rows_free_running():
    """cfg1 shape (64 x 64, 32 token rows) plus ragged layers, 20 steps, both
    sides forming the means from the same rows."""
    shapes = [(64, 64), (37, 100), (128, 256)]
    w = W.custom(shapes, grad_dtype="bf16", rows=32, cid=333, gamma=0.9)
    p = Params(gamma=0.9, eps=4.0)
    op = oparams(p)
    layers = H.allocate_layers(shapes, "bf16", rows=32, act_dtype="bf16")
    plan = H.make_plan(layers)
    state = [(np.eye(i), np.eye(o)) for i, o in shapes]
    fired = 0
    for t in range(20):
        step_in = []
        for i, L in enumerate(layers):
            A, Go = W.token_rows(w, i, t, dtype="bf16")
            G = W.gradient(w, i, t)
            H.set_rows(L, A, Go)
            H.set_inputs(L, G=G)
            step_in.append((A, Go, G))
        plan.step(p)
        torch.cuda.synchronize()
        for i, L in enumerate(layers):
            A, Go, G = step_in[i]
            st = H.get_stats(L)
            Lp, Rp = state[i]
            Li, Ri, dW, ost, a, g = O.layer_step_rows(Lp, Rp, A, Go, G, op)
            fired += int(ost.L.stab) + int(ost.R.stab)
            assert bool(ost.L.stab) == bool(st["stab_L"]) and bool(ost.R.stab) == bool(st["stab_R"])
            state[i] = (Li, Ri)
            check_close(H.get_dW(L), dW, TOL_STEP if t == 0 else TOL_FREE, i, t)
            ga, gg = H.get_means(L)
            np.testing.assert_array_max_ulp(ga, a.astype(np.float32), maxulp=2)
            np.testing.assert_array_max_ulp(gg, g.astype(np.float32), maxulp=2)
    plan.sync_factors()
    torch.cuda.synchronize()
    for i, L in enumerate(layers):
        Lg, Rg = H.get_factors(L)
        check_close(Lg, state[i][0], TOL_FREE, i, "L")
        check_close(Rg, state[i][1], TOL_FREE, i, "R")
    assert fired > 0


def test_update_every_f_steps():
    """Update frequency f = 3 (the paper updates every 10 iterations): mkor_step
    on update steps, mkor_precondition (stale factors) on the others."""
    shapes = [(64, 96), (100, 37)]
    w = W.custom(shapes, rows=16, cid=350)
    p = Params(gamma=0.9, eps=math.inf)
    op = oparams(p)
    layers = H.allocate_layers(shapes, "fp32")
    plan = H.make_plan(layers)
    state = [(np.eye(i), np.eye(o)) for i, o in shapes]
    for t in range(9):
        update = t % 3 == 0
        ins = []
        for i, L in enumerate(layers):
            a, g = W.rank1_vectors(w, i, t)
            G = W.gradient(w, i, t)
            H.set_inputs(L, a, g, G)
            ins.append((a, g, G))
        if update:
            plan.step(p)
        else:
            plan.precondition(p)
        torch.cuda.synchronize()
        for i, L in enumerate(layers):
            a, g, G = ins[i]
            Li, Ri, dW, _ = O.layer_step(*state[i], a, g, G, op, update=update)
            state[i] = (Li, Ri)
            check_close(H.get_dW(L), dW, TOL_STEP if t == 0 else TOL_FREE, i, t)


@pytest.mark.slow
def test_bert_large_means_from_16384_bf16_rows():
    """Full BERT-Large layer set with 16384 bf16 token rows per layer (14.5 GB of
    rows): means of sampled layers against the oracle, one full step."""
    w = W.BERT_LARGE
    sample = [0, 4, 5]
    layers = H.allocate_layers(w.shapes, w.grad_dtype, stats=False, rows=w.rows, act_dtype="bf16")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(77)
    host = {}
    for i, L in enumerate(layers):
        if i in sample:
            A, Go = W.token_rows(w, i, 0, dtype="bf16")
            H.set_rows(L, A, Go)
            host[i] = (A, Go)
        else:
            for k in ("A", "Gout"):
                tmp = torch.empty(L[k].shape, dtype=torch.float32, device="cuda")
                tmp.normal_(0.0, 1.0, generator=gen)
                L[k].copy_(tmp)
                del tmp
    plan = H.make_plan(layers)
    plan.step(Params(gamma=w.gamma))
    torch.cuda.synchronize()
    for i, (A, Go) in host.items():
        a, g = H.get_means(layers[i])
        _mean_check(a, A)
        _mean_check(g, Go)


def _plan_rows_per_block(shapes, rows):
    """The plan's rows per block of the mean partials: the largest power of
    two in [512, 8192] that gives at least 1024 blocks of (matrix, 512-column
    chunk, row block) over the plan, else 512."""
    for rpb in (8192, 4096, 2048, 1024):
        blocks = sum((-(-i // 512) + -(-o // 512)) * -(-rows // rpb) for i, o in shapes)
        if blocks >= 1024:
            return rpb
    return 512


# (layer count, shape, rows per layer) -> the plan's rows per block; the rows
# are never a multiple of it, so every matrix ends in a short block
INTERMEDIATE = [(8, (4096, 4096), 7500, 1024), (128, (512, 512), 10000, 2048), (96, (1024, 1024), 12000, 4096)]


@pytest.mark.parametrize("n,shape,rows,rpb", INTERMEDIATE)
def test_means_at_intermediate_row_blocks(n, shape, rows, rpb):
    """Plans whose size puts the mean partials at 1024, 2048 and 4096 rows per
    block (the small and the largest choices are covered above and at full
    size): every matrix's means against its float64 column means, sampled
    ones against the oracle, and their step against the oracle."""
    shapes = [shape] * n
    assert _plan_rows_per_block(shapes, rows) == rpb and rows % rpb
    layers = H.allocate_layers(shapes, "fp32", stats=False, rows=rows, act_dtype="bf16")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(rows)
    sample = [0, n // 2, n - 1]
    rng = np.random.default_rng(rows)
    host = {}
    for i, L in enumerate(layers):
        if i in sample:
            A = W.round_to_bf16(rng.standard_normal((rows, shape[0])).astype(np.float32))
            Go = W.round_to_bf16((rng.standard_normal((rows, shape[1])) * 1e-3).astype(np.float32))
            G = (rng.standard_normal(shape) * 1e-3).astype(np.float32)
            H.set_rows(L, A, Go)
            H.set_inputs(L, G=G)
            host[i] = (A, Go, G)
        else:
            for k in ("A", "Gout"):
                tmp = torch.empty(L[k].shape, dtype=torch.float32, device="cuda")
                tmp.normal_(0.0, 1.0, generator=gen)
                L[k].copy_(tmp)
                del tmp
    plan = H.make_plan(layers)
    p = Params(gamma=0.9, eps=math.inf)
    plan.step(p)
    torch.cuda.synchronize()
    for i, L in enumerate(layers):
        a, g = H.get_means(L)
        for got, key in ((a, "A"), (g, "Gout")):
            want = L[key].double().sum(dim=0).div(rows).float().cpu().numpy()
            np.testing.assert_array_max_ulp(got, want, maxulp=2)
    plan.sync_factors()
    torch.cuda.synchronize()
    op = oparams(p)
    for i, (A, Go, G) in host.items():
        a, g = H.get_means(layers[i])
        _mean_check(a, A)
        _mean_check(g, Go)
        Lo, Ro, dW, _ = O.layer_step(np.eye(shape[0]), np.eye(shape[1]), O.rank1_means(A), O.rank1_means(Go), G, op)
        check_close(H.get_dW(layers[i]), dW, TOL_STEP, i, "dW")
        Lg, Rg = H.get_factors(layers[i])
        check_close(Lg, Lo, TOL_STEP, i, "L")
        check_close(Rg, Ro, TOL_STEP, i, "R")


@pytest.mark.slow
def test_max_rows_means_and_step():
    """The largest token-row count the ABI accepts, MKOR_MAX_ROWS = 2^26 bf16
    rows for each of A and Gout of a 64 x 64 layer (8 GiB per matrix, so row
    offsets pass 2^32 bytes).  The means against the float64 column means of
    the same stored rows (streamed back in chunks, at 2 fp32 ulps), and the step
    they drive against the oracle."""
    import paper_2306_01685_amd as M

    n, d, CH = M.MAX_ROWS, 64, 1 << 22
    L = H.allocate_layers([(d, d)], "fp32", rows=n, act_dtype="bf16")[0]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(26)
    for key, std in (("A", 1.0), ("Gout", 1e-3)):
        tmp = torch.empty((CH, d), dtype=torch.float32, device="cuda")
        for r0 in range(0, n, CH):
            tmp.normal_(0.0, std, generator=gen)
            L[key][r0:r0 + CH].copy_(tmp)
        del tmp
    G = (np.random.default_rng(3).standard_normal((d, d)) * 1e-3).astype(np.float32)
    H.set_inputs(L, G=G)
    plan = H.make_plan([L])
    p = Params()
    plan.step(p)
    torch.cuda.synchronize()
    a, g = H.get_means(L)
    means = {}
    for key in ("A", "Gout"):
        s = np.zeros(d)
        for r0 in range(0, n, CH):
            s += L[key][r0:r0 + CH].float().cpu().numpy().astype(np.float64).sum(axis=0)
        means[key] = s / n
    np.testing.assert_array_max_ulp(a, means["A"].astype(np.float32), maxulp=2)
    np.testing.assert_array_max_ulp(g, means["Gout"].astype(np.float32), maxulp=2)
    Lo, Ro, dW, _ = O.layer_step(np.eye(d), np.eye(d), means["A"], means["Gout"], G, oparams(p))
    e = check_close(H.get_dW(L), dW, TOL_STEP, "dW")
    plan.sync_factors()
    torch.cuda.synchronize()
    Lg, Rg = H.get_factors(L)
    check_close(Lg, Lo, TOL_STEP, "L")
    check_close(Rg, Ro, TOL_STEP, "R")
    print("max rows: dW error", e)
