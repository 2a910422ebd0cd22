"""Out-of-bounds writes.  Every caller buffer and the plan's workspace sit
between guard regions filled with a byte pattern (harness.Guarded); after
multi-step runs at ragged sizes, whose edge tiles load clamped rows and must
never store past the edge, on every GEMM path (fp32 MFMA, the three-way bf16
split in both associations, bf16 factors), with the stabiliser's
diagonal-shift variants, rank-r and token-row layers, the fused optimizer, a
runtime mode switch and the no-allocation entry point, every guard must still
hold its pattern."""
import math

import pytest
import torch

from paper_2306_01685_amd import OPT_LAMB, OptParams, Params, binding as B, harness as H

pytestmark = pytest.mark.gpu

# (shape, G dtype, extra allocate_layers arguments)
SPECS = [
    ((37, 100), "fp32", {}), ((130, 250), "fp32", {}), ((250, 130), "bf16", {}),        # fp32 MFMA, ragged
    ((320, 192), "fp32", {}), ((576, 320), "bf16", {}), ((64, 448), "bf16", {}),         # split (576: swapped)
    ((320, 192), "fp32", dict(factor_dtype="bf16")), ((128, 704), "bf16", dict(factor_dtype="bf16")),
    ((96, 160), "fp32", dict(rank=2)),                                                   # rank-2
    ((200, 72), "fp32", dict(rows=1000, act_dtype="bf16")),                              # means from rows
    ((64, 96), "fp32", dict(second_order=[False])),                                      # first-order
]


def _layers(guards, optimizer=None):
    layers = []
    for shape, gdt, kw in SPECS:
        layers += H.allocate_layers([shape], gdt, guards=guards, optimizer=optimizer, **kw)
    return layers


def _fill(layers, gen):
    for L in layers:
        d_in, d_out = L["d_in"], L["d_out"]
        for k, std in (("a", 1.0 / math.sqrt(d_in)), ("g", 1.0 / math.sqrt(d_out)), ("G", 1e-3),
                       ("A", 1.0), ("Gout", 1e-3), ("W", 0.02)):
            if k in L:
                t = torch.empty(L[k].shape, dtype=torch.float32, device="cuda")
                t.normal_(0.0, std, generator=gen)
                L[k].copy_(t)


def test_guard_regions_intact_after_every_entry_point():
    guards = H.Guarded()
    layers = _layers(guards, optimizer="lamb")
    ws_bytes = B.workspace_size_raw(B.layer_descs(layers))
    ws = guards.empty((ws_bytes,), torch.uint8)
    plan = H.make_plan(layers, workspace=ws)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4242)
    torch.cuda.synchronize()
    assert guards.intact()
    for t in range(6):
        _fill(layers, gen)
        # eps = 2 and eps = 0 (every factor blended: the diagonal-shift variants)
        p = Params(gamma=0.9, zeta=0.5, eps=0.0 if t % 3 == 2 else 2.0)
        if t == 3:
            plan.precondition(p)
        elif t == 4:
            plan.step_opt(p, OptParams(kind=OPT_LAMB, step=1, lr=1e-3, store_dw=True))
        else:
            plan.step(p)
        if t == 1:
            plan.sync_factors()
        if t == 4:
            plan.set_second_order([0, 1, 0, 1, 0, 1, 0, 1, 0, 1, 0])
    plan.precondition_opt(Params(), OptParams(kind=OPT_LAMB, step=2, lr=1e-3))
    plan.sync_factors()
    torch.cuda.synchronize()
    assert guards.intact(), "a kernel wrote outside a caller buffer or the workspace"
    for L in layers:
        assert bool(torch.isfinite(L["dW"]).all())
    # the no-allocation entry point on the same buffers (its workspace is the
    # library's own array)
    small = [L for L in layers if L["d_in"] * L["d_out"] <= 64 * 704 and "opt_m" in L]
    _fill(small, gen)
    B.step_noalloc(small, Params(eps=2.0))
    torch.cuda.synchronize()
    assert guards.intact(), "the no-allocation step wrote outside a caller buffer"
