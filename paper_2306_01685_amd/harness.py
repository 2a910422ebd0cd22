"""Device-memory plumbing for a grouped layer list (torch tensors on the GPU).

Allocates the per-layer buffers that the C ABI consumes and moves host arrays
in and out of them.  No arithmetic of the method happens here.
"""
from __future__ import annotations

import numpy as np
import torch

from .binding import STATS_BYTES, MkorPlan, read_stats


class Guarded:
    """Device tensors carved out of larger buffers with a guard region of
    `guard` bytes on each side, filled with a byte pattern, so that a write
    past either end of a tensor shows up in intact()."""

    PATTERN = 0x7F   # 0x7F7F7F7F as fp32 is 3.39e38: finite, unlike anything a kernel writes here

    def __init__(self, guard=4096):
        assert guard % 256 == 0
        self.guard = guard
        self.raws = []

    def empty(self, shape, dtype, device="cuda"):
        nbytes = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        body = (nbytes + 255) // 256 * 256
        raw = torch.full((self.guard + body + self.guard,), self.PATTERN, dtype=torch.uint8, device=device)
        self.raws.append((raw, nbytes))
        return raw[self.guard:self.guard + nbytes].view(dtype).view(shape)

    def intact(self):
        """True when every guard region still holds the pattern (also the
        padding between a tensor's end and its guard)."""
        for raw, nbytes in self.raws:
            g = self.guard
            if not bool((raw[:g] == self.PATTERN).all()) or not bool((raw[g + nbytes:] == self.PATTERN).all()):
                return False
        return True


def allocate_layers(shapes, grad_dtype="fp32", device="cuda", second_order=None, stats=True,
                    rows=0, act_dtype="fp32", factor_dtype="fp32", rank=1, optimizer=None, gemm_path=None,
                    guards=None):
    """One dict of device tensors per (d_in, d_out); factors start as I.  With
    rows > 0 each second-order layer also gets token-row buffers A (rows x d_in)
    and Gout (rows x d_out), from which the library forms a and g.
    factor_dtype "bf16" stores Linv and Rinv in bf16 (half-precision factors).
    rank > 1 gives a and g the shapes (rank, d_in) and (rank, d_out): r vectors
    per factor (rank-r update).  optimizer "sgd" or "lamb" adds the weights W
    (zeros) and the optimizer state (opt_m, and opt_v for LAMB).  gemm_path
    ("auto", "fp32", "split") is set on the second-order layers when given.
    With guards (a Guarded), every tensor is carved out of a guarded buffer."""
    def new(shape, dtype):
        if guards is None:
            return torch.zeros(shape, dtype=dtype, device=device)
        t = guards.empty(shape, dtype, device)
        t.zero_()
        return t

    def eye(d, dtype):
        t = new((d, d), dtype)
        t.copy_(torch.eye(d, dtype=dtype, device=device))
        return t

    fdt = torch.bfloat16 if factor_dtype == "bf16" else torch.float32
    gdt = torch.bfloat16 if grad_dtype == "bf16" else torch.float32
    layers = []
    for i, (d_in, d_out) in enumerate(shapes):
        so = True if second_order is None else bool(second_order[i])
        L = dict(d_in=d_in, d_out=d_out, second_order=so,
                 G=new((d_in, d_out), gdt), dW=new((d_in, d_out), torch.float32))
        if so:
            L["Linv"] = eye(d_in, fdt)
            L["Rinv"] = eye(d_out, fdt)
            va = (rank, d_in) if rank > 1 else (d_in,)
            vg = (rank, d_out) if rank > 1 else (d_out,)
            L["a"] = new(va, torch.float32)
            L["g"] = new(vg, torch.float32)
        if so and gemm_path is not None:
            L["gemm_path"] = gemm_path
        if stats:
            L["stats"] = new((STATS_BYTES,), torch.uint8)
        if optimizer is not None:
            for k in ("W", "opt_m") + (("opt_v",) if optimizer == "lamb" else ()):
                L[k] = new((d_in, d_out), torch.float32)
        if so and rows:
            adt = torch.bfloat16 if act_dtype == "bf16" else torch.float32
            L["A"] = new((rows, d_in), adt)
            L["Gout"] = new((rows, d_out), adt)
        layers.append(L)
    return layers


def _put(dst: torch.Tensor, src: np.ndarray):
    t = torch.from_numpy(np.ascontiguousarray(src))
    dst.copy_(t.to(dst.dtype) if dst.dtype != t.dtype else t, non_blocking=False)


def set_inputs(L, a=None, g=None, G=None):
    """Copies host arrays into the layer's a, g and G (G given as float32; for
    a bf16 layer the values must already be bf16-representable)."""
    if a is not None:
        _put(L["a"], a)
    if g is not None:
        _put(L["g"], g)
    if G is not None:
        _put(L["G"], G)


def set_rows(L, A, Gout):
    """Copies host token rows into the layer's A and Gout (given as float32; for
    bf16 buffers the values must already be bf16-representable)."""
    _put(L["A"], A)
    _put(L["Gout"], Gout)


def get_means(L):
    return L["a"].cpu().numpy(), L["g"].cpu().numpy()


def set_factors(L, Linv, Rinv):
    """Copies host factors in (bf16 factors: the values must already be
    bf16-representable)."""
    _put(L["Linv"], np.asarray(Linv, dtype=np.float32))
    _put(L["Rinv"], np.asarray(Rinv, dtype=np.float32))


def get_factors(L):
    """The stored factors as float32 host arrays (bf16 values widened)."""
    return L["Linv"].float().cpu().numpy(), L["Rinv"].float().cpu().numpy()


def get_dW(L):
    return L["dW"].cpu().numpy()


def get_stats(L):
    return read_stats(L["stats"])


def make_plan(layers, workspace=None) -> MkorPlan:
    return MkorPlan(layers, workspace=workspace)
