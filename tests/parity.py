"""Shared helpers of the GPU parity tests: seeded states, error metrics, and a
free-running driver that steps the HIP path over a whole grouped layer list
while the float64 oracle follows a sample of its layers."""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle as O
import workloads as W
from oracle.half import layer_step_half, round_bf16
from oracle.optimizer import lamb_step
from paper_2306_01685_amd import Params, harness as H

TOL_STEP = 1e-4   # relative Frobenius error after one step from the same state
TOL_FREE = 1e-3   # after up to 50 independently accumulated steps
# bf16 factors (bars derived in tests/test_half_gpu.py): dW after one step
# from the same stored factors, and factors and dW after up to 50 steps
TOL_HALF_STEP = 2e-4
TOL_HALF_FREE = 2e-2
NEAR_TIE = 1e-4   # |nu - eps| / eps band in which either stabiliser decision is accepted


def rel(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = float(np.linalg.norm(b))
    if nb == 0.0:
        return float(np.linalg.norm(a))
    return float(np.linalg.norm(a - b)) / nb


def relmax(a, b) -> float:
    """Largest element-wise error relative to the largest reference element:
    catches an error confined to a few elements (a tile edge, one row), which
    the Frobenius norm of a large matrix averages away."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    mb = float(np.abs(b).max()) if b.size else 0.0
    d = float(np.abs(a - b).max()) if b.size else 0.0
    return d if mb == 0.0 else d / mb


def check_close(got, ref, tol, *ctx) -> float:
    """Asserts both the relative Frobenius error and the element-wise one
    (relmax) are within tol; returns the Frobenius error."""
    e, m = rel(got, ref), relmax(got, ref)
    assert e <= tol, (*ctx, "Frobenius", e)
    assert m <= tol, (*ctx, "element-wise", m)
    return e


def spd(seed, d, spread=0.25):
    """Seeded symmetric positive-definite fp32 matrix, bitwise symmetric."""
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((d, max(1, d // 2)))
    P = np.eye(d) + spread * (Q @ Q.T) / d
    P = 0.5 * (P + P.T)
    return P.astype(np.float32)


def oparams(p: Params) -> O.Params:
    return O.Params(gamma=p.gamma, zeta=p.zeta, eps=p.eps, norm_kind=p.norm_kind,
                    variant=p.variant, rescale=p.rescale, guard_nonfinite=p.guard_nonfinite)


def near_tie(nu, eps) -> bool:
    return math.isfinite(eps) and eps > 0 and abs(nu - eps) / eps < NEAR_TIE


def oracle_factor_step(P, x, p: O.Params, gpu_flag):
    """One oracle factor update, adopting the GPU's stabiliser decision only in
    the near-tie band."""
    nu = O.factor_norm(P, p.norm_kind)
    ov = bool(gpu_flag) if near_tie(nu, p.eps) else None
    return O.update_factor(P, x, p, ov)


class FreeRun:
    """Steps all layers of a workload on the GPU; the oracle follows `sample`.

    Inputs of sampled layers come from the workload generator; the other
    layers get seeded values drawn on the GPU (their values never reach a
    checked output, layers being independent).  half: bf16 factors, followed
    by the half-precision oracle (its state is the unrounded factor; the
    stored one is its bf16 rounding).  optimizer "lamb": every layer carries
    weights and moments for the fused LAMB step.
    """

    def __init__(self, w: W.Workload, params: Params, sample, explicit=False, bulk_seed=1234, gemm_path=None,
                 half=False, optimizer=None):
        self.w, self.p, self.op = w, params, oparams(params)
        self.sample = list(sample)
        self.explicit = explicit
        self.half = half
        self.layers = H.allocate_layers(w.shapes, w.grad_dtype, gemm_path=None if half else gemm_path,
                                        factor_dtype="bf16" if half else "fp32", optimizer=optimizer)
        self.opt_state = {}
        if optimizer is not None:
            for i in self.sample:
                d_in, d_out = w.shapes[i]
                W0 = (np.random.default_rng(777 + i).standard_normal((d_in, d_out)) * 0.02).astype(np.float32)
                self.layers[i]["W"].copy_(torch.from_numpy(W0))
                self.opt_state[i] = [W0.astype(np.float64), np.zeros((d_in, d_out)), np.zeros((d_in, d_out))]
        self.gen = torch.Generator(device="cuda")
        self.gen.manual_seed(bulk_seed)
        self.state = {}
        for i in range(w.n_layers):
            if w.init != "identity" or i in self.sample:
                L0, R0 = W.initial_factors(w, i)
                if w.init != "identity":
                    H.set_factors(self.layers[i], L0, R0)
                if i in self.sample:
                    self.state[i] = [L0.astype(np.float64), R0.astype(np.float64)]
        self.plan = H.make_plan(self.layers)
        self.t = 0
        self.flags = {i: [] for i in self.sample}

    def _inputs(self, t):
        host = {}
        for i, L in enumerate(self.layers):
            if i in self.sample:
                a, g = W.rank1_vectors(self.w, i, t, explicit=self.explicit)
                G = W.gradient(self.w, i, t)
                H.set_inputs(L, a, g, G)
                host[i] = (a, g, G)
            else:
                d_in, d_out = L["d_in"], L["d_out"]
                s_a = math.sqrt((2.0 if self.w.act_dist == "student_t4" else 1.0) / self.w.rows)
                L["a"].normal_(0.0, s_a, generator=self.gen)
                L["g"].normal_(0.0, self.w.grad_row_std / math.sqrt(self.w.rows), generator=self.gen)
                if L["G"].dtype == torch.bfloat16:
                    tmp = torch.empty((d_in, d_out), dtype=torch.float32, device="cuda")
                    tmp.normal_(0.0, self.w.G_std, generator=self.gen)
                    L["G"].copy_(tmp)
                    del tmp
                else:
                    L["G"].normal_(0.0, self.w.G_std, generator=self.gen)
        return host

    def step(self, precond_oracle=False, update=True, opt=None):
        """One step on both sides (update=False: the precondition-only call of
        an update-every-f schedule; opt: an OptParams for the fused optimizer
        step, followed by the oracle for the sampled layers' weights and
        moments); returns the oracle's dW per sampled layer when precond_oracle
        is set (else None)."""
        host = self._inputs(self.t)
        if opt is not None:
            (self.plan.step_opt if update else self.plan.precondition_opt)(self.p, opt)
        else:
            (self.plan.step if update else self.plan.precondition)(self.p)
        torch.cuda.synchronize()
        out = {}
        for i in self.sample:
            st = H.get_stats(self.layers[i])
            a, g, G = host[i]
            Lp, Rp = self.state[i]
            if update and self.half:
                # the half oracle updates from the stored (rounded) factor; it
                # adopts the GPU's stabiliser decision only in the near-tie band
                pre = precond_oracle or opt is not None
                Ln, Rn, dWh, ost = layer_step_half(Lp, Rp, a, g, G, self.op, precond=pre)
                ov = tuple(bool(st[f"stab_{s}"]) if (near_tie(fs.nu, self.op.eps) and fs.stab != bool(st[f"stab_{s}"]))
                           else None for s, fs in (("L", ost.L), ("R", ost.R)))
                if ov != (None, None):
                    Ln, Rn, dWh, ost = layer_step_half(Lp, Rp, a, g, G, self.op, ov, precond=pre)
                self.flags[i].append(((ost.L.stab, st["stab_L"], ost.L.nu), (ost.R.stab, st["stab_R"], ost.R.nu)))
            elif update:
                Ln, sL = oracle_factor_step(Lp, a, self.op, st["stab_L"])
                Rn, sR = oracle_factor_step(Rp, g, self.op, st["stab_R"])
                self.flags[i].append(((sL.stab, st["stab_L"], sL.nu), (sR.stab, st["stab_R"], sR.nu)))
            else:
                Ln, Rn = Lp, Rp
            self.state[i] = [Ln, Rn]
            if precond_oracle or opt is not None:
                if self.half:
                    if not update:
                        _, _, dWh, ost = layer_step_half(Ln, Rn, a, g, G, self.op, update=False)
                    dW = dWh
                else:
                    _, _, dW, ost = O.layer_step(Ln, Rn, a, g, G, self.op, update=False)
                out[i] = (dW, ost)
                if opt is not None and i in self.opt_state:
                    Wo, mo, vo = self.opt_state[i]
                    F = lambda x: float(np.float32(x))  # noqa: E731  (the ABI takes fp32 hyper-parameters)
                    self.opt_state[i][:] = list(lamb_step(Wo, mo, vo, dW, opt.step, F(opt.lr), F(opt.beta1),
                                                          F(opt.beta2), F(opt.eps), F(opt.weight_decay)))[:3]
        self.t += 1
        return out if precond_oracle else None

    def check_optimizer(self, tol):
        """Weights and moments of the sampled layers against the oracle's."""
        worst = 0.0
        for i, (Wo, mo, vo) in self.opt_state.items():
            L = self.layers[i]
            for name, x, y in (("W", L["W"], Wo), ("m", L["opt_m"], mo), ("v", L["opt_v"], vo)):
                e = rel(x.cpu().numpy(), y)
                worst = max(worst, e)
                assert e <= tol, (self.w.name, i, self.t, name, e)
        return worst

    def check_factors(self, tol):
        """Writes the current factors into their buffers (the plan keeps the
        last update pending) and compares them with the oracle's (bf16
        factors: with the bf16 rounding of the oracle's)."""
        self.plan.sync_factors()
        torch.cuda.synchronize()
        worst = 0.0
        for i in self.sample:
            Lg, Rg = H.get_factors(self.layers[i])
            Lo, Ro = self.state[i]
            if self.half:
                Lo, Ro = round_bf16(Lo), round_bf16(Ro)
            eL, eR = rel(Lg, Lo), rel(Rg, Ro)
            worst = max(worst, eL, eR)
            assert eL <= tol and eR <= tol, (self.w.name, i, self.t, eL, eR)
            if not self.half:   # bf16: a rounding flip is one ulp (2^-8) of an element
                mL, mR = relmax(Lg, Lo), relmax(Rg, Ro)
                assert mL <= tol and mR <= tol, (self.w.name, i, self.t, "element-wise", mL, mR)
        return worst

    def check_dW(self, oracle_out, tol):
        worst = 0.0
        for i, (dW, ost) in oracle_out.items():
            got = H.get_dW(self.layers[i])
            e = rel(got, dW)
            worst = max(worst, e)
            assert e <= tol, (self.w.name, i, self.t, e)
            if not self.half:
                m = relmax(got, dW)
                assert m <= tol, (self.w.name, i, self.t, "element-wise", m)
        return worst

    def check_flags(self):
        """Stabiliser decisions agree everywhere outside the near-tie band."""
        fired = 0
        for i, seq in self.flags.items():
            for t, pair in enumerate(seq):
                for (o, gflag, nu) in pair:
                    fired += int(o)
                    if not near_tie(nu, self.op.eps):
                        assert bool(o) == bool(gflag), (self.w.name, i, t, o, gflag, nu)
        return fired
