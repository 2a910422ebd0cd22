"""Float64 CPU oracle for MKOR's per-step hot path (arXiv 2306.01685).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the smoke check of ``__graft_entry__`` and
the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no helpers, no constants, no kernels) and never imports it.

What it computes, per layer, in the paper's order (Algorithm 1, the
second-order branch, with the rank-1 means handed in as inputs):

1. norm-based stabilisation of each inverse factor (Algorithm 1, the two
   stabilisation lines; "Norm-Based Stabilizer" paragraph and Section
   "Exploding Gradients Problem", which names the infinity norm);
2. the momentum rank-1 Sherman-Morrison update of each inverse factor
   (Algorithm 1, SM-based factor inversion; Eq. 4-7);
3. preconditioning  dW_hat = Linv . G . Rinv  with the updated factors
   (Algorithm 1, precondition line; Eq. 2);
4. rescaling to the original gradient norm (Algorithm 1, rescale line;
   "Rescaling Gradients" paragraph);
5. first-order layers pass the gradient through (Algorithm 1, else-branch).

Orientation used here (the paper writes the transpose): the stored gradient G
is d_in x d_out, Linv is d_in x d_in and is driven by the mean activation a,
Rinv is d_out x d_out and is driven by the mean output-gradient g.  Because
both factors are symmetric, (L^-1 dW R^-1)^T = R^-1 dW^T L^-1, so this is the
paper's update of Eq. 2 written for the transposed gradient.

Readings of passages the paper leaves open (each is listed with its reason in
the design notes of the repository):

* SM variant.  Eq. 6/7 as printed is not the inverse of the momentum
  accumulation of Eq. 4/5 (first term, sign and denominator differ).  The
  default ``EXACT`` variant is the Sherman-Morrison inverse of
  M_t = gamma * M_hat_{t-1} + (1 - gamma) x x^T, i.e.
  P_t = (1/gamma) (P_hat - k u u^T),  u = P_hat x,  s = x^T u,
  k = (1 - gamma) / (gamma + (1 - gamma) s).
  ``PAPER_EQ6`` evaluates the printed Eq. 6/7 literally:
  P_t = gamma P_hat + (1 - gamma) / (gamma^2 (1 + gamma (1 - gamma) s)) u u^T.
* Stabiliser acts on the inverse factor (Algorithm 1 and Eq. 11), strictly
  when the norm exceeds eps; the norm is the induced infinity norm (max
  absolute row sum), or max |entry| with ``norm_kind=1``.
* Rescale uses Frobenius norms; a zero preconditioned gradient gives dW = 0.
* Non-finite guard (the paper is silent): with ``guard_nonfinite`` a factor
  whose norm, s or update coefficient is not finite is left unchanged and
  flagged.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

EXACT = 0
PAPER_EQ6 = 1

NORM_INF = 0      # induced infinity norm: max_i sum_j |P_ij|
NORM_MAXABS = 1   # max_ij |P_ij|

NONFINITE_L = 1   # Linv update skipped (guard) or non-finite (no guard)
NONFINITE_R = 2   # Rinv update skipped (guard) or non-finite (no guard)
NONFINITE_SCALE = 4  # non-finite norm in the rescale


@dataclass
class Params:
    """Optimizer hyper-parameters of one step (Algorithm 1)."""
    gamma: float = 0.9          # momentum of the factor accumulation (Eq. 4/5)
    zeta: float = 0.5           # blend weight of the stabiliser (Eq. 9/10)
    eps: float = 100.0          # stabiliser threshold; math.inf disables it
    norm_kind: int = NORM_INF
    variant: int = EXACT
    rescale: bool = True
    guard_nonfinite: bool = True


@dataclass
class FactorStats:
    nu: float = 0.0         # norm of the factor before this step's update
    stab: bool = False      # stabiliser fired
    s: float = 0.0          # x^T P_hat x
    skipped: bool = False   # guard left the factor unchanged


@dataclass
class LayerStats:
    L: FactorStats = field(default_factory=FactorStats)
    R: FactorStats = field(default_factory=FactorStats)
    norm_G: float = 0.0
    norm_dW_hat: float = 0.0
    scale: float = 0.0
    nonfinite: int = 0


def rank1_means(rows: np.ndarray) -> np.ndarray:
    """Rank-1 approximation vector of Algorithm 1 (its first two lines and the
    "Rank-1 Approximation" paragraph): the average of the samples.

    ``rows`` holds one sample per row (b x d, the transpose of the paper's
    d x b matrix whose columns are the samples); returns the length-d float64
    mean (1/b) * sum_i rows[i, :].  Summed in float64 in row order.
    """
    R = np.asarray(rows, dtype=np.float64)
    if R.ndim != 2 or R.shape[0] == 0:
        raise ValueError("rows must be a non-empty b x d array")
    acc = np.zeros(R.shape[1], dtype=np.float64)
    for i in range(R.shape[0]):
        acc += R[i]
    return acc / R.shape[0]


def factor_norm(P: np.ndarray, norm_kind: int = NORM_INF) -> float:
    """Norm watched by the stabiliser: the infinity norm of the factor.

    The textbook induced infinity norm is the largest absolute row sum.
    """
    A = np.abs(np.asarray(P, dtype=np.float64))
    if A.size == 0:
        return 0.0
    if norm_kind == NORM_INF:
        return float(A.sum(axis=1).max())
    if norm_kind == NORM_MAXABS:
        return float(A.max())
    raise ValueError(f"unknown norm_kind {norm_kind}")


def stabilize(P: np.ndarray, nu: float, eps: float, zeta: float):
    """Norm-based stabiliser of Algorithm 1: blend the inverse factor toward I.

    Returns (P_hat, fired).  Fires strictly when nu > eps.
    """
    if nu > eps:
        d = P.shape[0]
        return zeta * P + (1.0 - zeta) * np.eye(d), True
    return P, False


def sm_update(P_hat: np.ndarray, x: np.ndarray, gamma: float, variant: int = EXACT):
    """Momentum rank-1 Sherman-Morrison update of one inverse factor.

    Returns (P_new, u, s, coefficient k) with u = P_hat x and s = x^T u.
    """
    u = P_hat @ x
    s = float(x @ u)
    if variant == EXACT:
        k = (1.0 - gamma) / (gamma + (1.0 - gamma) * s)
        P_new = (P_hat - k * np.outer(u, u)) / gamma
    elif variant == PAPER_EQ6:
        k = (1.0 - gamma) / (gamma * gamma * (1.0 + gamma * (1.0 - gamma) * s))
        P_new = gamma * P_hat + k * np.outer(u, u)
    else:
        raise ValueError(f"unknown variant {variant}")
    return P_new, u, s, k


def update_factor(P: np.ndarray, x: np.ndarray, p: Params, stab_override=None):
    """Stabilise then SM-update one factor (Algorithm 1, stabiliser + SM lines).

    ``stab_override`` (None, True or False) replaces the threshold decision;
    parity tests use it only when the oracle's norm sits within a relative
    1e-4 of eps, where fp32 and fp64 may legitimately decide differently.
    """
    P = np.asarray(P, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    st = FactorStats()
    st.nu = factor_norm(P, p.norm_kind)
    if stab_override is None:
        P_hat, st.stab = stabilize(P, st.nu, p.eps, p.zeta)
    else:
        st.stab = bool(stab_override)
        P_hat = p.zeta * P + (1.0 - p.zeta) * np.eye(P.shape[0]) if st.stab else P
    with np.errstate(all="ignore"):
        P_new, _u, st.s, k = sm_update(P_hat, x, p.gamma, p.variant)
    bad = not (math.isfinite(st.nu) and math.isfinite(st.s) and math.isfinite(k))
    if bad and p.guard_nonfinite:
        st.skipped = True
        return P.copy(), st
    st.skipped = bad
    return P_new, st


def precondition(Linv: np.ndarray, G: np.ndarray, Rinv: np.ndarray) -> np.ndarray:
    """dW_hat = Linv . G . Rinv (Eq. 2 for the stored orientation)."""
    X = np.asarray(Linv, np.float64) @ np.asarray(G, np.float64)
    return X @ np.asarray(Rinv, np.float64)


def rescale(G: np.ndarray, dW_hat: np.ndarray):
    """Scale dW_hat so that its Frobenius norm equals that of G.

    Returns (dW, norm_G, norm_dW_hat, scale); scale = 0 when dW_hat is zero.
    """
    nG = float(np.linalg.norm(np.asarray(G, np.float64)))
    nD = float(np.linalg.norm(dW_hat))
    scale = nG / nD if nD > 0.0 else 0.0
    return scale * dW_hat, nG, nD, scale


def layer_step(Linv, Rinv, a, g, G, p: Params, second_order: bool = True,
               stab_override=(None, None), update: bool = True, precond: bool = True):
    """One MKOR step for one layer.  Returns (Linv', Rinv', dW, LayerStats).

    ``update`` runs the factor half (stabiliser + SM), ``precond`` the
    precondition + rescale half; both together are one full step.
    """
    st = LayerStats()
    G64 = np.asarray(G, dtype=np.float64)
    Linv = np.asarray(Linv, dtype=np.float64)
    Rinv = np.asarray(Rinv, dtype=np.float64)
    if not second_order:
        return Linv.copy(), Rinv.copy(), G64.copy() if precond else None, st
    if update:
        Linv, st.L = update_factor(Linv, a, p, stab_override[0])
        Rinv, st.R = update_factor(Rinv, g, p, stab_override[1])
        if st.L.skipped:
            st.nonfinite |= NONFINITE_L
        if st.R.skipped:
            st.nonfinite |= NONFINITE_R
    dW = None
    if precond:
        with np.errstate(all="ignore"):
            dW_hat = precondition(Linv, G64, Rinv)
            if p.rescale:
                dW, st.norm_G, st.norm_dW_hat, st.scale = rescale(G64, dW_hat)
            else:
                dW = dW_hat
                st.norm_G = float(np.linalg.norm(G64))
                st.norm_dW_hat = float(np.linalg.norm(dW_hat))
                st.scale = 1.0
        if not (math.isfinite(st.norm_G) and math.isfinite(st.norm_dW_hat)):
            st.nonfinite |= NONFINITE_SCALE
    return Linv, Rinv, dW, st


def layer_step_rows(Linv, Rinv, A_rows, Gout_rows, G, p: Params, stab_override=(None, None)):
    """One MKOR step for one second-order layer from its token rows: a and g
    are the rank-1 means of the activation rows A_rows (b x d_in) and of the
    output-gradient rows Gout_rows (b x d_out), then ``layer_step``.  Returns
    (Linv', Rinv', dW, LayerStats, a, g)."""
    a = rank1_means(A_rows)
    g = rank1_means(Gout_rows)
    Li, Ri, dW, st = layer_step(Linv, Rinv, a, g, G, p, True, stab_override)
    return Li, Ri, dW, st, a, g


def oracle_step(layers, p: Params, update: bool = True, precond: bool = True,
                stab_overrides=None):
    """One step over a list of layers (Algorithm 1, "for each layer").

    ``layers`` is a list of dicts with keys Linv, Rinv, a, g, G and optional
    second_order (default True).  Returns a list of dicts with Linv, Rinv, dW
    and stats; the inputs are not modified.
    """
    out = []
    for i, L in enumerate(layers):
        ov = (None, None) if stab_overrides is None else stab_overrides[i]
        Li, Ri, dW, st = layer_step(L["Linv"], L["Rinv"], L["a"], L["g"], L["G"], p,
                                    bool(L.get("second_order", True)), ov, update, precond)
        out.append(dict(Linv=Li, Rinv=Ri, dW=dW, stats=st))
    return out
