"""Float64 CPU oracle of MKOR's rank-r extension.

TEST INFRASTRUCTURE ONLY (like the rest of this package): used by the tests,
never by the product path; shares no code with the HIP library.

The paper's section on extending MKOR to higher ranks takes a covariance
C = sum_i c_i c_i^T of rank r and applies the Sherman-Morrison identity once
per vector, each step from the previous step's inverse, O(r d^2) in all; it
leaves open where the vectors come from (an SVD would cost as much as an
inversion).  Reading taken here (listed with the others in the design
notes): the caller hands in the r vectors x_1 .. x_r of each factor, and one
step inverts the momentum accumulation of Eq. 4/5 with the rank-r sum in
place of the rank-1 term,

    M_t = gamma * M_hat_{t-1} + (1 - gamma) * sum_i x_i x_i^T,

by r sequential Sherman-Morrison updates of P^(0) = P_hat / gamma with
y_i = sqrt(1 - gamma) x_i:

    u_i = P^(i-1) y_i,   P^(i) = P^(i-1) - u_i u_i^T / (1 + y_i^T u_i).

The stabiliser acts on the factor before the update as in the rank-1 step.
For r = 1 this is the rank-1 EXACT update.  Only the EXACT variant has a
rank-r form (the printed Eq. 6/7 is not the inverse of an accumulation).
"""

from __future__ import annotations

import math

import numpy as np

from .mkor_oracle import EXACT, FactorStats, LayerStats, NONFINITE_L, NONFINITE_R, NONFINITE_SCALE
from .mkor_oracle import Params, factor_norm, rescale, precondition, stabilize


def sm_update_rank(P_hat: np.ndarray, X: np.ndarray, gamma: float) -> np.ndarray:
    """r sequential Sherman-Morrison updates (module docstring).  X is d x r."""
    X = np.asarray(X, dtype=np.float64).reshape(P_hat.shape[0], -1)
    P = np.asarray(P_hat, dtype=np.float64) / gamma
    for i in range(X.shape[1]):
        y = math.sqrt(1.0 - gamma) * X[:, i]
        u = P @ y
        P = P - np.outer(u, u) / (1.0 + float(y @ u))
    return P


def update_factor_rank(P: np.ndarray, X: np.ndarray, p: Params, stab_override=None):
    """Stabilise then rank-r update one factor.  Returns (P_new, FactorStats);
    FactorStats.s is x_1^T P_hat x_1 (the first vector's s)."""
    if p.variant != EXACT:
        raise ValueError("the rank-r update exists for the EXACT variant only")
    P = np.asarray(P, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64).reshape(P.shape[0], -1)
    st = FactorStats()
    st.nu = factor_norm(P, p.norm_kind)
    if stab_override is None:
        P_hat, st.stab = stabilize(P, st.nu, p.eps, p.zeta)
    else:
        st.stab = bool(stab_override)
        P_hat = p.zeta * P + (1.0 - p.zeta) * np.eye(P.shape[0]) if st.stab else P
    with np.errstate(all="ignore"):
        st.s = float(X[:, 0] @ P_hat @ X[:, 0])
        P_new = sm_update_rank(P_hat, X, p.gamma)
    bad = not (math.isfinite(st.nu) and np.all(np.isfinite(P_new)))
    if bad and p.guard_nonfinite:
        st.skipped = True
        return P.copy(), st
    st.skipped = bad
    return P_new, st


def layer_step_rank(Linv, Rinv, A, Gv, G, p: Params, stab_override=(None, None),
                    update: bool = True, precond: bool = True):
    """One MKOR step of one second-order layer with rank-r vectors: A is
    d_in x r (vectors driving Linv), Gv is d_out x r (driving Rinv).  Returns
    (Linv', Rinv', dW, LayerStats)."""
    st = LayerStats()
    Linv = np.asarray(Linv, dtype=np.float64)
    Rinv = np.asarray(Rinv, dtype=np.float64)
    G64 = np.asarray(G, dtype=np.float64)
    if update:
        Linv, st.L = update_factor_rank(Linv, A, p, stab_override[0])
        Rinv, st.R = update_factor_rank(Rinv, Gv, p, stab_override[1])
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
