"""Float64 CPU oracle of MKOR with half-precision (bf16) inverse factors.

TEST INFRASTRUCTURE ONLY (like the rest of this package): used by the tests,
never by the product path; shares no code with the HIP library.

The paper runs MKOR in half precision (Table 1 and its caption halve the
memory and communication for it; Section "Numerical Stability" argues that
the method needs only products, and its Lemma 2 bounds the quantisation
error of one factor update).  It does not say which quantities are rounded.
Reading taken here (listed with the other readings in the design notes):

* the stored state of each inverse factor is bf16 (8-bit significand, round
  to nearest, ties to even); the momentum rank-1 update (stabiliser, u = P x,
  Sherman-Morrison) is evaluated at full precision from the stored bf16
  value, and its result is rounded to bf16 when it is stored;
* the preconditioning takes the gradient rounded to bf16 (a no-op for a
  bf16 gradient), forms Y = G R^-1 with full-precision accumulation and
  rounds Y to bf16, then dW_hat = L^-1 Y with full-precision accumulation;
  the factors it uses are the freshly updated ones, before their rounding
  to storage;
* the rescale uses the norm of the bf16-rounded gradient.

So the state carried from step to step is the full-precision updated factor
P_t, whose stored value is bf16(P_t); the next update starts from bf16(P_t).
"""

from __future__ import annotations

import math

import numpy as np

from .mkor_oracle import (LayerStats, NONFINITE_L, NONFINITE_R, NONFINITE_SCALE, Params,
                          rescale, update_factor)

BF16_MANT = 8                    # significand bits, the implicit one included
BF16_EMIN = -126                 # exponent of the smallest normal, 2^-126
BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bf16 value, ties to even.

    bf16 keeps the float32 exponent range with an 8-bit significand: normal
    numbers are multiples of 2^(e - 7) for 2^e <= |x| < 2^(e + 1), e >= -126;
    below 2^-126 the spacing stays 2^-133 (subnormals).  A value at or beyond
    the midpoint between the largest finite bf16 and 2^128 becomes +-inf;
    NaN stays NaN.  Returned as float64 (every bf16 value is exact there).
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    fin = np.isfinite(x)
    out[~fin] = x[~fin]
    v = x[fin]
    a = np.abs(v)
    # exponent e with 2^e <= |v| < 2^(e+1); frexp gives |v| = m 2^k, m in [0.5, 1)
    _m, k = np.frexp(a)
    e = np.maximum(k - 1, BF16_EMIN)
    q = np.ldexp(1.0, e - (BF16_MANT - 1))          # spacing at that exponent
    r = np.rint(v / q) * q                          # rint: ties to even multiple
    big = np.abs(r) >= 2.0 ** 128
    r[big] = np.copysign(np.inf, r[big])
    out[fin] = r
    return out


def precondition_half(PL: np.ndarray, G_h: np.ndarray, PR: np.ndarray):
    """dW_hat = PL . bf16(G_h . PR) (Eq. 2 for the stored orientation, in the
    half-precision reading).  Returns (dW_hat, Y_h)."""
    Y = np.asarray(G_h, np.float64) @ np.asarray(PR, np.float64)
    Y_h = round_bf16(Y)
    return np.asarray(PL, np.float64) @ Y_h, Y_h


def layer_step_half(PL, PR, a, g, G, p: Params, stab_override=(None, None),
                    update: bool = True, precond: bool = True):
    """One MKOR step of one second-order layer with bf16 factors.

    ``PL``, ``PR`` are the current full-precision factors (for a fresh start,
    bf16 values: the caller's stored buffers).  Returns (PL', PR', dW, stats);
    the stored factors after the step are round_bf16(PL'), round_bf16(PR').
    """
    st = LayerStats()
    PL = np.asarray(PL, dtype=np.float64)
    PR = np.asarray(PR, dtype=np.float64)
    if update:
        QL, QR = round_bf16(PL), round_bf16(PR)
        PL, st.L = update_factor(QL, a, p, stab_override[0])
        PR, st.R = update_factor(QR, g, p, stab_override[1])
        if st.L.skipped:
            st.nonfinite |= NONFINITE_L
        if st.R.skipped:
            st.nonfinite |= NONFINITE_R
    dW = None
    if precond:
        G_h = round_bf16(G)
        with np.errstate(all="ignore"):
            dW_hat, _ = precondition_half(PL, G_h, PR)
            if p.rescale:
                dW, st.norm_G, st.norm_dW_hat, st.scale = rescale(G_h, dW_hat)
            else:
                dW = dW_hat
                st.norm_G = float(np.linalg.norm(G_h))
                st.norm_dW_hat = float(np.linalg.norm(dW_hat))
                st.scale = 1.0
        if not (math.isfinite(st.norm_G) and math.isfinite(st.norm_dW_hat)):
            st.nonfinite |= NONFINITE_SCALE
    return PL, PR, dW, st


def lemma2_bound(gamma: float, m: float, d: int, eps: float) -> float:
    """Lemma 2's order bound on the quantisation error of one factor update,
    (gamma + 4 (1 - gamma) / gamma^2 m^3 d^2) eps, with unit constant."""
    return (gamma + 4.0 * (1.0 - gamma) / (gamma * gamma) * m ** 3 * d * d) * eps
