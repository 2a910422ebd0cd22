"""Pins of the half-precision (bf16 factor) oracle against values fixed by the
mathematics and by an independent library routine (torch's float32 -> bf16
cast), plus Lemma 2's error bound."""
import math

import numpy as np
import pytest
import torch

import oracle as O
from oracle.half import BF16_MAX, layer_step_half, lemma2_bound, precondition_half, round_bf16


def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x32)).to(torch.bfloat16).to(torch.float64).numpy()


def test_round_matches_library_cast():
    rng = np.random.default_rng(3)
    x = np.concatenate([
        rng.standard_normal(200000) * 10.0 ** rng.uniform(-38, 38, 200000),
        rng.standard_normal(5000) * 1e-39,                      # bf16 subnormals
        rng.uniform(3.38e38, 3.4028e38, 200),                   # around the overflow threshold
    ]).astype(np.float32)
    assert np.array_equal(round_bf16(x.astype(np.float64)), _torch_bf16(x))


@pytest.mark.parametrize("x,want", [
    (1.0 + 2.0 ** -8, 1.0),                      # tie -> even significand
    (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),      # tie -> even (upwards)
    (1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -7),
    (-(1.0 + 2.0 ** -8), -1.0),
    (2.0 ** -133 * 1.5, 2.0 ** -132),            # subnormal tie
    (2.0 ** -133 * 2.5, 2.0 ** -132),
    (BF16_MAX, BF16_MAX),
    ((2.0 - 2.0 ** -8) * 2.0 ** 127, math.inf),  # midpoint to 2^128 rounds up, overflows
    (0.0, 0.0),
])
def test_round_hand_values(x, want):
    assert round_bf16(np.array([x]))[0] == want


def test_round_properties():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(10000) * 10.0 ** rng.uniform(-30, 30, 10000)
    r = round_bf16(x)
    assert np.array_equal(round_bf16(r), r)                     # idempotent
    assert np.all(np.abs(r - x) <= 2.0 ** -8 * np.abs(x))       # half an ulp, ulp <= 2^-7 |x|
    assert np.isnan(round_bf16(np.array([np.nan]))[0])


def test_exact_case_equals_fp64_step():
    # gamma = 1/2, P = I, a = e_0: u = e_0, s = 1, k = 1/2, so the update is
    # diag(1, 2, ..., 2) and every value on the way is a bf16 value.
    d_in, d_out = 6, 4
    p = O.Params(gamma=0.5, eps=math.inf, rescale=False)
    a = np.zeros(d_in); a[0] = 1.0
    g = np.zeros(d_out); g[2] = 1.0
    G = np.arange(d_in * d_out, dtype=np.float64).reshape(d_in, d_out) - 7.0
    PL, PR, dW, _ = layer_step_half(np.eye(d_in), np.eye(d_out), a, g, G, p)
    Lf, Rf, dWf, _ = O.layer_step(np.eye(d_in), np.eye(d_out), a, g, G, p)
    assert np.array_equal(PL, Lf) and np.array_equal(PR, Rf) and np.array_equal(dW, dWf)
    assert np.array_equal(np.diag(PL), [1, 2, 2, 2, 2, 2])


def test_intermediate_is_rounded():
    # 1x1: Y = bf16((1 + 2^-7)^2) = bf16(1 + 2^-6 + 2^-14) = 1 + 2^-6
    v = 1.0 + 2.0 ** -7
    dW_hat, Y = precondition_half(np.array([[1.0]]), np.array([[v]]), np.array([[v]]))
    assert Y[0, 0] == 1.0 + 2.0 ** -6
    assert dW_hat[0, 0] == 1.0 + 2.0 ** -6


def test_gradient_enters_rounded():
    p = O.Params(gamma=0.5, eps=math.inf, rescale=False)
    G = np.array([[1.0 + 2.0 ** -9]])            # rounds to 1
    _, _, dW, st = layer_step_half(np.eye(1), np.eye(1), np.zeros(1), np.zeros(1), G, p, update=False)
    assert dW[0, 0] == 1.0 and st.norm_G == 1.0


def test_stored_state_and_update_from_it():
    # Scalar factor: the exact update of P = 1 with x = 1/2, gamma = 3/4 is the
    # inverse of M = 3/4 + (1/4)(1/4), i.e. 16/13; its bf16 value is 158/128.
    # The next update starts from the stored 158/128: 1 / (3/4 * 128/158 + 1/16).
    p = O.Params(gamma=0.75, eps=math.inf, rescale=False)
    x = np.array([0.5])
    PL, PR, _, _ = layer_step_half(np.eye(1), np.eye(1), x, x, np.ones((1, 1)), p, precond=False)
    assert PL[0, 0] == pytest.approx(16.0 / 13.0, rel=1e-15)
    assert round_bf16(PL)[0, 0] == 158.0 / 128.0
    PL2, _, _, _ = layer_step_half(PL, PR, x, x, np.ones((1, 1)), p, precond=False)
    assert PL2[0, 0] == pytest.approx(1.0 / (0.75 * 128.0 / 158.0 + 1.0 / 16.0), rel=1e-15)


def test_preconditioning_uses_fresh_factor():
    # After one update PL = 16/13 (x = 1/2, gamma = 3/4) and PR = 4/3 (g = 0:
    # M = 3/4).  dW_hat = PL * bf16(1 * PR) = 16/13 * 171/128, with the
    # updated PL before its rounding to storage.
    p = O.Params(gamma=0.75, eps=math.inf, rescale=False)
    _, _, dW, _ = layer_step_half(np.eye(1), np.eye(1), np.array([0.5]), np.zeros(1), np.ones((1, 1)), p)
    assert dW[0, 0] == pytest.approx(16.0 / 13.0 * 171.0 / 128.0, rel=1e-15)


def _trajectory_factor(seed, d, steps=5, gamma=0.9):
    rng = np.random.default_rng(seed)
    P = np.eye(d)
    p = O.Params(gamma=gamma, eps=math.inf)
    for _ in range(steps):
        P, _ = O.update_factor(P, rng.standard_normal(d) / math.sqrt(d), p)
    return P


@pytest.mark.parametrize("d", [16, 64, 200])
def test_lemma2_bound(d):
    # One update from the bf16-quantised factor against the same update at
    # full precision: the difference stays within Lemma 2's bound, with the
    # measured quantisation error as eps and the largest entry as m.
    gamma = 0.9
    P = _trajectory_factor(d, d, gamma=gamma)
    x = np.random.default_rng(d + 1).standard_normal(d) / math.sqrt(d)
    p = O.Params(gamma=gamma, eps=math.inf)
    Q = round_bf16(P)
    eps = float(np.max(np.abs(Q - P)))
    m = float(max(np.max(np.abs(P)), np.max(np.abs(x))))
    P_half, _ = O.update_factor(Q, x, p)
    P_full, _ = O.update_factor(P, x, p)
    err = float(np.max(np.abs(round_bf16(P_half) - P_full)))
    assert eps > 0.0
    assert err <= lemma2_bound(gamma, m, d, eps) + float(np.max(np.abs(P_full))) * 2.0 ** -8


def test_half_step_close_to_full_precision():
    # The half-precision step differs from the float64 step by the bf16
    # quantisation only: relative errors of a few 2^-9.
    rng = np.random.default_rng(9)
    d_in, d_out = 48, 80
    Li, Ri = _trajectory_factor(1, d_in), _trajectory_factor(2, d_out)
    QL, QR = round_bf16(Li), round_bf16(Ri)
    a = rng.standard_normal(d_in) / math.sqrt(d_in)
    g = rng.standard_normal(d_out) / math.sqrt(d_out)
    G = rng.standard_normal((d_in, d_out)) * 1e-3
    p = O.Params()
    PL, PR, dW, _ = layer_step_half(QL, QR, a, g, G, p)
    Lf, Rf, dWf, _ = O.layer_step(QL, QR, a, g, G, p)
    assert np.array_equal(PL, Lf) and np.array_equal(PR, Rf)   # same update from the same stored factor
    e = np.linalg.norm(dW - dWf) / np.linalg.norm(dWf)
    assert 1e-5 < e < 8 * 2.0 ** -9
