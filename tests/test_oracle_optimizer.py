"""Pins of the backend-optimizer oracle (oracle/optimizer.py): hand-computed
steps and torch's own SGD and AdamW (library routines, CPU, float64)."""
import math

import numpy as np
import pytest
import torch

from oracle.optimizer import lamb_step, sgd_step


def test_sgd_hand_values():
    # W = 1, dW = 0.5, wd = 0.1, mu = 0.9, lr = 0.1:
    # d = 0.6, m = 0.6, W = 0.94; then d = 0.594, m = 0.54 + 0.594 = 1.134, W = 0.8266
    W, m = sgd_step(np.array([1.0]), np.zeros(1), np.array([0.5]), 0.1, 0.9, 0.1)
    assert W[0] == pytest.approx(0.94, abs=1e-15) and m[0] == pytest.approx(0.6, abs=1e-15)
    W, m = sgd_step(W, m, np.array([0.5]), 0.1, 0.9, 0.1)
    assert m[0] == pytest.approx(1.134, abs=1e-14) and W[0] == pytest.approx(0.8266, abs=1e-14)


def test_sgd_matches_torch():
    rng = np.random.default_rng(1)
    W0 = rng.standard_normal((7, 5))
    p = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=0.05, momentum=0.9, weight_decay=0.01)
    W, m = W0.copy(), np.zeros_like(W0)
    for k in range(5):
        g = rng.standard_normal((7, 5))
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        W, m = sgd_step(W, m, g, 0.05, 0.9, 0.01)
        assert np.allclose(W, p.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_lamb_without_trust_is_adamw():
    rng = np.random.default_rng(2)
    W0 = rng.standard_normal((6, 4))
    p = torch.nn.Parameter(torch.tensor(W0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=1e-2, betas=(0.9, 0.999), eps=1e-6, weight_decay=0.01)
    W, m, v = W0.copy(), np.zeros_like(W0), np.zeros_like(W0)
    for t in range(1, 6):
        g = rng.standard_normal((6, 4))
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        W, m, v, phi = lamb_step(W, m, v, g, t, 1e-2, 0.9, 0.999, 1e-6, 0.01, trust=False)
        assert phi == 1.0
        assert np.allclose(W, p.detach().numpy(), rtol=1e-12, atol=1e-14)


def test_lamb_first_step_trust_ratio():
    # t = 1, wd = 0, eps -> 0: m_hat = g, v_hat = g^2, r = sign(g), ||r|| = sqrt(n),
    # so W' = W - lr ||W|| / sqrt(n) sign(g)
    W = np.array([3.0, -4.0, 0.0, 12.0])           # ||W|| = 13
    g = np.array([0.5, -2.0, 1e-3, -7.0])
    Wn, m, v, phi = lamb_step(W, np.zeros(4), np.zeros(4), g, 1, 0.1, 0.9, 0.999, 0.0, 0.0)
    assert phi == pytest.approx(13.0 / 2.0, rel=1e-15)
    assert np.allclose(Wn, W - 0.1 * 6.5 * np.sign(g), rtol=0, atol=1e-14)
    assert np.allclose(m, 0.1 * g) and np.allclose(v, 0.001 * g * g)


def test_lamb_weight_decay_inside_trust_ratio():
    # LAMB adds the decay term to the adaptive step before the layer-wise
    # trust ratio is taken.  t = 1, eps = 0: m_hat = g, v_hat = g^2, so with
    # W = (2, 0), g = (-1, 1), wd = 0.5:  r = sign(g) + wd W = (0, 1),
    # ||W|| = 2, ||r|| = 1, phi = 2, W' = W - lr phi r = (2, -2 lr)
    W = np.array([2.0, 0.0])
    g = np.array([-1.0, 1.0])
    Wn, m, v, phi = lamb_step(W, np.zeros(2), np.zeros(2), g, 1, 0.25, 0.9, 0.999, 0.0, 0.5)
    assert phi == 2.0
    np.testing.assert_array_equal(Wn, np.array([2.0, -0.5]))


def test_lamb_zero_norms():
    # W = 0: phi = 1 (the raw adaptive step)
    Wn, _, _, phi = lamb_step(np.zeros(3), np.zeros(3), np.zeros(3), np.ones(3), 1, 0.5, 0.9, 0.999, 0.0, 0.0)
    assert phi == 1.0 and np.allclose(Wn, -0.5)
    # dW = 0 and wd = 0: r = 0, phi = 1, W unchanged
    W = np.arange(4.0)
    Wn, _, _, phi = lamb_step(W, np.zeros(4), np.zeros(4), np.zeros(4), 3, 0.5, 0.9, 0.999, 1e-6, 0.0)
    assert phi == 1.0 and np.array_equal(Wn, W)
