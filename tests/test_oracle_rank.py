"""Pins of the rank-r oracle (oracle/rank.py) against the mathematics: the
inverse of the accumulated factor computed by a library inversion, invariance
under the order of the vectors, zero vectors, the stabilised case, and the
rank-1 special case."""
import math

import numpy as np
import pytest

import oracle as O
from oracle.rank import layer_step_rank, sm_update_rank, update_factor_rank


def _spd(seed, d, spread=0.5):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((d, d))
    P = np.eye(d) + spread * (Q @ Q.T) / d
    return 0.5 * (P + P.T)


@pytest.mark.parametrize("d,r", [(1, 1), (2, 2), (5, 3), (16, 4), (64, 4), (40, 6)])
def test_rank_update_is_inverse_of_accumulation(d, r):
    rng = np.random.default_rng(d * 10 + r)
    P_hat = _spd(d + r, d)
    X = rng.standard_normal((d, r)) / math.sqrt(d)
    gamma = 0.9
    M = gamma * np.linalg.inv(P_hat) + (1.0 - gamma) * (X @ X.T)
    want = np.linalg.inv(M)
    got = sm_update_rank(P_hat, X, gamma)
    assert np.allclose(got, want, rtol=1e-10, atol=1e-12 * np.abs(want).max())


def test_rank_update_order_of_vectors_does_not_matter():
    rng = np.random.default_rng(7)
    P_hat = _spd(3, 24)
    X = rng.standard_normal((24, 4))
    a = sm_update_rank(P_hat, X, 0.8)
    b = sm_update_rank(P_hat, X[:, [2, 0, 3, 1]], 0.8)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-14)


def test_rank_update_zero_vectors_and_rank_one():
    P = _spd(4, 10)
    assert np.allclose(sm_update_rank(P, np.zeros((10, 3)), 0.75), P / 0.75, rtol=0, atol=1e-15)
    x = np.random.default_rng(5).standard_normal(10)
    p = O.Params(gamma=0.75, eps=math.inf)
    one, _ = O.update_factor(P, x, p)
    assert np.allclose(sm_update_rank(P, x[:, None], 0.75), one, rtol=1e-13, atol=1e-15)


def test_rank_update_stabilised_and_spd():
    rng = np.random.default_rng(11)
    P = 50.0 * _spd(8, 12)
    X = rng.standard_normal((12, 3))
    p = O.Params(gamma=0.9, zeta=0.5, eps=1.0)
    got, st = update_factor_rank(P, X, p)
    assert st.stab and st.nu == pytest.approx(np.abs(P).sum(axis=1).max())
    P_hat = 0.5 * P + 0.5 * np.eye(12)
    want = np.linalg.inv(0.9 * np.linalg.inv(P_hat) + 0.1 * X @ X.T)
    assert np.allclose(got, want, rtol=1e-10)
    assert st.s == pytest.approx(float(X[:, 0] @ P_hat @ X[:, 0]))
    # stays symmetric positive definite (Lemma 1's property, for rank r)
    assert np.allclose(got, got.T, atol=1e-12)
    np.linalg.cholesky(got)


def test_rank_update_rejects_printed_variant():
    with pytest.raises(ValueError):
        update_factor_rank(np.eye(3), np.ones((3, 2)), O.Params(variant=O.PAPER_EQ6))


def test_layer_step_rank_wiring():
    # A drives Linv (d_in), Gv drives Rinv (d_out); dW = rescaled Linv G Rinv
    rng = np.random.default_rng(2)
    d_in, d_out, r = 6, 9, 2
    A = rng.standard_normal((d_in, r))
    Gv = rng.standard_normal((d_out, r))
    G = rng.standard_normal((d_in, d_out))
    p = O.Params(gamma=0.9, eps=math.inf)
    L, R, dW, st = layer_step_rank(np.eye(d_in), np.eye(d_out), A, Gv, G, p)
    assert np.allclose(L, np.linalg.inv(0.9 * np.eye(d_in) + 0.1 * A @ A.T))
    assert np.allclose(R, np.linalg.inv(0.9 * np.eye(d_out) + 0.1 * Gv @ Gv.T))
    assert np.linalg.norm(dW) == pytest.approx(np.linalg.norm(G))
    assert np.allclose(dW / np.linalg.norm(dW), (L @ G @ R) / np.linalg.norm(L @ G @ R))
