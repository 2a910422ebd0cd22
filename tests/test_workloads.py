"""Synthetic input generator: reproducibility, shapes and distributions."""
import numpy as np
import pytest

import workloads as W


def test_config_shapes():
    assert W.SINGLE_64.shapes == ((64, 64),)
    assert W.BERT_BASE.n_layers == 72
    assert W.BERT_LARGE.n_layers == 144 and W.BERT_LARGE.grad_dtype == "bf16"
    assert W.SINGLE_8192.shapes == ((8192, 8192),) and W.SINGLE_8192.gamma == 0.95
    assert W.GPT2_XL.n_layers == 192
    # algorithmic sizes used for the roofline (factor elements, precondition flops)
    assert W.BERT_LARGE.factor_elems == 1_056_964_608
    assert abs(W.BERT_LARGE.precond_flops - 2.474e12) / 2.474e12 < 1e-3
    assert abs(W.GPT2_XL.precond_flops - 21.23e12) / 21.23e12 < 1e-3


def test_reproducible_and_independent():
    w = W.BERT_BASE
    a1, g1 = W.rank1_vectors(w, 5, 3)
    a2, g2 = W.rank1_vectors(w, 5, 3)
    np.testing.assert_array_equal(a1, a2)
    np.testing.assert_array_equal(g1, g2)
    a3, _ = W.rank1_vectors(w, 5, 4)
    assert not np.array_equal(a1, a3)
    G1, G2 = W.gradient(w, 0, 0), W.gradient(w, 0, 0)
    np.testing.assert_array_equal(G1, G2)
    assert G1.dtype == np.float32 and G1.shape == (768, 768)


def test_mean_distribution_explicit_vs_shortcut():
    w = W.custom([(512, 512)], rows=256, cid=900)
    ae, ge = W.rank1_vectors(w, 0, 0, explicit=True)
    a, g = W.rank1_vectors(w, 0, 0, explicit=False)
    # std of the mean of 256 N(0,1) rows is 1/16; grads 1e-3/16
    for v, s in ((ae, 1 / 16), (a, 1 / 16), (ge, 1e-3 / 16), (g, 1e-3 / 16)):
        assert abs(v.std() / s - 1) < 0.15


def test_student_t_rows_heavier_tail():
    w = W.custom([(256, 256)], rows=64, cid=901, act_dist="student_t4")
    a, _ = W.rank1_vectors(w, 0, 0, explicit=True)
    assert abs(a.std() / np.sqrt(2 / 64) - 1) < 0.2


def test_bf16_rounding():
    x = np.array([1.0, 1.00390625, 1.005859375, -3.3, np.float32(2 ** -130)], dtype=np.float32)
    r = W.round_to_bf16(x)
    assert (r.view(np.uint32) & 0xFFFF == 0).all()
    assert r[0] == 1.0
    assert r[1] == 1.0        # tie -> even
    assert r[2] == 1.0078125  # rounds up
    torch = pytest.importorskip("torch")
    t = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(r, t)
    G = W.gradient(W.BERT_LARGE, 0, 0)
    assert (G.view(np.uint32) & 0xFFFF == 0).all()


def test_perturbed_init_spd_symmetric():
    w = W.custom([(96, 80)], cid=902, init="perturbed")
    L, R = W.initial_factors(w, 0)
    assert L.shape == (96, 96) and R.shape == (80, 80)
    np.testing.assert_array_equal(L, L.T)
    np.linalg.cholesky(L.astype(np.float64))
    assert abs(np.trace(L) / 96 - 1.0 - 0.01 * 64 / 96) < 0.01


def test_token_rows_seeded_and_shaped():
    w = W.SINGLE_64
    A, Go = W.token_rows(w, 0, 3)
    assert A.shape == (32, 64) and Go.shape == (32, 64) and A.dtype == np.float32
    A2, Go2 = W.token_rows(w, 0, 3)
    np.testing.assert_array_equal(A, A2)
    np.testing.assert_array_equal(Go, Go2)
    assert not np.array_equal(A, W.token_rows(w, 0, 4)[0])
    Ab, Gb = W.token_rows(w, 0, 3, rows=7, dtype="bf16")
    assert Ab.shape == (7, 64)
    np.testing.assert_array_equal(Ab, W.round_to_bf16(Ab))
    assert 0.5 < float(A.std()) < 1.5 and float(Go.std()) < 1e-2
