"""MKOR-H's switching rule: the reference in oracle/hybrid.py against switch
points derived by hand, then the library's host-side policy
(mkor_hybrid_init / mkor_hybrid_observe) against the reference."""
import ctypes
import math

import numpy as np
import pytest

import paper_2306_01685_amd as M
from oracle.hybrid import hybrid_decisions
from paper_2306_01685_amd import binding as B


def _f32(xs):
    return [float(np.float32(x)) for x in xs]


def test_reference_geometric_decay_then_plateau():
    # L_t = q^t for t < 20, then q^20.  Windows of 4: while the loss decays
    # geometrically every window mean is q^4 times the previous one, so
    # r = 1 - q^4 = 0.3439 > 0.05; the first plateau window (k = 5) has
    # r = 1 - 4 q^4 / (1 + q + q^2 + q^3) = 0.2369 > 0.05; windows 6 and 7 have
    # r = 0: slow twice (patience 2), so the switch comes when window 7
    # closes, at iteration 8 * 4 = 32.
    q = 0.9
    losses = [q ** min(t, 20) for t in range(60)]
    dec, sw = hybrid_decisions(losses, window=4, patience=2, warmup=1, threshold=0.05)
    assert sw == 32
    assert dec[:31] == [1] * 31 and dec[31:] == [0] * 29


def test_reference_threshold_zero_never_switches_on_a_falling_loss():
    losses = [1.0 / (1 + t) for t in range(200)]
    dec, sw = hybrid_decisions(losses, window=5, patience=1, warmup=1, threshold=0.0)
    assert sw is None and set(dec) == {1}


def test_reference_rising_loss_and_warmup():
    # a rising loss has r < 0 in every window: the first evaluated window is
    # slow.  warmup = 1: windows 1, 2 slow -> switch at (2 + 1) * 3 = 9;
    # warmup = 4: windows 4, 5 -> (5 + 1) * 3 = 18.
    losses = [1.0 + 0.1 * t for t in range(40)]
    assert hybrid_decisions(losses, 3, 2, 1, 0.01)[1] == 9
    assert hybrid_decisions(losses, 3, 2, 4, 0.01)[1] == 18


def test_reference_patience_resets_on_a_fast_window():
    # window means 10, 9.95 (slow), 5 (fast: resets), 4.99 (slow), 4.98 (slow)
    means = [10.0, 9.95, 5.0, 4.99, 4.98]
    losses = [m for m in means for _ in range(2)]
    dec, sw = hybrid_decisions(losses, window=2, patience=2, warmup=1, threshold=0.01)
    assert sw == 10


def test_reference_zero_mean_window():
    # a zero previous mean gives r = 0 (no measurable decrease)
    losses = [0.0] * 6
    assert hybrid_decisions(losses, 2, 1, 1, 0.0)[1] is None
    assert hybrid_decisions(losses, 2, 1, 1, 1e-6)[1] == 4


@pytest.fixture(scope="module")
def lib():
    return M.load_library()


@pytest.mark.parametrize("seed", range(12))
def test_library_policy_matches_reference(lib, seed):
    rng = np.random.default_rng(seed)
    window = int(rng.integers(1, 12))
    patience = int(rng.integers(1, 4))
    warmup = int(rng.integers(1, 5))
    threshold = float(np.float32(rng.choice([0.0, 1e-3, 1e-2, 5e-2])))
    n = 400
    # a decaying loss with noise, flattening out part-way
    t = np.arange(n)
    base = 3.0 * np.exp(-t / rng.uniform(20, 120)) + 1.0
    losses = _f32(base * (1 + rng.normal(0, rng.choice([0.0, 1e-3, 2e-2]), n)))
    ref, ref_sw = hybrid_decisions(losses, window, patience, warmup, threshold)
    h = M.Hybrid(window=window, patience=patience, warmup=warmup, threshold=threshold)
    got = [int(h.observe(x)) for x in losses]
    assert got == ref, (window, patience, warmup, threshold)
    assert h.switched_at == ref_sw
    assert h.state.windows == n // window and h.state.count == n % window


def test_library_policy_validation(lib):
    st = B.mkor_hybrid_state()
    for bad in [B.mkor_hybrid_params(0, 1, 1, 0.01), B.mkor_hybrid_params(4, 0, 1, 0.01),
                B.mkor_hybrid_params(4, 1, 0, 0.01), B.mkor_hybrid_params(4, 1, 1, -0.5),
                B.mkor_hybrid_params(4, 1, 1, math.nan), B.mkor_hybrid_params(4, 1, 1, math.inf)]:
        assert lib.mkor_hybrid_init(ctypes.byref(bad), ctypes.byref(st)) == M.MKOR_INVALID_ARG
        assert M.last_error()
    assert lib.mkor_hybrid_init(None, ctypes.byref(st)) == M.MKOR_INVALID_ARG
    good = B.mkor_hybrid_params(2, 1, 1, 0.01)
    assert lib.mkor_hybrid_init(ctypes.byref(good), None) == M.MKOR_INVALID_ARG
    assert lib.mkor_hybrid_init(ctypes.byref(good), ctypes.byref(st)) == M.MKOR_OK
    assert st.second_order == 1 and st.switched_at == -1 and math.isnan(st.last_rate)
    out = ctypes.c_int32(7)
    for bad_loss in (math.nan, math.inf, -math.inf):
        assert lib.mkor_hybrid_observe(ctypes.byref(st), bad_loss, ctypes.byref(out)) == M.MKOR_INVALID_ARG
    assert st.observed == 0 and out.value == 7   # rejected losses leave everything unchanged
    assert lib.mkor_hybrid_observe(ctypes.byref(st), 1.0, None) == M.MKOR_OK
    assert lib.mkor_hybrid_observe(None, 1.0, ctypes.byref(out)) == M.MKOR_INVALID_ARG
