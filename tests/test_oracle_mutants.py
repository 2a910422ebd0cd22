"""Mistakes planted in the float64 oracle, on the CPU, each caught by its pins.

Every mutant below is one plausible slip in writing Algorithm 1 down: a wrong
sign, a dropped or swapped term, a transposed operand, a swapped side, a
stale operand, an off-by-one in a mean, a misread threshold.  Each is put in
place of the oracle function it touches, and the pins of
``tests/test_oracle.py`` (worked 2x2 examples, brute-force inversion of the
explicitly accumulated factor, closed forms, exact rationals, library
routines, invariants), called here as plain functions, must fail for it; the
same for the rank-r oracle (``tests/test_oracle_rank.py``) and the backend
optimizer's (``tests/test_oracle_optimizer.py``: hand values, torch's SGD and
AdamW).
The unmutated oracle passes all of them.  A mutant no pin catches would be a
hole in the pins.
"""
import math

import numpy as np
import pytest

import oracle as O
import oracle.half as HF
import oracle.hybrid as HY
import oracle.mkor_oracle as M
import oracle.optimizer as OPT
import oracle.rank as RK
import tests.test_hybrid as THY
import tests.test_oracle as T
import tests.test_oracle_half as TH
import tests.test_oracle_optimizer as TO
import tests.test_oracle_rank as TR

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# --------------------------------------------------------------- the pins

def _pins():
    return [
        ("golden_sm_exact", lambda: T.test_golden_sm_step("sm_exact_2x2.txt")),
        ("golden_sm_exact_stab", lambda: T.test_golden_sm_step("sm_exact_stab_2x2.txt")),
        ("golden_sm_eq6", lambda: T.test_golden_sm_step("sm_paper_eq6_2x2.txt")),
        ("golden_precond_rescale", T.test_golden_precond_rescale),
        ("golden_norms", T.test_golden_norms),
        ("norm_vs_numpy", lambda: T.test_norm_matches_numpy_linalg(17)),
        ("brute_force", lambda: T.test_exact_matches_inverse_of_accumulated_factor(5)),
        ("brute_force_stab", lambda: T.test_exact_with_stabiliser_matches_brute_force(16, 5.0, O.NORM_INF)),
        ("brute_force_stab_maxabs", lambda: T.test_exact_with_stabiliser_matches_brute_force(16, 2.5, O.NORM_MAXABS)),
        ("closed_form", T.test_closed_form_repeated_vector),
        ("scalar", T.test_scalar_case),
        ("zero_vector", T.test_zero_vector),
        ("rationals", lambda: T.test_exact_rational_accumulation(3)),
        ("spd_exact", lambda: T.test_factors_stay_spd_and_symmetric(O.EXACT)),
        ("spd_eq6", lambda: T.test_factors_stay_spd_and_symmetric(O.PAPER_EQ6)),
        ("eq11", T.test_stabiliser_blend_matches_eq11_expansion),
        ("thresholds", T.test_stabiliser_thresholds),
        ("kronecker", T.test_precondition_matches_kronecker_form),
        ("identity_factors", T.test_identity_and_scalar_factors_give_gradient),
        ("rescale_descent", T.test_rescale_norm_and_descent),
        ("layer_pairs", T.test_layer_pairs_a_with_left_and_g_with_right),
        ("first_order", T.test_first_order_layer_passes_gradient),
        ("guard", T.test_guard_nonfinite),
        ("means_rationals", T.test_rank1_means_exact_rationals),
        ("means_identical_rows", T.test_rank1_means_identical_rows_make_the_approximation_exact),
        ("means_invariances", T.test_rank1_means_invariances),
        ("layer_rows", T.test_layer_step_rows_uses_row_means),
        ("grouped_step", T.test_oracle_step_grouped_against_brute_force),
    ]


def _failing_pins():
    return _failing(_pins())


# --------------------------------------------------------------- the mutants
# Each returns {oracle attribute: replacement}; the replacement follows the
# original function with the one change its name says.

def _sm(change):
    def sm_update(P_hat, x, gamma, variant=O.EXACT):
        u = P_hat @ x
        s = float(x @ u)
        if variant == O.EXACT:
            k = (1.0 - gamma) / (gamma + (1.0 - gamma) * s)
            P_new = (P_hat - k * np.outer(u, u)) / gamma
            if change == "sign":
                P_new = (P_hat + k * np.outer(u, u)) / gamma
            elif change == "denominator":
                k = (1.0 - gamma) / (gamma + s)
                P_new = (P_hat - k * np.outer(u, u)) / gamma
            elif change == "no_inv_gamma":
                P_new = P_hat - k * np.outer(u, u)
            elif change == "s_xx":
                s = float(x @ x)
                k = (1.0 - gamma) / (gamma + (1.0 - gamma) * s)
                P_new = (P_hat - k * np.outer(u, u)) / gamma
            elif change == "momentum_swapped":
                k = gamma / ((1.0 - gamma) + gamma * s)
                P_new = (P_hat - k * np.outer(u, u)) / (1.0 - gamma)
        else:
            k = (1.0 - gamma) / (gamma * gamma * (1.0 + gamma * (1.0 - gamma) * s))
            P_new = gamma * P_hat + k * np.outer(u, u)
            if change == "eq6_sign":
                P_new = gamma * P_hat - k * np.outer(u, u)
            elif change == "eq6_gamma_power":
                k = (1.0 - gamma) / (gamma * (1.0 + gamma * (1.0 - gamma) * s))
                P_new = gamma * P_hat + k * np.outer(u, u)
        return P_new, u, s, k
    return {"sm_update": sm_update}


def _stabilize(change):
    def stabilize(P, nu, eps, zeta):
        fire = nu >= eps if change == "ge" else nu > eps
        if fire:
            I = np.eye(P.shape[0])
            return ((1.0 - zeta) * P + zeta * I if change == "blend_reversed" else zeta * P + (1.0 - zeta) * I), True
        return P, False
    return {"stabilize": stabilize}


def _norm(change):
    def factor_norm(P, norm_kind=O.NORM_INF):
        A = np.asarray(P, dtype=np.float64)
        if change != "no_abs":
            A = np.abs(A)
        if A.size == 0:
            return 0.0
        if norm_kind == O.NORM_INF:
            return float(A.sum(axis=0 if change == "columns" else 1).max())
        return float(A.max())
    return {"factor_norm": factor_norm}


def _update_factor(change):
    def update_factor(P, x, p, stab_override=None):
        P = np.asarray(P, dtype=np.float64)
        x = np.asarray(x, dtype=np.float64)
        st = O.FactorStats()
        st.nu = M.factor_norm(P, p.norm_kind)
        if change == "stab_after_update":
            P_new, _u, st.s, k = M.sm_update(P, x, p.gamma, p.variant)
            P_new, st.stab = M.stabilize(P_new, M.factor_norm(P_new, p.norm_kind), p.eps, p.zeta)
            return P_new, st
        P_hat, st.stab = M.stabilize(P, st.nu, p.eps, p.zeta)
        if stab_override is not None:
            st.stab = bool(stab_override)
            P_hat = p.zeta * P + (1.0 - p.zeta) * np.eye(P.shape[0]) if st.stab else P
        with np.errstate(all="ignore"):
            P_new, _u, st.s, k = M.sm_update(P_hat, x, p.gamma, p.variant)
            if change == "u_from_unblended":   # u and s from P, the rest from P_hat
                u = P @ x
                s = float(x @ u)
                k = (1.0 - p.gamma) / (p.gamma + (1.0 - p.gamma) * s)
                P_new = (P_hat - k * np.outer(u, u)) / p.gamma
        bad = not (math.isfinite(st.nu) and math.isfinite(st.s) and math.isfinite(k))
        if bad and p.guard_nonfinite:
            st.skipped = True
            return P.copy(), st
        st.skipped = bad
        return P_new, st
    return {"update_factor": update_factor}


def _precondition(change):
    def precondition(Linv, G, Rinv):
        L, G, R = (np.asarray(v, np.float64) for v in (Linv, G, Rinv))
        if change == "drops_right":
            return L @ G
        if change == "right_transposed":
            return L @ G @ R.T
        if change == "left_transposed":
            return L.T @ G @ R
        return (L @ G) @ R
    return {"precondition": precondition}


def _rescale(change):
    def rescale(G, dW_hat):
        nG = float(np.linalg.norm(np.asarray(G, np.float64)))
        nD = float(np.linalg.norm(dW_hat))
        if change == "inverted":
            scale = nD / nG if nG > 0.0 else 0.0
        elif change == "missing":
            scale = 1.0
        else:
            scale = nG / nD if nD > 0.0 else 0.0
        return scale * dW_hat, nG, nD, scale
    return {"rescale": rescale}


def _layer_step(change):
    original = M.layer_step

    def layer_step(Linv, Rinv, a, g, G, p, second_order=True, stab_override=(None, None),
                   update=True, precond=True):
        if change == "vectors_swapped":
            return original(Linv, Rinv, g, a, G, p, second_order, stab_override, update, precond)
        if change == "stale_factors" and second_order and update and precond:
            Li, Ri, _, st = original(Linv, Rinv, a, g, G, p, True, stab_override, True, False)
            _, _, dW, st2 = original(Linv, Rinv, a, g, G, p, True, stab_override, False, True)
            st.norm_G, st.norm_dW_hat, st.scale = st2.norm_G, st2.norm_dW_hat, st2.scale
            return Li, Ri, dW, st
        return original(Linv, Rinv, a, g, G, p, second_order, stab_override, update, precond)
    return {"layer_step": layer_step}


def _means(change):
    def rank1_means(rows):
        R = np.asarray(rows, dtype=np.float64)
        if R.ndim != 2 or R.shape[0] == 0:
            raise ValueError("rows must be a non-empty b x d array")
        if change == "bessel":
            return R.sum(axis=0) / max(R.shape[0] - 1, 1)
        return R.sum(axis=1) / R.shape[1]   # "axis": averages the wrong way
    return {"rank1_means": rank1_means}


def _oracle_step(change):
    def oracle_step(layers, p, update=True, precond=True, stab_overrides=None):
        out = []
        n = len(layers)
        for i, L in enumerate(layers):
            if stab_overrides is None:
                ov = (None, None)
            else:
                ov = stab_overrides[(i + 1) % n] if change == "override_shifted" else stab_overrides[i]
            so = True if change == "ignores_first_order" else bool(L.get("second_order", True))
            Li, Ri, dW, st = M.layer_step(L["Linv"], L["Rinv"], L["a"], L["g"], L["G"], p, so, ov, update, precond)
            out.append(dict(Linv=Li, Rinv=Ri, dW=dW, stats=st))
        return out
    return {"oracle_step": oracle_step}


MUTANTS = {
    "sm_sign": _sm("sign"),
    "sm_denominator_drops_1_minus_gamma": _sm("denominator"),
    "sm_missing_1_over_gamma": _sm("no_inv_gamma"),
    "sm_s_is_xTx": _sm("s_xx"),
    "sm_momentum_weights_swapped": _sm("momentum_swapped"),
    "eq6_sign": _sm("eq6_sign"),
    "eq6_gamma_power": _sm("eq6_gamma_power"),
    "stab_blend_reversed": _stabilize("blend_reversed"),
    "stab_fires_at_equality": _stabilize("ge"),
    "norm_column_sums": _norm("columns"),
    "norm_without_abs": _norm("no_abs"),
    "stab_after_update": _update_factor("stab_after_update"),
    "u_from_unblended_factor": _update_factor("u_from_unblended"),
    "precond_drops_right_factor": _precondition("drops_right"),
    "precond_right_transposed": _precondition("right_transposed"),
    "precond_left_transposed": _precondition("left_transposed"),
    "rescale_inverted": _rescale("inverted"),
    "rescale_missing": _rescale("missing"),
    "layer_vectors_swapped": _layer_step("vectors_swapped"),
    "layer_preconditions_with_stale_factors": _layer_step("stale_factors"),
    "means_divide_by_b_minus_1": _means("bessel"),
    "means_wrong_axis": _means("axis"),
    "step_ignores_first_order_flag": _oracle_step("ignores_first_order"),
    "step_override_shifted": _oracle_step("override_shifted"),
}


# ------------------------------------------------ the rank-r oracle and its pins

def _rank_pins():
    return [
        ("inverse_of_accumulation", lambda: [TR.test_rank_update_is_inverse_of_accumulation(d, r)
                                             for d, r in ((2, 2), (5, 3), (16, 4))]),
        ("order_of_vectors", TR.test_rank_update_order_of_vectors_does_not_matter),
        ("zero_vectors_and_rank_one", TR.test_rank_update_zero_vectors_and_rank_one),
        ("stabilised_and_spd", TR.test_rank_update_stabilised_and_spd),
        ("rejects_printed_variant", TR.test_rank_update_rejects_printed_variant),
        ("layer_wiring", TR.test_layer_step_rank_wiring),
    ]


def _rank_sm(change):
    def sm_update_rank(P_hat, X, gamma):
        X = np.asarray(X, dtype=np.float64).reshape(P_hat.shape[0], -1)
        P0 = np.asarray(P_hat, dtype=np.float64) / (1.0 if change == "no_inv_gamma" else gamma)
        P = P0
        for i in range(1 if change == "first_vector_only" else X.shape[1]):
            y = (1.0 - gamma) * X[:, i] if change == "no_sqrt" else math.sqrt(1.0 - gamma) * X[:, i]
            u = (P0 if change == "u_from_start" else P) @ y
            den = float(y @ u) if change == "drops_one" else 1.0 + float(y @ u)
            P = P + np.outer(u, u) / den if change == "sign" else P - np.outer(u, u) / den
        return P
    return {"sm_update_rank": sm_update_rank}


RANK_MUTANTS = {
    "rank_sign": _rank_sm("sign"),
    "rank_denominator_drops_1": _rank_sm("drops_one"),
    "rank_missing_1_over_gamma": _rank_sm("no_inv_gamma"),
    "rank_missing_sqrt_on_1_minus_gamma": _rank_sm("no_sqrt"),
    "rank_only_first_vector": _rank_sm("first_vector_only"),
    "rank_u_from_starting_factor": _rank_sm("u_from_start"),
}


# ---------------------------------------------- the optimizer oracle and its pins

def _opt_pins():
    return [
        ("sgd_hand", TO.test_sgd_hand_values),
        ("sgd_torch", TO.test_sgd_matches_torch),
        ("lamb_adamw", TO.test_lamb_without_trust_is_adamw),
        ("lamb_first_step", TO.test_lamb_first_step_trust_ratio),
        ("lamb_decay_in_trust", TO.test_lamb_weight_decay_inside_trust_ratio),
        ("lamb_zero_norms", TO.test_lamb_zero_norms),
    ]


def _sgd(change):
    def sgd_step(W, m, g, lr, momentum, wd):
        W = np.asarray(W, np.float64)
        g = np.asarray(g, np.float64)
        if change == "decay_after_momentum":
            m = momentum * np.asarray(m, np.float64) + g
            return W - lr * (m + wd * W), m
        d = g + wd * W
        m = momentum * np.asarray(m, np.float64) + (1.0 - momentum) * d
        return W - lr * m, m   # "dampened": momentum also scales the new term
    return {"sgd_step": sgd_step}


def _lamb(change):
    def lamb_step(W, m, v, g, t, lr, beta1, beta2, eps, wd, trust=True):
        W = np.asarray(W, np.float64)
        g = np.asarray(g, np.float64)
        m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
        v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * (np.abs(g) if change == "v_of_g" else g * g)
        m_hat = m if change == "no_bias_correction" else m / (1.0 - beta1 ** t)
        v_hat = v if change == "no_bias_correction" else v / (1.0 - beta2 ** t)
        adam = m_hat / (np.sqrt(v_hat + eps) if change == "eps_inside_sqrt" else np.sqrt(v_hat) + eps)
        r = adam if change == "decay_outside_trust" else adam + wd * W
        nW, nr = float(np.linalg.norm(W)), float(np.linalg.norm(r))
        ok = trust and nW > 0.0 and nr > 0.0
        phi = (nr / nW if change == "trust_inverted" else nW / nr) if ok else 1.0
        step = phi * r + (wd * W if change == "decay_outside_trust" else 0.0)
        return W - lr * step, m, v, phi
    return {"lamb_step": lamb_step}


OPT_MUTANTS = {
    "sgd_decay_after_momentum": _sgd("decay_after_momentum"),
    "sgd_dampened_momentum": _sgd("dampened"),
    "lamb_no_bias_correction": _lamb("no_bias_correction"),
    "lamb_eps_inside_sqrt": _lamb("eps_inside_sqrt"),
    "lamb_trust_ratio_inverted": _lamb("trust_inverted"),
    "lamb_decay_outside_trust_ratio": _lamb("decay_outside_trust"),
    "lamb_second_moment_of_abs_g": _lamb("v_of_g"),
}


# ------------------------------------------- the half-precision oracle and its pins

def _half_pins():
    return [
        ("round_vs_library_cast", TH.test_round_matches_library_cast),
        ("round_hand_values", lambda: [TH.test_round_hand_values(x, w) for x, w in (
            (1.0 + 2.0 ** -8, 1.0), (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6), (2.0 ** -133 * 1.5, 2.0 ** -132),
            ((2.0 - 2.0 ** -8) * 2.0 ** 127, math.inf))]),
        ("round_properties", TH.test_round_properties),
        ("exact_case", TH.test_exact_case_equals_fp64_step),
        ("intermediate_rounded", TH.test_intermediate_is_rounded),
        ("gradient_rounded", TH.test_gradient_enters_rounded),
        ("stored_state", TH.test_stored_state_and_update_from_it),
        ("fresh_factor", TH.test_preconditioning_uses_fresh_factor),
        ("lemma2", lambda: TH.test_lemma2_bound(64)),
        ("close_to_fp64", TH.test_half_step_close_to_full_precision),
    ]


def _round(change):
    def round_bf16(x):
        x = np.asarray(x, dtype=np.float64)
        out = np.empty_like(x)
        fin = np.isfinite(x)
        out[~fin] = x[~fin]
        v = x[fin]
        _m, k = np.frexp(np.abs(v))
        e = np.maximum(k - 1, HF.BF16_EMIN)
        q = np.ldexp(1.0, e - (HF.BF16_MANT - (2 if change == "seven_bits" else 1)))
        if change == "truncate":
            r = np.trunc(v / q) * q
        elif change == "ties_away":
            r = np.sign(v) * np.floor(np.abs(v) / q + 0.5) * q
        else:
            r = np.rint(v / q) * q
        big = np.abs(r) >= 2.0 ** 128
        r[big] = np.copysign(np.inf, r[big])
        out[fin] = r
        return out
    return {"round_bf16": round_bf16}


def _precond_half(change):
    def precondition_half(PL, G_h, PR):
        PL, G_h, PR = (np.asarray(v, np.float64) for v in (PL, G_h, PR))
        if change == "other_intermediate":          # (PL G) rounded, then times PR
            X = HF.round_bf16(PL @ G_h)
            return X @ PR, X
        Y = G_h @ PR
        Y_h = Y if change == "y_unrounded" else HF.round_bf16(Y)
        return PL @ Y_h, Y_h
    return {"precondition_half": precondition_half}


def _step_half(change):
    def layer_step_half(PL, PR, a, g, G, p, stab_override=(None, None), update=True, precond=True):
        st = O.LayerStats()
        PL = np.asarray(PL, dtype=np.float64)
        PR = np.asarray(PR, dtype=np.float64)
        if update:
            QL, QR = (PL, PR) if change == "update_from_unrounded" else (HF.round_bf16(PL), HF.round_bf16(PR))
            PL, st.L = O.update_factor(QL, a, p, stab_override[0])
            PR, st.R = O.update_factor(QR, g, p, stab_override[1])
        dW = None
        if precond:
            G64 = np.asarray(G, np.float64)
            G_h = G64 if change == "gradient_unrounded" else HF.round_bf16(G64)
            PLp, PRp = (HF.round_bf16(PL), HF.round_bf16(PR)) if change == "rounded_factor" else (PL, PR)
            with np.errstate(all="ignore"):
                dW_hat, _ = HF.precondition_half(PLp, G_h, PRp)
                Gn = G64 if change == "norm_of_unrounded_gradient" else G_h
                if p.rescale:
                    dW, st.norm_G, st.norm_dW_hat, st.scale = O.rescale(Gn, dW_hat)
                else:
                    dW = dW_hat
                    st.norm_G = float(np.linalg.norm(Gn))
                    st.norm_dW_hat = float(np.linalg.norm(dW_hat))
                    st.scale = 1.0
        return PL, PR, dW, st
    return {"layer_step_half": layer_step_half}


HALF_MUTANTS = {
    "bf16_truncates": _round("truncate"),
    "bf16_ties_away_from_zero": _round("ties_away"),
    "bf16_seven_bit_significand": _round("seven_bits"),
    "half_y_not_rounded": _precond_half("y_unrounded"),
    "half_rounds_the_other_intermediate": _precond_half("other_intermediate"),
    "half_update_from_unrounded_factor": _step_half("update_from_unrounded"),
    "half_preconditions_with_rounded_factor": _step_half("rounded_factor"),
    "half_gradient_not_rounded": _step_half("gradient_unrounded"),
    "half_norm_of_unrounded_gradient": _step_half("norm_of_unrounded_gradient"),
}


# ------------------------------------------------ the MKOR-H rule and its pins

def _hybrid_pins():
    return [(n, getattr(THY, n)) for n in sorted(dir(THY)) if n.startswith("test_reference_")]


def _hybrid(change):
    def hybrid_decisions(losses, window, patience, warmup, threshold):
        decisions, means = [], []
        slow, decision, switched = 0, 1, None
        for t in range(1, len(losses) + 1):
            if t % window == 0:
                mean = sum(float(x) for x in losses[t - window:t]) / window
                k = len(means)
                first = 0 if change == "counts_first_window" else 1
                if k >= first and k >= (warmup + 1 if change == "warmup_off_by_one" else warmup) and means:
                    prev = means[-1]
                    if change == "rate_sign":
                        rate = (mean - prev) / abs(prev) if prev != 0.0 else 0.0
                    elif change == "rate_not_relative":
                        rate = prev - mean
                    else:
                        rate = (prev - mean) / abs(prev) if prev != 0.0 else 0.0
                    is_slow = rate <= threshold if change == "le" else rate < threshold
                    if change == "patience_never_resets":
                        slow = slow + 1 if is_slow else slow
                    else:
                        slow = slow + 1 if is_slow else 0
                    need = patience + 1 if change == "patience_strict" else patience
                    if decision == 1 and slow >= need:
                        decision, switched = 0, t
                means.append(mean)
            decisions.append(decision)
        return decisions, switched
    return {"hybrid_decisions": hybrid_decisions}


HYBRID_MUTANTS = {
    "hybrid_rate_sign": _hybrid("rate_sign"),
    "hybrid_rate_not_relative": _hybrid("rate_not_relative"),
    "hybrid_le_threshold": _hybrid("le"),
    "hybrid_patience_never_resets": _hybrid("patience_never_resets"),
    "hybrid_patience_off_by_one": _hybrid("patience_strict"),
    "hybrid_warmup_off_by_one": _hybrid("warmup_off_by_one"),
}


def _failing(pins):
    failed = []
    for name, pin in pins:
        try:
            pin()
        except pytest.skip.Exception:
            pass
        except Exception:
            failed.append(name)
    return failed


def _plant(monkeypatch, repl, *modules):
    """The mutant replaces the name in every module that holds it (the
    oracle, the package re-export, a pin module that imported it by name)."""
    for name, fn in repl.items():
        for mod in modules:
            if hasattr(mod, name):
                monkeypatch.setattr(mod, name, fn)


def test_unmutated_oracles_pass_every_pin():
    assert _failing_pins() == []
    assert _failing(_rank_pins()) == []
    assert _failing(_opt_pins()) == []
    assert _failing(_half_pins()) == []
    assert _failing(_hybrid_pins()) == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_planted_mistake(monkeypatch, mutant):
    _plant(monkeypatch, MUTANTS[mutant], M, O)
    failed = _failing_pins()
    assert failed, f"no pin catches the mutant {mutant}"


@pytest.mark.parametrize("mutant", sorted(RANK_MUTANTS))
def test_rank_pins_catch_planted_mistake(monkeypatch, mutant):
    _plant(monkeypatch, RANK_MUTANTS[mutant], RK, TR)
    assert _failing(_rank_pins()), f"no rank-r pin catches the mutant {mutant}"


@pytest.mark.parametrize("mutant", sorted(OPT_MUTANTS))
def test_optimizer_pins_catch_planted_mistake(monkeypatch, mutant):
    _plant(monkeypatch, OPT_MUTANTS[mutant], OPT, TO)
    assert _failing(_opt_pins()), f"no optimizer pin catches the mutant {mutant}"


@pytest.mark.parametrize("mutant", sorted(HALF_MUTANTS))
def test_half_pins_catch_planted_mistake(monkeypatch, mutant):
    _plant(monkeypatch, HALF_MUTANTS[mutant], HF, TH)
    assert _failing(_half_pins()), f"no half-precision pin catches the mutant {mutant}"


@pytest.mark.parametrize("mutant", sorted(HYBRID_MUTANTS))
def test_hybrid_pins_catch_planted_mistake(monkeypatch, mutant):
    _plant(monkeypatch, HYBRID_MUTANTS[mutant], HY, THY)
    assert _failing(_hybrid_pins()), f"no MKOR-H pin catches the mutant {mutant}"
