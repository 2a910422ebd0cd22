// MKOR-H's switching rule (the paper's "Hybrid MKOR" subsection): watch how
// fast the training loss still falls and leave the second-order branch once
// the second-order updates stop paying for themselves.  Host-side only; the
// switch itself is mkor_set_second_order.
//
// The paper names the signal (the rate at which the loss decreases) and the
// direction (from second to first order, mid-training) but no formula.  The
// reading implemented here: losses are averaged over consecutive windows of
// `window` iterations; after each closed window k >= 1 the relative decrease
//     r_k = (m_{k-1} - m_k) / |m_{k-1}|      (0 when m_{k-1} = 0)
// of the window means is compared with `threshold`; once `patience`
// consecutive evaluated windows fall below it, the decision becomes
// first-order for the rest of training.  Windows before `warmup` closed
// windows are not evaluated.
#include "plan.h"

#include <cmath>

using namespace mkor;

namespace {

int check_hybrid(const mkor_hybrid_params* p) {
    if (p == nullptr) return fail(MKOR_INVALID_ARG, "hybrid params is NULL");
    if (p->window < 1) return fail(MKOR_INVALID_ARG, "window = %d must be >= 1", p->window);
    if (p->patience < 1) return fail(MKOR_INVALID_ARG, "patience = %d must be >= 1", p->patience);
    if (p->warmup < 1) return fail(MKOR_INVALID_ARG, "warmup = %d must be >= 1", p->warmup);
    if (!(p->threshold >= 0.f) || !std::isfinite(p->threshold))
        return fail(MKOR_INVALID_ARG, "threshold = %g must be finite and >= 0", (double)p->threshold);
    return MKOR_OK;
}

}  // namespace

extern "C" {

int mkor_hybrid_init(const mkor_hybrid_params* params, mkor_hybrid_state* state) {
    clear_error();
    if (state == nullptr) return fail(MKOR_INVALID_ARG, "state is NULL");
    const int st = check_hybrid(params);
    if (st != MKOR_OK) return st;
    *state = mkor_hybrid_state{};
    state->params = *params;
    state->second_order = 1;
    state->switched_at = -1;
    state->last_rate = NAN;
    return MKOR_OK;
}

int mkor_hybrid_observe(mkor_hybrid_state* state, float loss, int32_t* second_order) {
    clear_error();
    if (state == nullptr) return fail(MKOR_INVALID_ARG, "state is NULL");
    const int st = check_hybrid(&state->params);
    if (st != MKOR_OK) return st;
    if (!std::isfinite(loss)) return fail(MKOR_INVALID_ARG, "loss = %g is not finite", (double)loss);
    mkor_hybrid_state& s = *state;
    s.observed += 1;
    s.sum += (double)loss;
    s.count += 1;
    if (s.count == s.params.window) {
        const double mean = s.sum / s.params.window;
        if (s.windows >= 1) {
            const double prev = s.prev_mean;
            s.last_rate = prev != 0.0 ? (prev - mean) / std::fabs(prev) : 0.0;
            if (s.windows >= s.params.warmup) {
                s.slow = s.last_rate < (double)s.params.threshold ? s.slow + 1 : 0;
                if (s.second_order && s.slow >= s.params.patience) {
                    s.second_order = 0;
                    s.switched_at = s.observed;
                }
            }
        }
        s.prev_mean = mean;
        s.windows += 1;
        s.sum = 0.0;
        s.count = 0;
    }
    if (second_order != nullptr) *second_order = s.second_order;
    return MKOR_OK;
}

}  // extern "C"
