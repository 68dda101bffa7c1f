// Host parts of ADPSGD: the learning-rate schedules and the adaptive period
// controller (Algorithm 2's initial state, sampling and period decision).  No
// device call here, so the controller runs and is tested without a GPU; its
// rules are the inline functions of schedule.hpp, which the device reduction
// kernel also uses.
#include <algorithm>
#include <climits>
#include <cmath>
#include <limits>

#include "adpsgd.h"
#include "common.hpp"
#include "schedule.hpp"

namespace adpsgd {

bool hparams_valid(const adpsgd_hparams *hp, std::string *why) {
    auto bad = [&](const char *m) { if (why) *why = m; return false; };
    if (!hp) return bad("hparams is NULL");
    if (!(std::isfinite(hp->sigma) && hp->sigma >= 0)) return bad("sigma must be finite and >= 0");
    if (!(hp->momentum >= 0 && hp->momentum < 1)) return bad("momentum must be in [0, 1)");
    if (!(std::isfinite(hp->weight_decay) && hp->weight_decay >= 0)) return bad("weight_decay must be finite and >= 0");
    if (!(hp->h_lo > 0 && hp->h_lo <= hp->h_hi && std::isfinite(hp->h_hi))) return bad("need 0 < h_lo <= h_hi < inf");
    if (hp->lr_kind < ADPSGD_LR_CONST) return bad("unknown lr_kind");
    if (hp->period_mode != ADPSGD_PERIOD_CONST && hp->period_mode != ADPSGD_PERIOD_ADAPTIVE &&
        hp->period_mode != ADPSGD_PERIOD_ALG1)
        return bad("unknown period_mode");
    if (!(std::isfinite(hp->lr0) && hp->lr0 > 0)) return bad("lr0 must be finite and > 0");
    if (hp->total_steps < 1) return bad("total_steps must be >= 1");
    if (hp->p_init < 1) return bad("p_init must be >= 1");
    if (hp->p_max < 0 || (hp->p_max > 0 && hp->p_max < hp->p_init)) return bad("need p_max == 0 or p_max >= p_init");
    if (hp->k_s < 0) return bad("k_s must be >= 0");
    if (!(std::isfinite(hp->thr_lo) && std::isfinite(hp->thr_hi) && hp->thr_lo > 0 && hp->thr_lo <= hp->thr_hi))
        return bad("need 0 < thr_lo <= thr_hi");
    if (hp->lr_kind > ADPSGD_LR_WARMUP_STEP) return bad("unknown lr_kind");
    if (hp->sync_warmup_steps < 0) return bad("sync_warmup_steps must be >= 0");
    if (hp->p_switch_step < 0) return bad("p_switch_step must be >= 0");
    if (hp->p_switch_step > 0 && hp->period_mode == ADPSGD_PERIOD_ADAPTIVE)
        return bad("p_switch_step applies to the constant period modes only");
    if (hp->p_switch_step > 0 && (hp->p_after < 1 || (hp->p_max > 0 && hp->p_after > hp->p_max)))
        return bad("p_after must be in [1, p_max] when p_switch_step is set");
    if (hp->avg_momentum != 0 && hp->avg_momentum != 1) return bad("avg_momentum must be 0 or 1");
    return true;
}

int32_t p_max_of(const adpsgd_hparams *hp) { return hp->p_max > 0 ? hp->p_max : INT32_MAX; }

SchedRule rule_of(const adpsgd_hparams *hp) {
    SchedRule r{};
    r.period_mode = hp->period_mode;
    r.p_after = hp->p_after;
    r.p_max = p_max_of(hp);
    r.k_s = hp->k_s;
    r.warmup = hp->sync_warmup_steps;
    r.p_switch_step = hp->p_switch_step;
    r.thr_lo = hp->thr_lo;
    r.thr_hi = hp->thr_hi;
    return r;
}

}  // namespace adpsgd

using namespace adpsgd;

extern "C" double adpsgd_lr(const adpsgd_hparams *hp, int64_t t) {
    if (!hp) return std::numeric_limits<double>::quiet_NaN();
    switch (hp->lr_kind) {
    case ADPSGD_LR_STEP: {
        // two 10x decays, at the half and three-quarter points of the schedule
        const int n_decays = (t >= hp->total_steps / 2) + (t >= (3 * hp->total_steps) / 4);
        double g = hp->lr0;
        for (int d = 0; d < n_decays; ++d) g *= 0.1;
        return g;
    }
    case ADPSGD_LR_COSINE:
        return 0.5 * hp->lr0 * (1.0 + std::cos(M_PI * (double)t / (double)hp->total_steps));
    case ADPSGD_LR_WARMUP_STEP: {
        // 90 "epochs" of E steps: a linear ramp over the first 8 (lr0, 2 lr0, ...,
        // 8 lr0), then 8 lr0 with 10x decays at epochs 30 and 60
        const int64_t E = std::max<int64_t>(1, hp->total_steps / 90);
        if (t < 8 * E) return hp->lr0 * (double)(1 + t / E);
        double g = 8.0 * hp->lr0;
        if (t >= 30 * E) g *= 0.1;
        if (t >= 60 * E) g *= 0.1;
        return g;
    }
    default:
        return hp->lr0;
    }
}

extern "C" int adpsgd_sched_init(const adpsgd_hparams *hp, adpsgd_state *st) {
    std::string why;
    if (!st) return fail(ADPSGD_EINVAL, "state is NULL");
    if (!hparams_valid(hp, &why)) return fail(ADPSGD_EINVAL, why);
    *st = adpsgd_state{};
    st->p = hp->p_init;
    return ok();
}

extern "C" int adpsgd_sched_step(const adpsgd_hparams *hp, adpsgd_state *st, int32_t *sync_due) {
    if (!hp || !st || !sync_due) return fail(ADPSGD_EINVAL, "NULL hparams, state or output");
    const SchedRule r = rule_of(hp);
    const int64_t t = st->t;
    st->cnt += 1;
    st->p = period_at(r, st->p, t);
    *sync_due = adpsgd::sync_due(r, st->cnt, st->p, t) ? 1 : 0;
    st->t = t + 1;
    return ok();
}

extern "C" int adpsgd_sched_on_sync(const adpsgd_hparams *hp, adpsgd_state *st, int64_t t, double S,
                                    double *margin) {
    if (!hp || !st) return fail(ADPSGD_EINVAL, "NULL hparams or state");
    SchedState s{st->t, st->cnt, st->nC2, st->C2, st->p, 0};
    double m = std::numeric_limits<double>::quiet_NaN();
    const bool finite = apply_sync(rule_of(hp), t, adpsgd_lr(hp, t), S, &s, &m);
    if (margin) *margin = m;
    st->cnt = s.cnt;
    if (!finite) return fail(ADPSGD_ENONFINITE, "variance S is not finite");
    st->nC2 = s.nC2;
    st->C2 = s.C2;
    st->p = s.p;
    return ok();
}
