// Algorithm 2's step counter and period controller as inline functions shared
// by the host controller (adpsgd_sched_step, adpsgd_sched_on_sync) and the
// device reduction kernel, so that a decision taken on the GPU during a run is
// the same fp64 computation, in the same order, as the host's.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "adpsgd.h"

namespace adpsgd {

#define ADPSGD_HD __host__ __device__ __forceinline__

// The hyper-parameters that decide when a sync happens and how p moves.
struct SchedRule {
    int32_t period_mode;     // ADPSGD_PERIOD_*
    int32_t p_after;         // the period from p_switch_step on (constant modes)
    int32_t p_max;           // upper bound on p (>= 1)
    int32_t pad_;
    int64_t k_s;             // syncs after steps t < k_s sample C2
    int64_t warmup;          // steps t < warmup sync every step, with no controller update
    int64_t p_switch_step;   // 0: the period never switches
    double thr_lo, thr_hi;   // the bands of Algorithm 2's period decision
};

// Controller state between steps, as in adpsgd_state: t is the next step, cnt
// the steps since the last sync.  On the device it is written only at syncs,
// so the counter after step t' >= t is cnt + (t' - t) + 1.
struct SchedState {
    int64_t t;
    int64_t cnt;
    int64_t nC2;
    double C2;
    int32_t p;
    int32_t pad_;
};

// The period in force at step t: constant modes may switch to p_after
// (Section III-A's two-phase strategies, Section V-B's decreasing period).
ADPSGD_HD int32_t period_at(const SchedRule &r, int32_t p, int64_t t) {
    return (r.period_mode != ADPSGD_PERIOD_ADAPTIVE && r.p_switch_step > 0 && t >= r.p_switch_step) ? r.p_after
                                                                                                   : p;
}

// Does a sync follow step t?  cnt already counts step t (Algorithm 2, lines
// 5 and 8); p is the period in force.  Warm-up steps always sync; Algorithm
// 1's test is t mod p == 0.
ADPSGD_HD bool sync_due(const SchedRule &r, int64_t cnt, int32_t p, int64_t t) {
    if (t < r.warmup) return true;
    if (r.period_mode == ADPSGD_PERIOD_ALG1) return (t % p) == 0;
    return cnt >= p;
}

// Is the sync after step t one whose outcome may move p?
ADPSGD_HD bool sync_decisive(const SchedRule &r, int64_t t) {
    return r.period_mode == ADPSGD_PERIOD_ADAPTIVE && t >= r.k_s && t >= r.warmup;
}

// Algorithm 2's sampling and period decision after the sync that followed
// step t, with S the summed variance and gamma step t's rate: the counter
// restarts; in the sampling phase (t < K_s) C2 becomes the running mean of
// S / gamma; afterwards p moves by one when S leaves
// [thr_lo gamma C2, thr_hi gamma C2] (p within [1, p_max]).  The sync took
// place whatever S is, so the counter restarts in every case; a non-finite S
// then returns false with C2, nC2 and p untouched.
// margin (may be null): signed relative distance of S to the nearer band edge.
ADPSGD_HD bool apply_sync(const SchedRule &r, int64_t t, double gamma, double S, SchedState *st, double *margin) {
    if (margin) *margin = __builtin_nan("");
    st->cnt = 0;
    if (!__builtin_isfinite(S)) return false;
    if (r.period_mode != ADPSGD_PERIOD_ADAPTIVE || t < r.warmup) return true;
    if (t < r.k_s) {
        st->nC2 += 1;
        st->C2 += (S / gamma - st->C2) / (double)st->nC2;
        return true;
    }
    const double lo = r.thr_lo * gamma * st->C2;
    const double hi = r.thr_hi * gamma * st->C2;
    if (margin && lo > 0) {
        const double m_lo = S / lo - 1.0, m_hi = S / hi - 1.0;
        *margin = __builtin_fabs(m_lo) < __builtin_fabs(m_hi) ? m_lo : m_hi;
    }
    if (S < lo) {
        if (st->p < r.p_max) st->p += 1;
    } else if (S > hi) {
        if (st->p > 1) st->p -= 1;
    }
    return true;
}

#undef ADPSGD_HD

}  // namespace adpsgd
