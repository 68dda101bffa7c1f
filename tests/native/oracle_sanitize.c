/*
 * Test infrastructure: runs every entry point of the CPU oracle on small
 * ragged problems (an empty tensor, K = 1, odd sizes, every period mode,
 * averaged momentum, the warm-up prefix and the period switch) so that a build
 * with AddressSanitizer and UndefinedBehaviorSanitizer can check the oracle's
 * memory accesses and integer arithmetic.  It includes the oracle's source.
 */
#include "../../oracle/adpsgd_oracle.c"

#include <stdio.h>

#define NEW(type, n) ((type *)calloc((size_t)((n) > 0 ? (n) : 1), sizeof(type)))

static int one(int32_t K, const int64_t *off, int32_t T, int32_t mode, int32_t avg_m, int64_t warm,
               int64_t switch_step, int32_t p_after, int64_t steps)
{
    orc_problem pb;
    memset(&pb, 0, sizeof pb);
    pb.K = K;
    pb.T = T;
    pb.P = off[T];
    pb.offsets = off;
    pb.seed = 11;
    pb.sigma = 0.1;
    pb.momentum = 0.9;
    pb.weight_decay = 5e-4;
    pb.h_lo = 1e-2;
    pb.h_hi = 1.0;
    pb.lr_kind = (int32_t)(steps % 4);
    pb.period_mode = mode;
    pb.lr0 = 0.05;
    pb.total_steps = steps;
    pb.k_s = mode == 1 ? steps / 4 : 0;
    pb.thr_lo = 0.7;
    pb.thr_hi = 1.3;
    pb.p_init = 3;
    pb.avg_momentum = avg_m;
    pb.sync_warmup_steps = warm;
    pb.p_switch_step = switch_step;
    pb.p_after = p_after;
    pb.p_max = (mode == 1 && steps % 2) ? 4 : 0;   /* a cap on the adaptive period in some runs */
    const int64_t P = pb.P;

    double *h = NEW(double, P), *xs = NEW(double, P);
    double *x = NEW(double, K * P), *v = NEW(double, K * P);
    orc_problem_data(&pb, NULL, P, h, xs);

    orc_state st;
    orc_state_init(&pb, &st);
    const int64_t cap = 8;   /* smaller than the sync count: the log must stop at cap */
    orc_sync_rec *log = NEW(orc_sync_rec, cap);
    double *var_log = NEW(double, cap * T), *tv = NEW(double, steps), *tg = NEW(double, steps);
    const int64_t n_sync = orc_run(&pb, NULL, P, &st, steps, h, xs, x, v, log, cap, var_log, tv, tg);
    if (n_sync < 0) return 1;

    /* a subset of the elements (every third, ascending), constant modes only */
    if (mode != 1 && P > 0) {
        const int64_t n = (P + 2) / 3;
        int64_t *idx = NEW(int64_t, n);
        for (int64_t j = 0; j < n; ++j) idx[j] = 3 * j;
        double *hs = NEW(double, n), *xss = NEW(double, n), *xsub = NEW(double, K * n), *vsub = NEW(double, K * n);
        orc_problem_data(&pb, idx, n, hs, xss);
        orc_state s2;
        orc_state_init(&pb, &s2);
        if (orc_run(&pb, idx, n, &s2, steps, hs, xss, xsub, vsub, NULL, 0, NULL, NULL, NULL) < 0) return 1;
        double *xbar = NEW(double, n), *vbar = NEW(double, n);
        orc_mean_trajectory(&pb, idx, n, 0, steps, hs, xss, xbar, vbar);
        free(idx); free(hs); free(xss); free(xsub); free(vsub); free(xbar); free(vbar);
    }

    double *var = NEW(double, T);
    (void)orc_variance(&pb, NULL, P, x, var);
    (void)orc_grad_norm2(&pb, P, x, h, xs);
    orc_local_step(&pb, NULL, P, steps, h, xs, x, v);
    (void)orc_average(&pb, NULL, P, x, v, var);

    double *xbar = NEW(double, P), *vbar = NEW(double, P);
    orc_mean_trajectory(&pb, NULL, P, 0, steps, h, xs, xbar, vbar);

    /* the schedule alone on scripted variances, then the controller directly */
    double *S = NEW(double, steps);
    for (int64_t t = 0; t < steps; ++t) S[t] = (double)((t * 7) % 5) * 1e-3;
    int64_t *sync_t = NEW(int64_t, cap);
    int32_t *sync_p = NEW(int32_t, cap);
    orc_state s3;
    orc_state_init(&pb, &s3);
    (void)orc_schedule_trace(&pb, &s3, steps, S, sync_t, sync_p, cap);
    (void)orc_controller(&pb, &s3, steps, 1e-3);
    (void)orc_controller(&pb, &s3, steps, NAN);
    for (int64_t t = 0; t < 3 * steps; ++t) (void)orc_lr(&pb, t);

    free(h); free(xs); free(x); free(v); free(log); free(var_log); free(tv); free(tg);
    free(var); free(xbar); free(vbar); free(S); free(sync_t); free(sync_p);
    printf("ok K=%d P=%lld T=%d mode=%d avg_m=%d syncs=%lld\n", K, (long long)P, T, mode, avg_m, (long long)n_sync);
    return 0;
}

int main(void)
{
    const int64_t ragged[] = {0, 5, 5, 1029, 4000, 4003};   /* an empty tensor, odd sizes */
    const int64_t single[] = {0, 4096};
    const int64_t empty[] = {0, 0, 0};
    for (int32_t mode = 0; mode < 3; ++mode) {
        if (one(3, ragged, 5, mode, mode == 0, 0, 0, 0, 40)) return 1;
        if (one(8, single, 1, mode, 0, 4, mode == 1 ? 0 : 20, 2, 41)) return 1;
        if (one(1, ragged, 5, mode, 1, 0, 0, 0, 13)) return 1;
        if (one(4, empty, 2, mode, 0, 0, 0, 0, 10)) return 1;
    }

    uint32_t out[4], ctr[4] = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu}, key[2] = {1u, 2u};
    double z[4], zz[2];
    orc_philox4x32_10(ctr, key, out);
    orc_normals4(7, 0xffffffffu, 1, 2, 0, z);
    orc_box_muller(0u, 0xffffffffu, zz);   /* the smallest log argument */
    uint32_t *words = NEW(uint32_t, 4 * 64);
    double *normals = NEW(double, 4 * 64);
    orc_philox_groups(5, 1, 2, 0, 0xffffffffu - 63u, 64, words);   /* counter word 0 near 2^32 */
    orc_normals_groups(5, 1, 2, 0, 0, 64, normals);
    free(words);
    free(normals);
    printf("all ok\n");
    return 0;
}
