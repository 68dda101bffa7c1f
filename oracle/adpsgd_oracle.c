/*
 * ORACLE -- test infrastructure, not product code.
 *
 * A plain, slow CPU reference of the ADPSGD hot path (Jiang and Agrawal,
 * "Adaptive Periodic Averaging", arXiv 2007.06134), written from the paper in
 * fp64.  Only the test suite, the smoke check and the bench's CPU-baseline leg
 * may load it.  It shares no code, header, table or helper with the HIP
 * library; the two meet only through the seeded inputs (seed, sizes and
 * hyper-parameters).
 *
 * What it computes, in the paper's order (Algorithm 2, Section III-B):
 *   per step t (the paper's iteration k):
 *     cnt += 1
 *     every worker k takes a local momentum-SGD step on its own replica
 *     if cnt == p:  cnt = 0; average the replicas; S_t = variance of the
 *                   pre-average replicas (Var[.] of Section II-B, per tensor);
 *                   broadcast the average; then either sample C2 (t < K_s) or
 *                   move p by +-1 against the 0.7 / 1.3 thresholds.
 * The paper trains CNNs; here the per-worker gradient is the noisy quadratic
 * stand-in g = h*(x - x*) + sigma*z (the mini-batch gradient of eq. (3) replaced
 * by an exact gradient plus Gaussian noise), with momentum 0.9 (Section IV-A)
 * and coupled weight decay.
 *
 * Readings of points the paper leaves open (each is stated where it is used):
 *   - RunningAverage is the cumulative arithmetic mean of S/gamma over the
 *     sampling-phase syncs.
 *   - The sync test uses Algorithm 2's counter in both period modes; a constant
 *     period is Algorithm 2 without controller updates.
 *   - Momentum buffers are not averaged by default; only the parameters are
 *     (avg_momentum = 1 averages them too, the other reading).
 *   - p never drops below 1 and, when a cap p_max is given, never exceeds it.
 *   - The variance divides by K (not K-1) and sums over parameters.
 *
 * The paper's other strategies, as options of the same loop:
 *   - a warm-up prefix that syncs after every step with no controller update
 *     (the p = 1 warm-up of Sections III-B and IV-C);
 *   - the gradual warm-up learning rate of Section IV-C;
 *   - Algorithm 1's own test, sync when t mod p == 0;
 *   - a constant period that changes at a given step (the two-phase strategies
 *     of Section III-A and the decreasing period of Section V-B).
 *
 * Conventions the paper does not give (noise law and its generator):
 *   Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11), key = (seed low 32 bits,
 *   seed high 32 bits), counter = (float4 group g = i/4, worker k, step t, tag);
 *   tag 0 = gradient noise, 1 = curvature h, 2 = optimum x*.  One call gives the
 *   four values of elements 4g..4g+3.  Uniform U(r) = (r >> 8) * 2^-24; the
 *   Box-Muller log argument is ((r0 >> 8) + 1) * 2^-24 in (0, 1].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_PI 3.14159265358979323846

/* ---- Philox4x32-10, from its published definition (SC'11, Sec. 5) ---------
 * Each round multiplies counter words 0 and 2 by two fixed odd constants,
 * takes the 64-bit products, and mixes:
 *   out0 = hi(M1*c2) ^ c1 ^ k0,  out1 = lo(M1*c2),
 *   out2 = hi(M0*c0) ^ c3 ^ k1,  out3 = lo(M0*c0);
 * the key is bumped by the Weyl constants between rounds. */
static const uint32_t PH_M0 = 0xD2511F53u, PH_M1 = 0xCD9E8D57u;
static const uint32_t PH_W0 = 0x9E3779B9u, PH_W1 = 0xBB67AE85u;

void orc_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)PH_M0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)PH_M1 * (uint64_t)c2;
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        uint32_t n3 = (uint32_t)p0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += PH_W0;
        k1 += PH_W1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static void philox_seeded(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                          uint32_t out[4])
{
    uint32_t ctr[4] = {c0, c1, c2, c3};
    uint32_t key[2] = {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)};
    orc_philox4x32_10(ctr, key, out);
}

/* Uniform in [0,1) from the top 24 bits. */
static double unif24(uint32_t r) { return (double)(r >> 8) * (1.0 / 16777216.0); }

/* Box-Muller (1958): two uniforms -> two independent N(0,1). */
static void box_muller(uint32_t ra, uint32_t rb, double *z0, double *z1)
{
    double u1 = ((double)(ra >> 8) + 1.0) * (1.0 / 16777216.0);   /* (0, 1] */
    double u2 = unif24(rb);                                      /* [0, 1) */
    double radius = sqrt(-2.0 * log(u1));
    *z0 = radius * cos(2.0 * ORC_PI * u2);
    *z1 = radius * sin(2.0 * ORC_PI * u2);
}

void orc_normals4(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, double z[4])
{
    uint32_t r[4];
    philox_seeded(seed, c0, c1, c2, c3, r);
    box_muller(r[0], r[1], &z[0], &z[1]);
    box_muller(r[2], r[3], &z[2], &z[3]);
}

/* Raw Box-Muller pair of two 32-bit words (exposed for special-case checks). */
void orc_box_muller(uint32_t ra, uint32_t rb, double z[2])
{
    box_muller(ra, rb, &z[0], &z[1]);
}

/* Generator dumps over consecutive groups g0 .. g0+n-1 with counter words
 * (g, c1, c2, c3): raw words out[4n] and the matching normals z[4n]. */
void orc_philox_groups(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3,
                       int64_t g0, int64_t n, uint32_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j)
        philox_seeded(seed, (uint32_t)(g0 + j), c1, c2, c3, out + 4 * j);
}

void orc_normals_groups(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3,
                        int64_t g0, int64_t n, double *z)
{
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j)
        orc_normals4(seed, (uint32_t)(g0 + j), c1, c2, c3, z + 4 * j);
}

/* ---- problem description ------------------------------------------------ */
typedef struct {
    int32_t K;                 /* workers (the paper's n) */
    int32_t T;                 /* tensors */
    int64_t P;                 /* parameters per replica */
    const int64_t *offsets;    /* [T+1], offsets[0] = 0, offsets[T] = P */
    uint64_t seed;
    double sigma, momentum, weight_decay, h_lo, h_hi;
    int32_t lr_kind;           /* 0 constant, 1 step decay, 2 cosine, 3 gradual warm-up + steps */
    int32_t period_mode;       /* 0 constant period, 1 adaptive (Algorithm 2),
                                  2 constant period with Algorithm 1's test (k mod p == 0) */
    double lr0;
    int64_t total_steps;
    int64_t k_s;
    double thr_lo, thr_hi;
    int32_t p_init;
    int32_t avg_momentum;      /* 1: a sync averages the momentum buffers too */
    int64_t sync_warmup_steps; /* steps before this one sync every step, no controller */
    int64_t p_switch_step;     /* constant modes: period p_after from this step on (0: never) */
    int32_t p_after;
    int32_t p_max;             /* upper bound on the adaptive period; 0: none */
} orc_problem;

typedef struct {
    int64_t t;       /* next step index */
    int64_t cnt;     /* steps since the last sync */
    int64_t nC2;     /* syncs folded into C2 */
    double C2;
    int32_t p;
    int32_t pad_;
} orc_state;

typedef struct {
    int64_t t;       /* step after which the sync happened */
    int32_t p;       /* period in force for that sync */
    int32_t pad_;
    double S;        /* sum over tensors of the per-tensor variance */
    double C2;       /* C2 after this sync's update */
    double gamma;    /* learning rate of step t */
} orc_sync_rec;

/* Learning rate of 0-based step t.  Step decay: x0.1 at floor(N/2) and again
 * at floor(3N/4) (the paper decays by 10x at 1/2 and 3/4 of training,
 * Section IV-B); cosine: lr0 * (1 + cos(pi t / N)) / 2.  Gradual warm-up
 * (Section IV-C: 90 epochs; the rate starts at lr0 and grows by lr0 each epoch
 * for 8 epochs, stays at 8 lr0, and is cut by 10x at epochs 30 and 60), with
 * an epoch of E = floor(N / 90) steps (at least one). */
double orc_lr(const orc_problem *pb, int64_t t)
{
    double N = (double)pb->total_steps;
    switch (pb->lr_kind) {
    case 1: {
        double g = pb->lr0;
        if (t >= pb->total_steps / 2) g *= 0.1;
        if (t >= (3 * pb->total_steps) / 4) g *= 0.1;
        return g;
    }
    case 2:
        return pb->lr0 * 0.5 * (1.0 + cos(ORC_PI * (double)t / N));
    case 3: {
        int64_t E = pb->total_steps / 90;
        if (E < 1) E = 1;
        int64_t epoch = t / E;
        if (epoch < 8) return pb->lr0 * (double)(epoch + 1);
        double g = 8.0 * pb->lr0;
        if (epoch >= 30) g *= 0.1;
        if (epoch >= 60) g *= 0.1;
        return g;
    }
    default:
        return pb->lr0;
    }
}

/* Curvature and optimum of element i: h = exp(ln lo + u (ln hi - ln lo)),
 * u uniform (tag 1); x* ~ N(0,1) (tag 2). */
void orc_problem_data(const orc_problem *pb, const int64_t *idx, int64_t n, double *h, double *xs)
{
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        int64_t i = idx ? idx[j] : j;
        uint32_t g = (uint32_t)(i / 4);
        int lane = (int)(i % 4);
        uint32_t r[4];
        philox_seeded(pb->seed, g, 0, 0, 1, r);
        double u = unif24(r[lane]);
        h[j] = exp(log(pb->h_lo) + u * (log(pb->h_hi) - log(pb->h_lo)));
        double z[4];
        orc_normals4(pb->seed, g, 0, 0, 2, z);
        xs[j] = z[lane];
    }
}

/* One local step t on every worker (Algorithm 2's update, with heavy-ball
 * momentum as in PyTorch SGD: d = g + wd*x; v = mu*v + d; x = x - gamma*v).
 * x and v are [K][n] over the selected elements idx[0..n) (all if idx NULL). */
void orc_local_step(const orc_problem *pb, const int64_t *idx, int64_t n, int64_t t,
                    const double *h, const double *xs, double *x, double *v)
{
    double gamma = orc_lr(pb, t);
    for (int32_t k = 0; k < pb->K; ++k) {
        double *xk = x + (int64_t)k * n;
        double *vk = v + (int64_t)k * n;
#pragma omp parallel
        {
            /* one generator call serves the four elements of a group: keep the
             * last group's normals (same values as noise(), computed once) */
            int64_t g_memo = -1;
            double z4[4] = {0, 0, 0, 0};
#pragma omp for schedule(static)
            for (int64_t j = 0; j < n; ++j) {
                int64_t i = idx ? idx[j] : j;
                if (i / 4 != g_memo) {
                    g_memo = i / 4;
                    orc_normals4(pb->seed, (uint32_t)g_memo, (uint32_t)k, (uint32_t)t, 0, z4);
                }
                double z = z4[i % 4];
                double g = h[j] * (xk[j] - xs[j]) + pb->sigma * z;
                double d = g + pb->weight_decay * xk[j];
                vk[j] = pb->momentum * vk[j] + d;
                xk[j] = xk[j] - gamma * vk[j];
            }
        }
    }
}

/* Element range [jb, je) of tensor tau within the ascending selection idx. */
static void tensor_range(const orc_problem *pb, const int64_t *idx, int64_t n, int32_t tau,
                         int64_t *jb, int64_t *je)
{
    if (!idx) { *jb = pb->offsets[tau]; *je = pb->offsets[tau + 1]; return; }
    int64_t lo = 0, hi = n;                 /* first j with idx[j] >= offsets[tau] */
    while (lo < hi) { int64_t m = (lo + hi) / 2; if (idx[m] < pb->offsets[tau]) lo = m + 1; else hi = m; }
    *jb = lo;
    hi = n;                                 /* first j with idx[j] >= offsets[tau+1] */
    while (lo < hi) { int64_t m = (lo + hi) / 2; if (idx[m] < pb->offsets[tau + 1]) lo = m + 1; else hi = m; }
    *je = lo;
}

/* The synchronization step of Algorithm 2 (average, then broadcast):
 *   xbar_i  = (1/K) sum_k x_{k,i}
 *   var_tau = (1/K) sum_k sum_{i in tau} (xbar_i - x_{k,i})^2      (pre-average x)
 *   x_{k,i} = xbar_i for every k; momentum untouched unless avg_momentum, in
 *   which case v_{k,i} = (1/K) sum_j v_{j,i} as well (v may then not be NULL).
 * S = sum_tau var_tau is the paper's S_k (Var[.] of Section II-B with the squared
 * norm).  Returns S; var_out[T] receives the per-tensor terms. */
double orc_average(const orc_problem *pb, const int64_t *idx, int64_t n, double *x, double *v,
                   double *var_out)
{
    if (pb->avg_momentum && v) {
#pragma omp parallel for schedule(static)
        for (int64_t j = 0; j < n; ++j) {
            double s = 0.0;
            for (int32_t k = 0; k < pb->K; ++k) s += v[(int64_t)k * n + j];
            double vbar = s / (double)pb->K;
            for (int32_t k = 0; k < pb->K; ++k) v[(int64_t)k * n + j] = vbar;
        }
    }
    const int32_t K = pb->K;
    double *xbar = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        double s = 0.0;
        for (int32_t k = 0; k < K; ++k) s += x[(int64_t)k * n + j];
        xbar[j] = s / (double)K;
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t tau = 0; tau < pb->T; ++tau) {
        int64_t jb, je;
        tensor_range(pb, idx, n, tau, &jb, &je);
        double acc = 0.0;
        for (int32_t k = 0; k < K; ++k)
            for (int64_t j = jb; j < je; ++j) {
                double dev = xbar[j] - x[(int64_t)k * n + j];
                acc += dev * dev;
            }
        var_out[tau] = acc / (double)K;
    }
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j)
        for (int32_t k = 0; k < K; ++k) x[(int64_t)k * n + j] = xbar[j];
    free(xbar);
    double S = 0.0;
    for (int32_t tau = 0; tau < pb->T; ++tau) S += var_out[tau];
    return S;
}

/* The inter-worker variance of the current replicas without averaging them:
 * var_tau = (1/K) sum_k sum_{i in tau} (xbar_i - x_{k,i})^2, and their sum
 * Var[W] of Section II-B (returned). */
double orc_variance(const orc_problem *pb, const int64_t *idx, int64_t n, const double *x, double *var_out)
{
    const int32_t K = pb->K;
    double *xbar = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    for (int64_t j = 0; j < n; ++j) {
        double s = 0.0;
        for (int32_t k = 0; k < K; ++k) s += x[(int64_t)k * n + j];
        xbar[j] = s / (double)K;
    }
    double S = 0.0;
    for (int32_t tau = 0; tau < pb->T; ++tau) {
        int64_t jb, je;
        tensor_range(pb, idx, n, tau, &jb, &je);
        double acc = 0.0;
        for (int32_t k = 0; k < K; ++k)
            for (int64_t j = jb; j < je; ++j) {
                double dev = xbar[j] - x[(int64_t)k * n + j];
                acc += dev * dev;
            }
        var_out[tau] = acc / (double)K;
        S += var_out[tau];
    }
    free(xbar);
    return S;
}

/* |grad F(xbar)|^2 at the replica mean, F(x) = 1/2 sum h (x - x*)^2 + wd/2 |x|^2:
 * the gradient norm whose gamma-weighted average over iterations is the
 * convergence metric of eq. (metric1). */
double orc_grad_norm2(const orc_problem *pb, int64_t n, const double *x, const double *h, const double *xs)
{
    double acc = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        double s = 0.0;
        for (int32_t k = 0; k < pb->K; ++k) s += x[(int64_t)k * n + j];
        double xbar = s / (double)pb->K;
        double g = h[j] * (xbar - xs[j]) + pb->weight_decay * xbar;
        acc += g * g;
    }
    return acc;
}

/* Period controller after a sync at step t with variance S (Algorithm 2's
 * sampling and period decision).  Inactive in the constant modes and during the warm-up prefix
 * (there the run synchronizes every step and Algorithm 2 has not started).
 * The period stays within [1, p_max]: the decrease could reach 0, and the paper
 * gives no upper bound, so one is an option (p_max = 0: none).
 * Returns 0, or -4 if S is not finite (state unchanged). */
int orc_controller(const orc_problem *pb, orc_state *st, int64_t t, double S)
{
    if (!isfinite(S)) return -4;
    if (pb->period_mode != 1 || t < pb->sync_warmup_steps) return 0;
    double gamma = orc_lr(pb, t);
    if (t < pb->k_s) {
        /* sampling phase: running (cumulative) mean of S / gamma */
        st->nC2 += 1;
        st->C2 += (S / gamma - st->C2) / (double)st->nC2;
    } else if (S < pb->thr_lo * gamma * st->C2) {
        if (pb->p_max <= 0 || st->p < pb->p_max) st->p += 1;
    } else if (S > pb->thr_hi * gamma * st->C2) {
        if (st->p > 1) st->p -= 1;
    }
    return 0;
}

void orc_state_init(const orc_problem *pb, orc_state *st)
{
    memset(st, 0, sizeof(*st));
    st->p = pb->p_init;
}

/* Start of step t: count it (Algorithm 2's counter), apply the two-phase
 * constant period (Section III-A strategies, Section V-B), and say whether a
 * sync follows it: every step of the p = 1 warm-up prefix (Sections III-B,
 * IV-C); t mod p == 0 under Algorithm 1's test; cnt == p under Algorithm 2's
 * (written >= so a period that shrinks under the counter still ends). */
static int begin_step(const orc_problem *pb, orc_state *st, int64_t t)
{
    st->cnt += 1;
    if (pb->period_mode != 1 && pb->p_switch_step > 0 && t >= pb->p_switch_step) st->p = pb->p_after;
    if (t < pb->sync_warmup_steps) return 1;
    if (pb->period_mode == 2) return (t % st->p) == 0;
    return st->cnt >= st->p;
}

/* The schedule alone, driven by scripted variances: S_by_step[t] is taken as
 * the variance of a sync after step t.  Records the sync steps and the period
 * in force for each (up to cap); returns the sync count or -4 on a non-finite S. */
int64_t orc_schedule_trace(const orc_problem *pb, orc_state *st, int64_t n_steps,
                           const double *S_by_step, int64_t *sync_t, int32_t *sync_p, int64_t cap)
{
    int64_t n_sync = 0;
    for (int64_t s = 0; s < n_steps; ++s) {
        int64_t t = st->t;
        int sync = begin_step(pb, st, t);
        st->t = t + 1;
        if (!sync) continue;
        st->cnt = 0;
        if (n_sync < cap) { sync_t[n_sync] = t; sync_p[n_sync] = st->p; }
        n_sync += 1;
        int rc = orc_controller(pb, st, t, S_by_step[t]);
        if (rc) return rc;
    }
    return n_sync;
}

/* Run steps st->t .. st->t + n_steps - 1 of Algorithm 2 on the selection idx
 * (idx NULL: all P elements; a strict subset is allowed only with a constant
 * period, where the sync schedule does not depend on the data).
 * x, v: [K][n], updated in place.  Each sync appends a record to log (up to
 * log_cap) and its per-tensor variances to var_log[cap][T] (if non-NULL).
 * If trace_var / trace_gn are given ([n_steps] each), every step records the
 * variance of the replicas after it, before any sync (Var[W_{t+1}]), and
 * |grad F|^2 at their mean.  Returns the number of syncs, or a negative error. */
int64_t orc_run(const orc_problem *pb, const int64_t *idx, int64_t n, orc_state *st,
                int64_t n_steps, const double *h, const double *xs, double *x, double *v,
                orc_sync_rec *log, int64_t log_cap, double *var_log, double *trace_var, double *trace_gn)
{
    if (idx && n != pb->P && pb->period_mode == 1) return -1;
    double *var = (double *)malloc((size_t)pb->T * sizeof(double));
    int64_t n_sync = 0;
    for (int64_t s = 0; s < n_steps; ++s) {
        int64_t t = st->t;
        int sync = begin_step(pb, st, t);
        orc_local_step(pb, idx, n, t, h, xs, x, v);
        if (trace_var) trace_var[s] = orc_variance(pb, idx, n, x, var);
        if (trace_gn) trace_gn[s] = orc_grad_norm2(pb, n, x, h, xs);
        if (sync) {
            st->cnt = 0;
            double S = orc_average(pb, idx, n, x, v, var);
            int32_t p_used = st->p;
            int rc = orc_controller(pb, st, t, S);
            if (n_sync < log_cap) {
                if (log) {
                    log[n_sync].t = t; log[n_sync].p = p_used;
                    log[n_sync].S = S; log[n_sync].C2 = st->C2; log[n_sync].gamma = orc_lr(pb, t);
                }
                if (var_log) memcpy(var_log + n_sync * pb->T, var, (size_t)pb->T * sizeof(double));
            }
            n_sync += 1;
            if (rc) { st->t = t + 1; free(var); return rc; }
        }
        st->t = t + 1;
    }
    free(var);
    return n_sync;
}

/* The replica mean under any sync schedule.  Syncs replace each x_k by the mean
 * and leave v alone (or replace it by its mean), so they preserve both means;
 * the dynamics are affine in
 * (x, v), so the means follow one momentum-SGD run driven by the K-averaged
 * noise: zbar = (1/K) sum_k z_k.  xbar, vbar: [n], updated in place. */
void orc_mean_trajectory(const orc_problem *pb, const int64_t *idx, int64_t n, int64_t t0,
                         int64_t n_steps, const double *h, const double *xs,
                         double *xbar, double *vbar)
{
    double *zsum = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    for (int64_t t = t0; t < t0 + n_steps; ++t) {
        double gamma = orc_lr(pb, t);
        for (int64_t j = 0; j < n; ++j) zsum[j] = 0.0;
        for (int32_t k = 0; k < pb->K; ++k) {
#pragma omp parallel
            {
                int64_t g_memo = -1;              /* one generator call per group */
                double z4[4] = {0, 0, 0, 0};
#pragma omp for schedule(static)
                for (int64_t j = 0; j < n; ++j) {
                    int64_t i = idx ? idx[j] : j;
                    if (i / 4 != g_memo) {
                        g_memo = i / 4;
                        orc_normals4(pb->seed, (uint32_t)g_memo, (uint32_t)k, (uint32_t)t, 0, z4);
                    }
                    zsum[j] += z4[i % 4];
                }
            }
        }
#pragma omp parallel for schedule(static)
        for (int64_t j = 0; j < n; ++j) {
            double zbar = zsum[j] / (double)pb->K;
            double g = h[j] * (xbar[j] - xs[j]) + pb->sigma * zbar;
            double d = g + pb->weight_decay * xbar[j];
            vbar[j] = pb->momentum * vbar[j] + d;
            xbar[j] = xbar[j] - gamma * vbar[j];
        }
    }
    free(zsum);
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
