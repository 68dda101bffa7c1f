/*
 * adpsgd.h -- C ABI of the MI355X (gfx950) ADPSGD hot path.
 *
 * ADPSGD is adaptive periodic parameter averaging SGD (Jiang and Agrawal,
 * arXiv 2007.06134, Algorithm 2).  K simulated workers keep stacked fp32
 * parameter replicas x[K][P] and momentum buffers m[K][P] in one GPU's HBM.
 * Each local step applies momentum SGD to every replica with a noisy diagonal
 * quadratic gradient; every p steps the replicas are averaged, the
 * inter-worker parameter variance is reduced per tensor, and the period
 * controller moves p to keep that variance near gamma * C2.  During a run the
 * controller's decisions are taken on the device (so the GPU never waits for
 * the host) and replayed and checked on the host; the same controller is
 * callable on the host alone (adpsgd_sched_*).
 *
 * Conventions shared by every call:
 *   - Every call returns an int status: ADPSGD_OK (0) or a negative code below.
 *     adpsgd_last_error() gives a message for the calling thread's last error.
 *   - Arguments are validated before anything is enqueued; on a validation
 *     error nothing runs and the context is unchanged.
 *   - Device buffers are caller-owned (the library never allocates or frees
 *     them).  Host arrays are read during the call and never retained, except
 *     where stated.
 *   - Calls on a context make its device (the one current at adpsgd_init)
 *     current while they run and restore the caller's device afterwards.
 *   - One context is used by one host thread at a time.  A context pointer that
 *     adpsgd_init did not return, or that was destroyed, is refused with
 *     ADPSGD_EINVAL (so is a second adpsgd_destroy).
 *   - The entry points are bracketed by roctx ranges (rocprofv3 --marker-trace).
 *   - Step indices t are 0-based: step t is the paper's iteration k = t.
 *
 * Readings of points the paper leaves open, used throughout:
 *   - The sync follows Algorithm 2's counter in both period modes: syncs
 *     happen after 0-based steps p-1, 2p-1, ... (a constant period is
 *     Algorithm 2 with no controller updates).
 *   - Momentum buffers stay local; only parameters are averaged (unless
 *     avg_momentum is set).
 *   - RunningAverage(C2, S/gamma) is the cumulative mean over sampling syncs.
 *   - p stays within [1, p_max].
 *   - Variance: (1/K) sum_k sum_{i in tensor} (xbar_i - x_{k,i})^2, taken on
 *     the replicas just before they are replaced by their mean.
 */
#ifndef ADPSGD_H
#define ADPSGD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Only the functions below are exported from the shared library. */
#define ADPSGD_API __attribute__((visibility("default")))

/* ---- status codes ---------------------------------------------------------- */
#define ADPSGD_OK 0
#define ADPSGD_EINVAL (-1)     /* invalid argument; nothing was enqueued           */
#define ADPSGD_ESTATE (-2)     /* call not valid in the context's current state    */
#define ADPSGD_EDEVICE (-3)    /* a HIP runtime call failed (see adpsgd_last_error) */
#define ADPSGD_ENONFINITE (-4) /* the variance S was NaN or infinite; p, C2 kept  */

/* ---- learning-rate schedules: gamma_t for 0-based step t ------------------- */
#define ADPSGD_LR_CONST 0  /* gamma_t = lr0                                             */
#define ADPSGD_LR_STEP 1   /* lr0 * 0.1 from t = floor(N/2), * 0.01 from floor(3N/4);
                              the paper's 10x decays at 1/2 and 3/4 of training (Sec. IV-B) */
#define ADPSGD_LR_COSINE 2 /* lr0 * (1 + cos(pi t / N)) / 2                              */
#define ADPSGD_LR_WARMUP_STEP 3 /* gradual warm-up then step decay (Sec. IV-C): with
                              E = floor(N / 90) steps per "epoch", lr0 * (1 + floor(t / E))
                              for t < 8 E (0.1 -> 0.8 for lr0 = 0.1), then 8 lr0, x0.1 from
                              t = 30 E, x0.01 from t = 60 E                               */

/* ---- period modes ----------------------------------------------------------- */
#define ADPSGD_PERIOD_CONST 0    /* CPSGD, Algorithm 1: p = p_init throughout            */
#define ADPSGD_PERIOD_ADAPTIVE 1 /* ADPSGD, Algorithm 2: C2 sampling, then p +- 1        */
#define ADPSGD_PERIOD_ALG1 2     /* CPSGD with Algorithm 1's test: sync after every step t
                                    with t mod p == 0 (after steps 0, p, 2p, ...)           */

/* ---- launch policies of adpsgd_run (adpsgd_set_launch_policy) ----------------- */
#define ADPSGD_LAUNCH_HYBRID 0  /* default: steps the host can plan run as plain steps or
                                   fused syncs; after a decisive sync the host waits for
                                   its outcome while the GPU has queued work, else the
                                   device decides the next steps itself.  A run in a
                                   constant-period mode on a problem of K * P < 2^24
                                   (launch-bound) and up to 65536 steps, with timing off,
                                   is captured once as a HIP graph of the same launches and
                                   replayed while runs repeat with the same start state,
                                   length and step launch shape                            */
#define ADPSGD_LAUNCH_DEVICE 1  /* every step is decided on the device (step + optional
                                   sync + reduction per step)                              */
#define ADPSGD_LAUNCH_HOST 2    /* the host waits for every decision it needs; the device
                                   only confirms syncs the host planned                    */

typedef struct adpsgd_ctx adpsgd_ctx; /* opaque, owned by the library */

/* Hyper-parameters (Algorithm 2's Require line: p_init, K_s; Section IV-A:
 * momentum; the noisy quadratic stand-in for the mini-batch gradient of
 * eq. (3): g_k = h * (x_k - x*) + sigma * z_k, z_k ~ N(0,1) from Philox4x32-10
 * keyed by seed with counter (i/4, k, t, 0); h ~ LogUniform[h_lo, h_hi]
 * (counter tag 1) and x* ~ N(0,1) (tag 2) per element). */
typedef struct {
    uint64_t seed;
    double sigma;        /* noise standard deviation, >= 0                       */
    double momentum;     /* heavy-ball coefficient, in [0, 1)                     */
    double weight_decay; /* coupled L2: d = g + weight_decay * x, >= 0            */
    double h_lo, h_hi;   /* curvature range, 0 < h_lo <= h_hi                     */
    int32_t lr_kind;     /* ADPSGD_LR_*                                           */
    int32_t period_mode; /* ADPSGD_PERIOD_*                                       */
    double lr0;          /* base learning rate, > 0                               */
    int64_t total_steps; /* N: the schedule's length (step decay / cosine), >= 1  */
    int32_t p_init;      /* initial (or constant) averaging period, >= 1          */
    int32_t p_max;       /* upper bound on p; 0 means INT32_MAX                   */
    int64_t k_s;         /* syncs after steps t < k_s sample C2 (Algorithm 2)     */
    double thr_lo;       /* p += 1 if S < thr_lo * gamma_t * C2 (paper: 0.7)      */
    double thr_hi;       /* p -= 1 if S > thr_hi * gamma_t * C2 (paper: 1.3)      */
    int64_t sync_warmup_steps; /* steps t < this sync after every step with no controller
                                  update (the paper's p = 1 warm-up, Sec. III-B, IV-C);
                                  Algorithm 2 then starts with cnt = 0, p = p_init; 0 = none */
    int64_t p_switch_step;     /* constant mode: from step p_switch_step on, the period is
                                  p_after (Sec. III-A strategies, the decreasing-period
                                  baseline of Sec. V-B); 0 = never                           */
    int32_t p_after;           /* the period after p_switch_step, >= 1 when used            */
    int32_t avg_momentum;      /* 1: a sync also replaces every momentum buffer by the mean
                                  of the K buffers; 0: momentum stays local (default)        */
} adpsgd_hparams;

/* Caller-owned device memory, on the device current at adpsgd_init. */
typedef struct {
    float *x;               /* [K][P] replicas, row-major (rows row_stride apart), 16-byte
                               aligned; rows zeroed by init                                 */
    float *m;               /* [K][P] momentum buffers, same layout; rows zeroed by init     */
    float *h;               /* [P] curvatures, written by init                               */
    float *xstar;           /* [P] optimum, written by init                                  */
    void *workspace;        /* >= adpsgd_workspace_bytes(...) bytes, 256-byte aligned;
                               tile, chunk and window tables, partial sums and the device
                               copy of the controller state (the records of the reductions
                               go to pinned host memory that the library allocates)          */
    size_t workspace_bytes;
    void *stream;           /* hipStream_t for every launch and copy; NULL = null stream     */
    int64_t row_stride;     /* elements from one row of x (and of m) to the next, >= P;
                               0 means P.  A multiple of 4 keeps every row 16-byte aligned,
                               so whole float4 groups move with vector accesses when P is
                               not a multiple of 4 (about 2x faster than P rows packed back
                               to back); a multiple of 256 also starts every row on a 1 KB
                               boundary, so a wave's 1 KB of a row is one aligned kilobyte.
                               adpsgd_padded_row_stride gives the stride to use with the
                               single-allocation layout described there.
                               The library never touches the padding.                       */
} adpsgd_buffers;

/* The row stride (in floats) for P parameters that the fastest buffer layout
 * uses: the least 256 n >= P with n odd (0 for P <= 0).  The layout is one
 * allocation of 2K + 2 rows of that stride holding the K rows of x, then the
 * K rows of m, then h and xstar as rows 2K and 2K + 1.  Every kernel streams
 * all of those rows at the same element offset at once, and how far apart
 * they start decides how fast (through how HBM addresses interleave over
 * channels, presumably): measured on MI355X at K = 8, P = 138M, this layout
 * runs the local step 1% and the fused step + sync 2.5% faster than x, m, h
 * and xstar in separate allocations, and the fused step + sync up to 10%
 * faster than rows an even number of kilobytes apart. */
ADPSGD_API int64_t adpsgd_padded_row_stride(int64_t P);

/* Controller state on the host (Algorithm 2's inputs and counters).  x and m
 * are the device part of the state and stay in the caller's buffers. */
typedef struct {
    int64_t t;       /* next step index                          */
    int64_t cnt;     /* steps since the last sync (Alg. 2 cnt)   */
    int64_t nC2;     /* sampling syncs folded into C2            */
    double C2;       /* sampled constant C2                      */
    int32_t p;       /* current averaging period                 */
    int32_t reserved;
} adpsgd_state;

/* One record per synchronization. */
typedef struct {
    int64_t t;       /* the sync followed step t                               */
    int32_t p;       /* period in force for this sync                          */
    int32_t reserved;
    double S;        /* sum over tensors of the per-tensor variance (S_k)      */
    double C2;       /* C2 after this sync                                     */
    double gamma;    /* learning rate of step t                                */
    double margin;   /* signed relative distance of S to the nearer threshold,
                        S / (thr * gamma * C2) - 1; NaN when no decision made  */
} adpsgd_sync_rec;

/* One record per local step of a traced run. */
typedef struct {
    int64_t t;          /* the step                                                   */
    int32_t synced;     /* 1 if a sync followed it                                    */
    int32_t p;          /* period in force                                            */
    double var;         /* inter-worker parameter variance after step t and before any
                           sync: sum over tensors of (1/K) sum_k |x_k - xbar|^2, i.e.
                           Var[W_{t+1}] of Sec. II-B (equal to S at a sync step)      */
    double grad_norm2;  /* |grad F(xbar)|^2 at the replica mean after step t, with
                           F(x) = 1/2 sum h (x - x*)^2 + wd/2 |x|^2: the quantity whose
                           gamma-weighted average is the convergence metric of
                           eq. (metric1)                                              */
    double gamma;       /* learning rate of step t                                    */
} adpsgd_step_rec;

/* Per-kernel device time, from HIP events around the sampled launches. */
typedef struct {
    double step_ms;     int64_t step_launches;     /* plain local step            */
    double fused_ms;    int64_t fused_launches;    /* last step of a period + sync */
    double average_ms;  int64_t average_launches;  /* separate mean/broadcast/var */
    double segsum_ms;   int64_t segsum_launches;   /* reduction: per-tensor sums and,
                                                      in a run, the period decision */
    double trace_ms;    int64_t trace_launches;    /* traced plain step (step + variance) */
    int64_t graph_captures;  /* runs captured as a HIP graph (ADPSGD_LAUNCH_HYBRID), and */
    int64_t graph_replays;   /* runs replayed from one; counted whether timing is on or off */
} adpsgd_timing;

/* Bytes of device workspace for K workers, P parameters and T tensors with
 * boundaries offsets[0..T] (host).  Returns 0 if the arguments are invalid. */
ADPSGD_API size_t adpsgd_workspace_bytes(int32_t K, int64_t P, int32_t T, const int64_t *offsets);

/* Create a context (Algorithm 2's initial state, and w_{0,i} = w_0 = 0).
 * K >= 1 workers; P >= 0 parameters; T >= 1 tensors with host offsets[T+1],
 * non-decreasing, offsets[0] = 0, offsets[T] = P (empty tensors allowed).
 * Fills h and xstar from the seed, zeroes x and m, and waits for the stream.
 * With K * P >= 2^24 it first times, on those buffers, the local step's launch
 * shapes (adpsgd_set_step_launch), the separate sync with and without an
 * occupancy cap and, where x and m take 256 MB to 1 GiB, the syncs with cached
 * and with non-temporal accesses, and keeps the fastest of each (the results
 * are the same bits whichever wins).
 * P/4 and the step count must stay below 2^32 (Philox counter words).  Any
 * K * P that fits the device is accepted: a kernel grid beyond what one
 * dispatch holds (2^32 work-items) is issued as several launches. */
ADPSGD_API int adpsgd_init(int32_t K, int64_t P, const int64_t *tensor_offsets, int32_t T,
                const adpsgd_hparams *hp, const adpsgd_buffers *buf, adpsgd_ctx **out);

/* Zero x and m and reset the controller state to t = 0, cnt = 0, p = p_init,
 * C2 = 0.  h and xstar are kept.  Asynchronous. */
ADPSGD_API int adpsgd_reset(adpsgd_ctx *c);

/* Enqueue n >= 0 plain local steps t .. t+n-1 on every worker (Algorithm 2's
 * update): d = h (x - x*) + sigma z + wd x; m = mu m + d; x = x - gamma_t m.
 * Advances t and cnt by n; a constant period that switches at p_switch_step
 * (hparams) becomes p_after in the state once a step t >= p_switch_step is
 * taken, as in adpsgd_sched_step.  Asynchronous. */
ADPSGD_API int adpsgd_local_steps(adpsgd_ctx *c, int32_t n);

/* Synchronize now (Algorithm 2's sync): xbar = mean of the K replicas,
 * var_out[tau] = (1/K) sum_k sum_{i in tau} (xbar_i - x_{k,i})^2 (host, [T],
 * fp64), every replica set to xbar, momentum untouched, cnt = 0.  Blocks until
 * var_out is valid. */
ADPSGD_API int adpsgd_average(adpsgd_ctx *c, double *var_out);

/* One local step followed by the synchronization, in a single pass over x and
 * m (same results and state as adpsgd_local_steps(c, 1) then adpsgd_average).
 * Blocks. */
ADPSGD_API int adpsgd_step_average(adpsgd_ctx *c, double *var_out);

/* Period controller (Algorithm 2's sampling and period decision) for a sync
 * after step t - 1 with S = sum(var[0..T)), as adpsgd_sched_on_sync.
 * Sampling phase (t-1 < k_s): C2 <- running mean of S / gamma; otherwise
 * p + 1 if S < thr_lo gamma C2, p - 1 if S > thr_hi gamma C2.  Constant mode and the warm-up prefix: no
 * change.  *next_period (may be NULL) receives p.  ENONFINITE if S is NaN or
 * infinite: the counter still restarts (the sync took place), while p, C2 and
 * nC2 are unchanged. */
ADPSGD_API int adpsgd_schedule(adpsgd_ctx *c, const double *var, int32_t *next_period);

/* Run n_steps steps of Algorithm 2 from the current state: local steps, a sync
 * whenever adpsgd_sched_step says one is due (fused into that step), and the
 * controller after every sync.  Syncs whose outcome the host has not read back
 * are decided on the device by the same rules in the same fp64 arithmetic, so
 * the GPU does not wait for the host; the host replays every step and returns
 * ESTATE if a device decision ever differs from its own.  log (host, log_cap
 * records) and var_log (host, [log_cap][T], may be NULL) receive the first
 * log_cap syncs; *n_syncs (may be NULL) the count of all syncs.  No sync is
 * forced at the end.  Returns when all enqueued work has finished.  On
 * ENONFINITE the run stops at that sync, whose update of p and C2 is withheld
 * (its counter restarts, as at every sync); steps already enqueued after it
 * complete (with their syncs, logged) and are counted in the state (a run
 * replayed as a graph has enqueued all its steps).  The graph of a
 * constant-period run (ADPSGD_LAUNCH_HYBRID) is captured on a stream of the
 * library's own and launched on the context's stream; it holds pinned record
 * slots, one per sync, until the context is destroyed. */
ADPSGD_API int adpsgd_run(adpsgd_ctx *c, int64_t n_steps, adpsgd_sync_rec *log, int64_t log_cap,
               double *var_log, int64_t *n_syncs);

/* adpsgd_run that also records every step in trace[0 .. trace_cap) (host):
 * plain steps run as a step that also reduces the variance and the gradient
 * norm at the mean without averaging (the same HBM traffic as a plain step),
 * sync steps as the fused step + sync that also reports the gradient norm.
 * The period-averaged variance V_t of Sec. III-A (eq. (vt)) follows from the
 * records: Var[W_k] is 0 at the first step of a period and trace[k-1].var at
 * the others. */
ADPSGD_API int adpsgd_run_traced(adpsgd_ctx *c, int64_t n_steps, adpsgd_sync_rec *log, int64_t log_cap,
                                 double *var_log, adpsgd_step_rec *trace, int64_t trace_cap,
                                 int64_t *n_syncs);

ADPSGD_API int adpsgd_get_state(const adpsgd_ctx *c, adpsgd_state *out);
/* Restore a state saved by adpsgd_get_state (x, m restored by the caller):
 * t >= 0, cnt >= 0, nC2 >= 0, 1 <= p <= p_max, C2 finite. */
ADPSGD_API int adpsgd_set_state(adpsgd_ctx *c, const adpsgd_state *in);

/* Launch shape of the plain local step: block = 64, 128 or 256 threads (float4
 * groups of one worker's row per workgroup, a chunk); lds_bytes of LDS reserved
 * per block, which the kernel does not use: it only holds each CU to
 * floor(160 KB / lds_bytes) resident blocks (0: no reservation); and
 * row_chunks = S, the block order: the K blocks of a chunk run on one XCD, and
 * an XCD takes S chunks of one worker's row before the same S chunks of the
 * next worker's (1: the K workers of each chunk in turn).  The fastest shape
 * differs with the problem and the machine, so when K * P >= 2^24 adpsgd_init
 * times (64, 0, 1), (64, 8192, 1), (128, 0, 1), (256, 0, 1), (64, 8192, 16),
 * (64, 8192, 32) and (64, 8192, 64) on the context's buffers and keeps the
 * fastest (else (256, 0, 1)).  set: block 64, 128 or 256 with lds_bytes in
 * [0, 65536] and row_chunks in [1, 4096], or block 0 for the timed choice (the
 * others ignored); every shape computes the same bits.  EINVAL otherwise. */
ADPSGD_API int adpsgd_set_step_launch(adpsgd_ctx *c, int32_t block, int32_t lds_bytes, int32_t row_chunks);
ADPSGD_API int adpsgd_get_step_launch(const adpsgd_ctx *c, int32_t *block, int32_t *lds_bytes,
                                      int32_t *row_chunks);

/* How adpsgd_run launches its steps (ADPSGD_LAUNCH_*); every policy computes the
 * same results.  EINVAL for an unknown policy. */
ADPSGD_API int adpsgd_set_launch_policy(adpsgd_ctx *c, int32_t policy);

/* Per-kernel HIP-event timing (off by default).  every = 0: off; every >= 1:
 * HIP events around every every-th launch of each kernel kind (1: all), so the
 * events disturb the timed work little; adpsgd_timing then holds the sampled
 * launches.  Setting or reading it waits for the stream; setting it clears the
 * totals.  EINVAL for every < 0. */
ADPSGD_API int adpsgd_set_timing(adpsgd_ctx *c, int32_t every);
ADPSGD_API int adpsgd_get_timing(adpsgd_ctx *c, adpsgd_timing *out);

/* Release the context (host memory and events).  Waits for the stream.  The
 * caller's device buffers are untouched.  NULL is accepted. */
ADPSGD_API int adpsgd_destroy(adpsgd_ctx *c);

/* Message for the calling thread's last failed call (empty if none). */
ADPSGD_API const char *adpsgd_last_error(void);

/* ---- synchronization without allocation ------------------------------------ */

/* For callers that cannot allocate device memory (tight serving loops,
 * harnesses that forbid hipMalloc): the separate synchronization of
 * adpsgd_average with no context.  It waits for its stream before returning,
 * so it cannot itself be recorded into a HIP graph.  x [K][P] (device, rows
 * row_stride elements apart, 0 meaning P; 16-byte aligned) is replaced by the
 * replica mean in every row, and var_out[T] (host) receives the per-tensor
 * variances (1/K) sum_k sum_{i in tau} (xbar_i - x_{k,i})^2 of the replicas
 * before the mean; tensor_offsets[T+1] (host) as for adpsgd_init.  The
 * replicas get the same bits as adpsgd_average gives a context of the same
 * shape; the variances agree to rounding (another summation order).  Blocks
 * until var_out is valid; runs on `stream` (NULL: the null stream) of the
 * current device.
 * It allocates nothing: the tile table, the partial sums and the variances
 * live in a 64 MiB array of device memory that the library reserves on each
 * GPU it runs on, for the life of the process (problems of up to about 2
 * million sync tiles of 256 elements, e.g. 5e8 parameters; larger ones get
 * EINVAL).  Calls on one GPU share that array: calls that overlap on one GPU
 * (other threads, other streams) race and must be serialized by the caller. */
ADPSGD_API int adpsgd_average_noalloc(int32_t K, int64_t P, int64_t row_stride, const int64_t *tensor_offsets,
                                      int32_t T, float *x, double *var_out, void *stream);

/* ---- generator dumps (the device code the steps use) ------------------------ */

/* dev_out[4j .. 4j+3] = Philox4x32-10(key = (seed mod 2^32, seed >> 32),
 * counter = (g0 + j, c1, c2, c3)) for j < n_groups; device uint32 [4 n_groups].
 * Asynchronous on stream. */
ADPSGD_API int adpsgd_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                       int64_t n_groups, uint32_t *dev_out, void *stream);

/* dev_out[4j .. 4j+3] = the four Box-Muller normals of the same words:
 * (z0, z1) = sqrt(-2 ln u1) (cos 2 pi u2, sin 2 pi u2) with
 * u1 = ((r0 >> 8) + 1) 2^-24, u2 = (r1 >> 8) 2^-24, and likewise (z2, z3)
 * from (r2, r3).  Device float [4 n_groups].  Asynchronous on stream. */
ADPSGD_API int adpsgd_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                       int64_t n_groups, float *dev_out, void *stream);

/* ---- host-only controller (no GPU needed) ------------------------------------ */

/* Learning rate gamma_t of 0-based step t under hp's schedule. */
ADPSGD_API double adpsgd_lr(const adpsgd_hparams *hp, int64_t t);

/* Initial controller state: t = cnt = nC2 = 0, C2 = 0, p = p_init. */
ADPSGD_API int adpsgd_sched_init(const adpsgd_hparams *hp, adpsgd_state *st);

/* Begin step t = st->t (Algorithm 2's counter and its sync test): cnt += 1,
 * the period in force is set (p_after from p_switch_step on, constant modes),
 * and *sync_due = 1 if a sync follows this step: always during the warm-up
 * prefix, t mod p == 0 in ADPSGD_PERIOD_ALG1, cnt >= p otherwise.  Advances
 * st->t.  EINVAL on a NULL pointer. */
ADPSGD_API int adpsgd_sched_step(const adpsgd_hparams *hp, adpsgd_state *st, int32_t *sync_due);

/* Apply Algorithm 2's counter restart, sampling and period decision for a sync
 * after step t with variance S: cnt = 0; in adaptive mode after the warm-up
 * prefix, C2 sampling (t < k_s) or p +- 1.  *margin (may be NULL) receives the decision margin (NaN if no
 * decision).  ENONFINITE if S is not finite: cnt = 0 as after every sync,
 * with p, C2 and nC2 unchanged; EINVAL on a NULL pointer. */
ADPSGD_API int adpsgd_sched_on_sync(const adpsgd_hparams *hp, adpsgd_state *st, int64_t t, double S,
                         double *margin);

#ifdef __cplusplus
}
#endif
#endif /* ADPSGD_H */
