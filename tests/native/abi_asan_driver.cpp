// Host-side AddressSanitizer driver for the library's C ABI: every entry point,
// every launch policy, traced runs, checkpoint state, timing, error paths.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <vector>
#include <cmath>
#include <cstring>
#include "adpsgd.h"

#define CK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e), __LINE__); return 1;} } while(0)
#define OKC(x) do { int rc = (x); if (rc != 0) { printf("adpsgd error %d (%s) at %d\n", rc, adpsgd_last_error(), __LINE__); return 1;} } while(0)

static adpsgd_hparams hp_of(int mode, int p_init, int64_t N, int64_t k_s) {
    adpsgd_hparams h{};
    h.seed = 7; h.sigma = 0.1; h.momentum = 0.9; h.weight_decay = 5e-4; h.h_lo = 1e-2; h.h_hi = 1.0;
    h.lr_kind = ADPSGD_LR_STEP; h.period_mode = mode; h.lr0 = 0.05; h.total_steps = N; h.p_init = p_init;
    h.p_max = 0; h.k_s = k_s; h.thr_lo = 0.7; h.thr_hi = 1.3;
    return h;
}

static int one(int K, std::vector<int64_t> sizes, int mode, int p_init, int64_t N, int64_t k_s, int policy, bool traced,
               bool pad_rows = false) {
    std::vector<int64_t> off(1, 0);
    for (auto s : sizes) off.push_back(off.back() + s);
    const int T = (int)sizes.size();
    const int64_t P = off.back();
    adpsgd_hparams hp = hp_of(mode, p_init, N, k_s);
    size_t ws = adpsgd_workspace_bytes(K, P, T, off.data());
    if (!ws) { printf("workspace 0\n"); return 1; }
    float *x, *m, *h, *xs; void *w;
    const int64_t ld = pad_rows ? (P + 255) / 256 * 256 : P;  // rows 1 KB aligned
    CK(hipMalloc(&x, 4 * (size_t)K * ld + 16)); CK(hipMalloc(&m, 4 * (size_t)K * ld + 16));
    CK(hipMalloc(&h, 4 * (size_t)P + 16)); CK(hipMalloc(&xs, 4 * (size_t)P + 16)); CK(hipMalloc(&w, ws));
    adpsgd_buffers b{x, m, h, xs, w, ws, nullptr, pad_rows ? ld : 0};
    adpsgd_ctx *c = nullptr;
    OKC(adpsgd_init(K, P, off.data(), T, &hp, &b, &c));
    OKC(adpsgd_set_launch_policy(c, policy));
    OKC(adpsgd_set_timing(c, 3));
    int32_t blk = 0, lds = 0, rch = 0;
    OKC(adpsgd_get_step_launch(c, &blk, &lds, &rch));
    OKC(adpsgd_set_step_launch(c, 64, 8192, 32));
    if (adpsgd_set_step_launch(c, 96, 0, 1) != ADPSGD_EINVAL || adpsgd_set_step_launch(c, 64, 0, 0) != ADPSGD_EINVAL ||
        adpsgd_get_step_launch(c, &blk, nullptr, &rch) != ADPSGD_EINVAL) {
        printf("expected EINVAL\n"); return 1;
    }
    std::vector<adpsgd_sync_rec> log(N);
    std::vector<double> var((size_t)N * T);
    std::vector<adpsgd_step_rec> tr(N);
    int64_t n = 0;
    if (traced) OKC(adpsgd_run_traced(c, N / 2, log.data(), (int64_t)log.size(), var.data(), tr.data(), (int64_t)tr.size(), &n));
    else OKC(adpsgd_run(c, N / 2, log.data(), (int64_t)log.size(), var.data(), &n));
    adpsgd_state st;
    OKC(adpsgd_get_state(c, &st));
    // a small log capacity and no var log
    OKC(adpsgd_run(c, N - N / 2, log.data(), 3, nullptr, &n));
    OKC(adpsgd_set_state(c, &st));
    std::vector<double> v(T);
    OKC(adpsgd_local_steps(c, 3));
    OKC(adpsgd_step_average(c, v.data()));
    OKC(adpsgd_average(c, v.data()));
    int32_t np = 0;
    OKC(adpsgd_schedule(c, v.data(), &np));
    adpsgd_timing tm;
    OKC(adpsgd_get_timing(c, &tm));
    // error paths leave the context usable
    if (adpsgd_run(c, -1, nullptr, 0, nullptr, nullptr) != ADPSGD_EINVAL) { printf("expected EINVAL\n"); return 1; }
    if (adpsgd_set_launch_policy(c, 9) != ADPSGD_EINVAL) { printf("expected EINVAL\n"); return 1; }
    OKC(adpsgd_set_step_launch(c, 0, 0, 0));
    OKC(adpsgd_reset(c));
    OKC(adpsgd_run(c, 5, nullptr, 0, nullptr, &n));
    OKC(adpsgd_destroy(c));
    CK(hipFree(x)); CK(hipFree(m)); CK(hipFree(h)); CK(hipFree(xs)); CK(hipFree(w));
    printf("ok K=%d P=%lld T=%d mode=%d policy=%d traced=%d rows=%s syncs=%lld timed steps=%lld\n", K, (long long)P, T,
           mode, policy, (int)traced, pad_rows ? "padded" : "packed", (long long)n, (long long)tm.step_launches);
    fflush(stdout);
    return 0;
}

// A constant-period run replayed as a HIP graph (timing off, hybrid policy) on
// the null stream or a stream of the caller's: captured once, replayed, captured
// again for a new start state and after a launch-shape change; each replay must
// leave the bits of the host-waiting policy's eager launches.  Then the
// no-allocation sync on copies of the replicas against adpsgd_average.
static int graph_and_noalloc(bool own_stream) {
    const std::vector<int64_t> sizes = {5000, 77, 1, 0, 1024, 3, 70000, 263};
    std::vector<int64_t> off(1, 0);
    for (auto v : sizes) off.push_back(off.back() + v);
    const int T = (int)sizes.size(), K = 4;
    const int64_t P = off.back(), N = 60;
    adpsgd_hparams hp = hp_of(ADPSGD_PERIOD_CONST, 4, N, 0);
    hipStream_t st = nullptr;
    if (own_stream) CK(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    std::vector<float> ref((size_t)K * P), got((size_t)K * P);
    for (int pass = 0; pass < 2; ++pass) {   // pass 0: eager reference; pass 1: graph replays
        size_t ws = adpsgd_workspace_bytes(K, P, T, off.data());
        float *x, *m, *h, *xs; void *w;
        CK(hipMalloc(&x, 4 * (size_t)K * P)); CK(hipMalloc(&m, 4 * (size_t)K * P));
        CK(hipMalloc(&h, 4 * (size_t)P)); CK(hipMalloc(&xs, 4 * (size_t)P)); CK(hipMalloc(&w, ws));
        adpsgd_buffers b{x, m, h, xs, w, ws, st, 0};
        adpsgd_ctx *c = nullptr;
        OKC(adpsgd_init(K, P, off.data(), T, &hp, &b, &c));
        OKC(adpsgd_set_launch_policy(c, pass == 0 ? ADPSGD_LAUNCH_HOST : ADPSGD_LAUNCH_HYBRID));
        std::vector<adpsgd_sync_rec> log(N);
        std::vector<double> var((size_t)N * T);
        int64_t n = 0;
        for (int rep = 0; rep < 3; ++rep) {
            OKC(adpsgd_reset(c));
            OKC(adpsgd_run(c, N, log.data(), rep == 1 ? 2 : (int64_t)log.size(), rep == 2 ? nullptr : var.data(), &n));
            CK(hipMemcpy(pass == 0 ? ref.data() : got.data(), x, 4 * (size_t)K * P, hipMemcpyDeviceToHost));
            if (pass == 1 && std::memcmp(ref.data(), got.data(), 4 * (size_t)K * P) != 0) {
                printf("graph replay %d differs from the eager run\n", rep); return 1;
            }
            std::vector<double> v(T);
            OKC(adpsgd_local_steps(c, 2));   // eager work between the replays
            OKC(adpsgd_average(c, v.data()));
        }
        OKC(adpsgd_run(c, 7, log.data(), (int64_t)log.size(), var.data(), &n));   // a new start state
        OKC(adpsgd_set_step_launch(c, 128, 0, 1));
        OKC(adpsgd_reset(c));
        OKC(adpsgd_run(c, N, log.data(), (int64_t)log.size(), var.data(), &n));   // a new launch shape
        adpsgd_timing tm;
        OKC(adpsgd_get_timing(c, &tm));
        if (pass == 1 && (tm.graph_captures != 3 || tm.graph_replays != 5)) {
            printf("graph captures %lld replays %lld\n", (long long)tm.graph_captures, (long long)tm.graph_replays);
            return 1;
        }
        if (pass == 1) {
            // the no-allocation sync on a copy of the replicas, against adpsgd_average
            float *x2;
            CK(hipMalloc(&x2, 4 * (size_t)K * P));
            OKC(adpsgd_local_steps(c, 3));
            // the steps are asynchronous on the context's stream, and a device-to-device
            // copy does not block the host: copy on that stream and wait for it
            CK(hipMemcpyAsync(x2, x, 4 * (size_t)K * P, hipMemcpyDeviceToDevice, st));
            CK(hipStreamSynchronize(st));
            std::vector<double> v1(T), v2(T);
            OKC(adpsgd_average(c, v1.data()));
            OKC(adpsgd_average_noalloc(K, P, 0, off.data(), T, x2, v2.data(), st));
            std::vector<float> a((size_t)K * P), bb((size_t)K * P);
            CK(hipMemcpy(a.data(), x, 4 * (size_t)K * P, hipMemcpyDeviceToHost));
            CK(hipMemcpy(bb.data(), x2, 4 * (size_t)K * P, hipMemcpyDeviceToHost));
            if (std::memcmp(a.data(), bb.data(), 4 * (size_t)K * P) != 0) { printf("no-alloc sync differs\n"); return 1; }
            for (int i = 0; i < T; ++i)
                if (std::fabs(v1[i] - v2[i]) > 1e-12 * std::fabs(v1[i])) { printf("no-alloc variance differs\n"); return 1; }
            // a smaller problem next (K = 2, the first three tensors)
            const int64_t P2 = off[3];
            OKC(adpsgd_average_noalloc(2, P2, P, off.data(), 3, x2, v2.data(), st));
            CK(hipFree(x2));
        }
        OKC(adpsgd_destroy(c));
        CK(hipFree(x)); CK(hipFree(m)); CK(hipFree(h)); CK(hipFree(xs)); CK(hipFree(w));
    }
    if (st) CK(hipStreamDestroy(st));
    printf("ok graph replays and no-alloc sync (%s stream)\n", own_stream ? "own" : "null");
    fflush(stdout);
    return 0;
}

int main() {
    if (graph_and_noalloc(false) || graph_and_noalloc(true)) return 1;
    const std::vector<int64_t> ragged = {5000, 77, 1, 0, 1024, 3, 70000, 263};
    // more chunk partials than the finishing block's LDS holds: the window
    // tables (a split run of small tensors and one tensor of over 32 chunks)
    std::vector<int64_t> many;
    uint32_t r = 12345;
    for (int i = 0; i < 3300; ++i) {
        r = r * 1664525u + 1013904223u;
        many.push_back(1 + (r >> 8) % 300);
        if (i == 2500) many.push_back(9000001);
    }
    for (int policy = 0; policy < 3; ++policy)
        for (int traced = 0; traced < 2; ++traced) {
            if (one(8, ragged, ADPSGD_PERIOD_ADAPTIVE, 1, 120, 30, policy, traced)) return 1;
            if (one(8, ragged, ADPSGD_PERIOD_ADAPTIVE, 1, 60, 15, policy, traced, true)) return 1;
            if (one(3, ragged, ADPSGD_PERIOD_ADAPTIVE, 2, 90, 20, policy, traced)) return 1;
            if (one(32, {300000}, ADPSGD_PERIOD_CONST, 4, 40, 0, policy, traced)) return 1;
            if (one(4, {0, 0}, ADPSGD_PERIOD_ALG1, 3, 20, 0, policy, traced)) return 1;
            if (one(2, many, ADPSGD_PERIOD_ADAPTIVE, 2, 24, 6, policy, traced)) return 1;
            // x and m take 320 MB, between the last-level cache and 1 GiB: init
            // times the cached and non-temporal sync variants as well as the
            // step's launch shapes
            if (one(8, {5000000}, ADPSGD_PERIOD_ADAPTIVE, 2, 16, 4, policy, traced, true)) return 1;
        }
    printf("all ok\n");
    fflush(stdout);
    return 0;
}
