// Test infrastructure: the library's host code under AddressSanitizer and
// UndefinedBehaviorSanitizer, with no GPU.  Runs every path that needs no
// device: workspace planning (tile, chunk and window tables) on regular,
// ragged, empty and many-tensor partitions; adpsgd_init's validation and the
// plan it builds before its first HIP call (which fails on a machine without
// a GPU, so the context is built and released again); the host controller
// (adpsgd_sched_*) and the learning-rate schedules over every mode, with caps,
// warm-up prefixes, period switches and non-finite variances; the argument
// checks of the generator dumps and of adpsgd_average_noalloc; and calls with
// pointers that are not live contexts.  Prints "all ok" at the end.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <vector>

#include "adpsgd.h"

static int g_fail = 0;
#define EXPECT(cond)                                                          \
    do {                                                                      \
        if (!(cond)) {                                                        \
            std::printf("FAILED at line %d: %s (%s)\n", __LINE__, #cond, adpsgd_last_error()); \
            ++g_fail;                                                         \
        }                                                                     \
    } while (0)

static adpsgd_hparams hparams(int mode, int lr_kind, int p_init, int64_t N, int64_t k_s) {
    adpsgd_hparams h;
    std::memset(&h, 0, sizeof h);
    h.seed = 11;
    h.sigma = 0.1;
    h.momentum = 0.9;
    h.weight_decay = 5e-4;
    h.h_lo = 1e-2;
    h.h_hi = 1.0;
    h.lr_kind = lr_kind;
    h.period_mode = mode;
    h.lr0 = 0.05;
    h.total_steps = N;
    h.p_init = p_init;
    h.k_s = k_s;
    h.thr_lo = 0.7;
    h.thr_hi = 1.3;
    return h;
}

static std::vector<int64_t> offsets_of(const std::vector<int64_t> &sizes) {
    std::vector<int64_t> off(1, 0);
    for (int64_t s : sizes) off.push_back(off.back() + s);
    return off;
}

// Workspace sizes of partitions that take every plan: one tile per chunk,
// chunks of 1024 tiles, more chunk partials than one window (window tables),
// empty tensors, and odd sizes.
static void workspace_plans() {
    std::vector<std::vector<int64_t>> parts = {
        {4096},
        {0, 0, 0},
        {1, 3, 5, 7, 0, 255, 256, 257},
        std::vector<int64_t>(3301, 37),                    // many small tensors: windows
        {600000, 17, 1300000, 0, 5},                       // chunks of 1024 tiles
        {int64_t(1) << 28, 3, int64_t(1) << 27},           // large tensors, no memory touched
    };
    std::vector<int64_t> mixed;
    for (int i = 0; i < 5000; ++i) mixed.push_back(i % 7 == 0 ? 300000 : 20 + (i % 13));
    parts.push_back(mixed);                                 // windows with large tensors between runs
    for (const auto &sz : parts) {
        const std::vector<int64_t> off = offsets_of(sz);
        for (int K : {1, 3, 8, 65536}) {
            const size_t ws = adpsgd_workspace_bytes(K, off.back(), (int32_t)sz.size(), off.data());
            EXPECT(ws > 0 && ws % 256 == 0);
        }
    }
    // refused: K out of range, decreasing offsets, wrong last offset, NULL, T = 0
    std::vector<int64_t> bad = {0, 9, 8};
    EXPECT(adpsgd_workspace_bytes(0, 8, 1, offsets_of({8}).data()) == 0);
    EXPECT(adpsgd_workspace_bytes(65537, 8, 1, offsets_of({8}).data()) == 0);
    EXPECT(adpsgd_workspace_bytes(2, 8, 2, bad.data()) == 0);
    EXPECT(adpsgd_workspace_bytes(2, 9, 1, offsets_of({8}).data()) == 0);
    EXPECT(adpsgd_workspace_bytes(2, 8, 1, nullptr) == 0);
    EXPECT(adpsgd_workspace_bytes(2, 0, 0, offsets_of({}).data()) == 0);
}

// adpsgd_init up to its first device call: validation errors, then a valid
// call whose plan is built and released again when the runtime has no device.
static void init_paths() {
    alignas(256) static unsigned char arena[1 << 16];
    float *f = reinterpret_cast<float *>(arena);
    adpsgd_hparams hp = hparams(ADPSGD_PERIOD_ADAPTIVE, ADPSGD_LR_STEP, 4, 100, 25);
    adpsgd_ctx *c = nullptr;
    std::vector<int64_t> sizes = {1000, 7, 0, 4093};
    std::vector<int64_t> off = offsets_of(sizes);
    const int64_t P = off.back();
    const size_t ws = adpsgd_workspace_bytes(8, P, 4, off.data());
    adpsgd_buffers b{f, f, f, f, arena, ws, nullptr, 0};
    EXPECT(adpsgd_init(8, P, off.data(), 4, &hp, &b, nullptr) == ADPSGD_EINVAL);
    EXPECT(adpsgd_init(8, P, off.data(), 4, nullptr, &b, &c) == ADPSGD_EINVAL && c == nullptr);
    EXPECT(adpsgd_init(8, P, off.data(), 4, &hp, nullptr, &c) == ADPSGD_EINVAL);
    adpsgd_buffers mis = b;
    mis.x = f + 1;
    EXPECT(adpsgd_init(8, P, off.data(), 4, &hp, &mis, &c) == ADPSGD_EINVAL);
    adpsgd_buffers small = b;
    small.workspace_bytes = ws - 1;
    EXPECT(adpsgd_init(8, P, off.data(), 4, &hp, &small, &c) == ADPSGD_EINVAL);
    adpsgd_buffers stride = b;
    stride.row_stride = P - 1;
    EXPECT(adpsgd_init(8, P, off.data(), 4, &hp, &stride, &c) == ADPSGD_EINVAL);
    adpsgd_hparams bad = hp;
    bad.momentum = 1.0;
    EXPECT(adpsgd_init(8, P, off.data(), 4, &bad, &b, &c) == ADPSGD_EINVAL);
    // a valid call: the plan is built; without a device the first HIP call fails
    // and the partly built context is released (ASan checks that release)
    const int rc = adpsgd_init(8, P, off.data(), 4, &hp, &b, &c);
    EXPECT(rc == ADPSGD_EDEVICE && c == nullptr);
    std::vector<int64_t> many(3301, 37);
    std::vector<int64_t> moff = offsets_of(many);
    const size_t mws = adpsgd_workspace_bytes(3, moff.back(), 3301, moff.data());
    std::vector<unsigned char> big(mws + 256);
    void *wsp = reinterpret_cast<void *>((reinterpret_cast<uintptr_t>(big.data()) + 255) / 256 * 256);
    adpsgd_buffers mb{f, f, f, f, wsp, mws, nullptr, 0};
    EXPECT(adpsgd_init(3, moff.back(), moff.data(), 3301, &hp, &mb, &c) == ADPSGD_EDEVICE && c == nullptr);
}

// The host controller over every mode against its own invariants.
static void controller_paths() {
    const int modes[] = {ADPSGD_PERIOD_CONST, ADPSGD_PERIOD_ADAPTIVE, ADPSGD_PERIOD_ALG1};
    const int lrs[] = {ADPSGD_LR_CONST, ADPSGD_LR_STEP, ADPSGD_LR_COSINE, ADPSGD_LR_WARMUP_STEP};
    uint64_t rng = 12345;
    auto next = [&]() { rng = rng * 6364136223846793005ull + 1442695040888963407ull; return (double)(rng >> 11) * 0x1p-53; };
    for (int mode : modes)
        for (int lr : lrs)
            for (int variant = 0; variant < 4; ++variant) {
                const int64_t N = 500;
                adpsgd_hparams hp = hparams(mode, lr, 3, N, mode == ADPSGD_PERIOD_ADAPTIVE ? 100 : 0);
                if (variant == 1) hp.p_max = 6;
                if (variant == 2) hp.sync_warmup_steps = 37;
                if (variant == 3 && mode != ADPSGD_PERIOD_ADAPTIVE) { hp.p_switch_step = 250; hp.p_after = 7; }
                adpsgd_state st;
                EXPECT(adpsgd_sched_init(&hp, &st) == ADPSGD_OK);
                int64_t syncs = 0;
                for (int64_t t = 0; t < N; ++t) {
                    const double g = adpsgd_lr(&hp, t);
                    EXPECT(std::isfinite(g) && g > 0);
                    int32_t due = 0;
                    EXPECT(adpsgd_sched_step(&hp, &st, &due) == ADPSGD_OK);
                    if (!due) continue;
                    ++syncs;
                    double S = g * (0.2 + 1.6 * next());
                    if (t % 97 == 96) S = std::numeric_limits<double>::quiet_NaN();
                    double margin = 0.0;
                    const int rc = adpsgd_sched_on_sync(&hp, &st, t, S, &margin);
                    EXPECT(rc == (std::isfinite(S) ? ADPSGD_OK : ADPSGD_ENONFINITE));
                    EXPECT(st.cnt == 0 && st.p >= 1 && (hp.p_max == 0 || st.p <= hp.p_max));
                }
                EXPECT(st.t == N && syncs > 0);
            }
    adpsgd_hparams hp = hparams(ADPSGD_PERIOD_ADAPTIVE, ADPSGD_LR_CONST, 3, 10, 0);
    adpsgd_state st;
    int32_t due;
    EXPECT(adpsgd_sched_step(nullptr, &st, &due) == ADPSGD_EINVAL);
    EXPECT(adpsgd_sched_step(&hp, nullptr, &due) == ADPSGD_EINVAL);
    EXPECT(adpsgd_sched_on_sync(&hp, nullptr, 0, 1.0, nullptr) == ADPSGD_EINVAL);
    EXPECT(adpsgd_sched_init(&hp, nullptr) == ADPSGD_EINVAL);
    EXPECT(std::isnan(adpsgd_lr(nullptr, 0)));
    hp.p_init = 0;
    EXPECT(adpsgd_sched_init(&hp, &st) == ADPSGD_EINVAL);
}

// Entry points that must refuse before touching a device.
static void refusals() {
    double var[4];
    int64_t off[2] = {0, int64_t(1) << 30};
    EXPECT(adpsgd_average_noalloc(2, off[1], 0, off, 1, reinterpret_cast<float *>(256), var, nullptr) == ADPSGD_EINVAL);
    EXPECT(adpsgd_average_noalloc(0, 8, 0, off, 1, nullptr, var, nullptr) == ADPSGD_EINVAL);
    int64_t bad[3] = {0, 9, 8};
    EXPECT(adpsgd_average_noalloc(2, 8, 0, bad, 2, nullptr, var, nullptr) == ADPSGD_EINVAL);
    EXPECT(adpsgd_philox_dump(0, 0, 0, 0, -1, 8, nullptr, nullptr) == ADPSGD_EINVAL);
    EXPECT(adpsgd_normal_dump(0, 0, 0, 0, (int64_t(1) << 32) - 4, 8, nullptr, nullptr) == ADPSGD_EINVAL);
    // pointers that are not live contexts are refused without being touched
    alignas(64) static unsigned char junk[256];
    adpsgd_ctx *fake = reinterpret_cast<adpsgd_ctx *>(junk);
    adpsgd_state st;
    EXPECT(adpsgd_local_steps(fake, 1) == ADPSGD_EINVAL);
    EXPECT(adpsgd_get_state(fake, &st) == ADPSGD_EINVAL);
    EXPECT(adpsgd_destroy(fake) == ADPSGD_EINVAL);
    EXPECT(adpsgd_destroy(nullptr) == ADPSGD_OK);
    EXPECT(adpsgd_run(nullptr, 1, nullptr, 0, nullptr, nullptr) == ADPSGD_EINVAL);
    EXPECT(std::strlen(adpsgd_last_error()) > 0);
}

int main() {
#ifdef HOST_SANITIZE_PLANT
    {   // a planted one-element heap overflow: the test expects ASan to stop here
        std::vector<int64_t> v(5, 1);
        volatile int64_t *p = v.data();
        std::printf("%lld\n", (long long)p[5]);
    }
#endif
    workspace_plans();
    init_paths();
    controller_paths();
    refusals();
    if (g_fail) {
        std::printf("%d failures\n", g_fail);
        return 1;
    }
    std::printf("all ok\n");
    return 0;
}
