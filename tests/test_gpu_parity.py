"""Parity of the HIP path (through the C ABI) with the CPU oracle, on cuda:0.

Bars: Philox words bit-exact; fp32 parameters within 1e-4 max relative error
(per tensor, against max(|oracle|, 1e-2 rms)) and momentum buffers within 3e-4
(against max(|oracle|, rms)); per-tensor variances within 1e-3 relative; the
sequence of sync steps identical (tests/helpers.py holds the bars).
"""
import sys

import numpy as np
import pytest

import oracle
import oracle.oracle as OO
import workloads as W
from helpers import MOM_FLOOR, MOM_TOL, PARAM_TOL, VAR_TOL, assert_same_syncs, gpu_run, max_rel_err, rel_err

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def A():
    import torch
    assert torch.cuda.is_available()
    import paper_2007_06134_amd as A
    return A


def _tiny(K=4, sizes=(4096,), **kw):
    base = dict(name="tiny", K=K, sizes=tuple(sizes), seed=21, sigma=0.1, momentum=0.9,
                weight_decay=5e-4, h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.05,
                total_steps=40, period_mode=W.PERIOD_CONST, p_init=10**6, k_s=0)
    base.update(kw)
    return W.Workload(**base)


# ---------------------------------------------------------------- generator

@pytest.mark.parametrize("seed,c,g0,n", [
    (0, (0, 0, 0), 0, 4096), (1, (3, 17, 0), 12345, 1000),
    ((7 << 32) | 99, (31, 4999, 1), 2**32 - 777, 777), (0xDEADBEEFCAFEBABE, (5, 6, 2), 1, 4096 * 3 + 5),
])
def test_philox_words_bit_exact(A, seed, c, g0, n):
    import torch
    _say(f"philox dump seed={seed} c={c} g0={g0} n={n}")
    out = torch.zeros(4 * n, dtype=torch.int32, device="cuda")
    A.adpsgd_philox_dump(seed, *c, g0, n, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32).reshape(n, 4)
    want = oracle.philox_groups(seed, *c, g0, n)
    assert np.array_equal(got, want)


def test_normals_match_oracle(A):
    import torch
    n = 1 << 18
    _say("normal dump")
    out = torch.zeros(4 * n, dtype=torch.float32, device="cuda")
    A.adpsgd_normal_dump(77, 2, 9, 0, 0, n, out.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    want = oracle.normals_groups(77, 2, 9, 0, 0, n)
    err = np.abs(got - want) / np.maximum(1.0, np.abs(want))
    # fp32 log/sqrt/sincospi against fp64: a few ulp of the result
    assert err.max() < 2e-6, err.max()


@pytest.mark.parametrize("P", [1, 5, 4096, 10_001])
def test_problem_data_matches_oracle(A, P):
    w = _tiny(K=2, sizes=(P,), h_lo=1e-3)
    _say(f"problem data P={P}")
    with A.Adpsgd.from_workload(w) as eng:
        h = eng.h.double().cpu().numpy()
        xs = eng.xstar.double().cpu().numpy()
        assert not eng.x.any() and not eng.m.any()
    h_o, xs_o = oracle.problem_data(w)
    assert rel_err(h, h_o) < 2e-6
    assert np.max(np.abs(xs - xs_o) / np.maximum(1.0, np.abs(xs_o))) < 2e-6


# ---------------------------------------------------------------- local steps and sync

@pytest.mark.parametrize("K", [1, 2, 3, 4, 8, 12, 16, 24, 32, 48])
@pytest.mark.parametrize("sizes", [(4096 * 3 + 4,), (5000, 3, 5001, 993)])   # aligned / ragged P
def test_local_steps_match_oracle(A, K, sizes):
    w = _tiny(K=K, sizes=sizes)
    n = 7
    _say(f"local steps K={K} P={w.P}")
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(n)
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
        st = eng.get_state()
    r = oracle.Oracle(w).run(n_steps=n)
    assert r.n_syncs == 0 and st.t == n and st.cnt == n
    assert max_rel_err(x, r.x, w.offsets()) < PARAM_TOL
    assert max_rel_err(m, r.v, w.offsets(), floor=MOM_FLOOR) < MOM_TOL


# K = 12, 24: the sync-tile kernel with K as an argument (two rows per wave);
# 25: the same with a ragged last wave; 33, 48, 64: four rows per wave (33
# ragged); 3: the loop kernel for the separate sync (one row per wave when a
# step comes first); 65: the loop kernel
@pytest.mark.parametrize("K", [1, 3, 8, 12, 24, 25, 32, 33, 48, 64, 65])
@pytest.mark.parametrize("sizes", [(4096 * 3 + 4,), (5000, 3, 0, 5001, 993, 1), (8192, 4096, 12)])
def test_average_matches_oracle(A, K, sizes):
    w = _tiny(K=K, sizes=sizes)
    n = 6
    _say(f"average K={K} sizes={sizes}")
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(n)
        var = eng.average()
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
        assert eng.get_state().cnt == 0
    o = oracle.Oracle(w)
    r = o.run(n_steps=n)
    S_o, var_o = o.average(r.x)
    off = w.offsets()
    assert all(np.array_equal(x[k], x[0]) for k in range(K))   # every replica holds the mean
    assert max_rel_err(x, r.x, off) < PARAM_TOL
    assert max_rel_err(m, r.v, off, floor=MOM_FLOOR) < MOM_TOL   # momentum untouched
    if K == 1:
        assert np.all(var == 0.0)
    empty = np.diff(off) == 0
    assert np.all(var[empty] == 0.0)
    assert rel_err(var[~empty], var_o[~empty]) < VAR_TOL


@pytest.mark.parametrize("K", [2, 3, 5, 8, 12, 24, 25, 32, 33, 48, 64, 65])
def test_fused_sync_equals_step_then_sync(A, K):
    w = _tiny(K=K, sizes=(4099, 1, 8000, 6))
    _say(f"fused vs separate K={K}")
    with A.Adpsgd.from_workload(w) as a, A.Adpsgd.from_workload(w) as b:
        a.local_steps(4); va = a.step_average()
        b.local_steps(5); vb = b.average()
        # the replicas are bitwise equal (the same order of the mean); for a
        # compiled K the separate sync gives each wave two rows, so its
        # variance sums round in another order
        assert np.allclose(va, vb, rtol=1e-12, atol=0.0)
        assert a.get_state().t == b.get_state().t == 5
        import torch
        assert torch.equal(a.x, b.x) and torch.equal(a.m, b.m)


@pytest.mark.parametrize("K", [3, 8, 12, 24, 25, 32, 33, 48, 64, 65])
def test_second_sync_has_zero_variance(A, K):
    w = _tiny(K=K, sizes=(3000, 5000))
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(3)
        v1 = eng.average()
        v2 = eng.average()
    assert np.all(v1 > 0)
    if K & (K - 1) == 0 and K <= 64:
        assert np.all(v2 == 0.0)      # the pairwise mean of equal values is exact
    else:
        assert np.all(v2 <= 1e-9 * v1)  # one rounding of the mean per element


# ---------------------------------------------------------------- whole runs

@pytest.mark.parametrize("key", list(W.parity_workloads()))
def test_run_matches_oracle(A, key):
    w = W.parity_workloads()[key]
    _say(f"run {key}: K={w.K} P={w.P} T={w.T} N={w.total_steps}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    recs = g["recs"]
    assert_same_syncs(recs, r, w)
    assert g["n_syncs"] == r.n_syncs
    assert rel_err(recs["S"], r.S) < VAR_TOL
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    off = w.offsets()
    ex, em = max_rel_err(g["x"], r.x, off), max_rel_err(g["m"], r.v, off, floor=MOM_FLOOR)
    _say(f"  {key}: {r.n_syncs} syncs, err x {ex:.2e} m {em:.2e} "
         f"var {rel_err(g['var'], r.var):.2e}, min |margin| {np.nanmin(np.abs(recs['margin'])) if w.period_mode else float('nan'):.2e}")
    assert ex < PARAM_TOL
    assert em < MOM_TOL
    assert g["state"].t == w.total_steps and g["state"].p == r.state.p
    if w.period_mode == W.PERIOD_ADAPTIVE:
        assert rel_err([g["state"].C2], [r.state.C2]) < VAR_TOL


@pytest.mark.parametrize("K", [3, 5, 8, 16, 32])
def test_chunks_of_many_tensors_match_oracle(A, K):
    """The sync-tile kernel takes one block per aligned chunk of 256 elements
    and splits its sums over the tensors in the chunk: runs of 1- and 3-element
    tensors put up to 256 tensors in one chunk, between larger ones that start
    and end inside chunks.  Adaptive runs with fused syncs, a traced run and
    separate syncs (the loop kernel at K = 3) against the oracle, per tensor."""
    sizes = (1,) * 300 + (5000,) + (3,) * 90 + (0, 257) + (1,) * 40 + (999,)
    w = _tiny(K=K, sizes=sizes, p_init=2, total_steps=30, period_mode=W.PERIOD_ADAPTIVE, k_s=8)
    _say(f"chunks of many tensors: K={K} P={w.P} T={w.T}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    assert_same_syncs(g["recs"], r, w)
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    # x against the whole vector's rms floor: for a tensor of one element the
    # per-tensor floor of 1e-2 rms is that element's own magnitude, so the fp32
    # curvature's 2e-6 relative error, which reaches x as ~2e-6 absolute, would be
    # judged relative to |x| alone wherever x passes near zero
    assert max_rel_err(g["x"], r.x, [0, w.P]) < PARAM_TOL
    with A.Adpsgd.from_workload(w) as eng:
        recs, _, n, steps = eng.run_traced(12)
    rt = oracle.Oracle(w).run(n_steps=12, trace=True)
    assert rel_err(steps["var"], rt.trace_var) < VAR_TOL
    assert rel_err(steps["grad_norm2"], rt.trace_grad_norm2) < VAR_TOL
    ws = w.replace(period_mode=W.PERIOD_CONST, p_init=10**6, k_s=0)   # three steps, no sync among them
    with A.Adpsgd.from_workload(ws) as eng:
        eng.local_steps(3)
        var = eng.average()
    o = oracle.Oracle(ws)
    r3 = o.run(n_steps=3)
    _, var_o = o.average(r3.x)
    nz = np.diff(w.offsets()) > 0
    assert rel_err(var[nz], var_o[nz]) < VAR_TOL and np.all(var[~nz] == 0)


def _sizes_with_tiles(n_tiles, seed, max_size):
    """Ragged tensor sizes (log-uniform in [1, max_size]) whose sync tiles (cut
    at multiples of 256 elements, never across a tensor) number exactly n_tiles."""
    rng = np.random.default_rng(seed)
    sizes, start, tiles = [], 0, 0
    while tiles < n_tiles:
        size = int(np.exp(rng.uniform(0.0, np.log(max_size))))
        t = (start + size + 255) // 256 - start // 256
        if tiles + t >= n_tiles:      # last tensor: end inside the tile that completes the count
            end = (start // 256 + n_tiles - tiles - 1) * 256 + 1 + int(rng.integers(0, 255))
            size = end - start
            t = n_tiles - tiles
        sizes.append(size)
        start += size
        tiles += t
    return tuple(sizes)


@pytest.mark.parametrize("n_tiles,max_size", [(2048, 60_000), (2049, 60_000), (8300, 60_000), (4500, 400)])
def test_reduction_paths_match_oracle(A, n_tiles, max_size):
    """Tile counts on either side of each change of the variance reduction's
    path: every tile its own chunk (up to 2048 tiles, one launch), then chunks
    of tiles summed first (two launches); with thousands of small tensors the
    chunk partials outgrow the finishing block's LDS window and pass through it
    in several windows."""
    sizes = _sizes_with_tiles(n_tiles, n_tiles, max_size)
    w = W.Workload(name=f"tiles_{n_tiles}", K=4, sizes=sizes, seed=n_tiles, sigma=0.1, momentum=0.9,
                   weight_decay=5e-4, h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.05,
                   total_steps=16, period_mode=W.PERIOD_ADAPTIVE, p_init=2, k_s=6)
    _say(f"reduction paths: {n_tiles} tiles, T={w.T}, P={w.P}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    recs = g["recs"]
    assert_same_syncs(recs, r, w)
    assert rel_err(recs["S"], r.S) < VAR_TOL
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    off = w.offsets()
    assert max_rel_err(g["x"], r.x, off) < PARAM_TOL
    assert max_rel_err(g["m"], r.v, off, floor=MOM_FLOOR) < MOM_TOL


def test_reduction_windows_with_large_tensors_match_oracle(A):
    """More chunk partials than the finishing block's LDS window, with tensors
    of more than 32 chunks (over 8.4M elements) between runs of small ones:
    each large tensor is reduced in a window of its own, and a run of small
    tensors longer than one window is split."""
    rng = np.random.default_rng(2669)
    small = lambda n: [int(s) for s in rng.integers(1, 300, size=n)]
    sizes = tuple(small(1200) + [8_700_001] + small(2500) + [9_000_003] + small(100))
    w = W.Workload(name="windows_large", K=2, sizes=sizes, seed=2669, sigma=0.1, momentum=0.9,
                   weight_decay=5e-4, h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.05,
                   total_steps=10, period_mode=W.PERIOD_ADAPTIVE, p_init=2, k_s=4)
    _say(f"reduction windows: T={w.T}, P={w.P}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    recs = g["recs"]
    assert_same_syncs(recs, r, w)
    assert rel_err(recs["S"], r.S) < VAR_TOL
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    off = w.offsets()
    assert max_rel_err(g["x"], r.x, off) < PARAM_TOL
    assert max_rel_err(g["m"], r.v, off, floor=MOM_FLOOR) < MOM_TOL


@pytest.mark.parametrize("extra", [1, 2, 3])
@pytest.mark.parametrize("key", ["resnet18_like", "many_small"])
def test_padded_and_packed_rows_match_oracle(A, key, extra):
    """P not a multiple of 4: rows padded to a multiple of 4 elements (whole
    float4 groups move with vector accesses, the last group of each row
    masked) and rows packed back to back (scalar accesses) give the same bits
    and match the oracle."""
    w0 = W.parity_workloads()[key]
    sizes = list(w0.sizes)
    sizes[-1] += extra
    w = w0.replace(sizes=tuple(sizes), total_steps=60, k_s=15)
    assert w.P % 4 == extra
    _say(f"rows {key}: K={w.K} P={w.P}")
    gp, gk = gpu_run(w, pad_rows=True), gpu_run(w, pad_rows=False)
    assert gp["recs"].tobytes() == gk["recs"].tobytes() and gp["var"].tobytes() == gk["var"].tobytes()
    assert np.array_equal(gp["x"], gk["x"]) and np.array_equal(gp["m"], gk["m"])
    r = oracle.Oracle(w).run()
    assert_same_syncs(gp["recs"], r, w)
    assert rel_err(gp["var"], r.var, floor=1e-300) < VAR_TOL
    assert max_rel_err(gp["x"], r.x, w.offsets()) < PARAM_TOL
    assert max_rel_err(gp["m"], r.v, w.offsets(), floor=MOM_FLOOR) < MOM_TOL


def test_period_one_replicas_stay_identical(A):
    w = _tiny(K=8, sizes=(6000, 2001), p_init=1, total_steps=12)
    with A.Adpsgd.from_workload(w) as eng:
        recs, _, n = eng.run(12)
        x = eng.x.double().cpu().numpy()
    assert n == 12 and list(recs["t"]) == list(range(12))
    assert all(np.array_equal(x[k], x[0]) for k in range(8))
    xbar, _ = oracle.Oracle(w).mean_trajectory(12)
    assert max_rel_err(x[0], xbar, w.offsets()) < PARAM_TOL


def test_runs_are_bit_reproducible(A):
    w = W.parity_workloads()["many_small"].replace(total_steps=600, k_s=150)
    a, b = gpu_run(w), gpu_run(w)
    assert np.array_equal(a["x"], b["x"]) and np.array_equal(a["m"], b["m"])
    assert np.array_equal(a["var"], b["var"]) and a["recs"].tobytes() == b["recs"].tobytes()


@pytest.mark.parametrize("key", ["resnet18_like", "many_small", "vgg16_adaptive", "k3_adaptive", "k24_adaptive",
                                 "k25_adaptive"])
def test_launch_policies_agree_bitwise(A, key):
    """Host-planned, device-decided and host-waiting launches give the same bits:
    every step runs the same update code and every sync the same reduction and
    controller, whichever kernel the driver chose for it."""
    if key in ("k3_adaptive", "k24_adaptive", "k25_adaptive"):
        w = _tiny(K=int(key[1:key.index("_")]), sizes=(5000, 77, 1024, 3), p_init=2, total_steps=120,
                  period_mode=W.PERIOD_ADAPTIVE, k_s=30)
    else:
        w = W.parity_workloads()[key]
    _say(f"launch policies {key}: K={w.K} P={w.P} N={w.total_steps}")
    runs = {pol: gpu_run(w, policy=pol) for pol in (A.LAUNCH_HYBRID, A.LAUNCH_DEVICE, A.LAUNCH_HOST)}
    base = runs[A.LAUNCH_HYBRID]
    for pol, g in runs.items():
        assert g["n_syncs"] == base["n_syncs"], pol
        assert g["recs"].tobytes() == base["recs"].tobytes(), pol
        assert np.array_equal(g["var"], base["var"]), pol
        assert np.array_equal(g["x"], base["x"]) and np.array_equal(g["m"], base["m"]), pol
        assert (g["state"].t, g["state"].cnt, g["state"].p, g["state"].C2) == \
            (base["state"].t, base["state"].cnt, base["state"].p, base["state"].C2), pol


def _graph_case(key):
    pw = W.parity_workloads()
    return {
        "quad_small": pw["quad_small"],                       # K = 4, P = 65,536, period 4
        "vgg16_const8": pw["vgg16_const8"],                   # K = 8, 32 ragged tensors, period 8
        "alg1_switch": pw["resnet18_like"].replace(           # Algorithm 1's test, a period switch
            period_mode=W.PERIOD_ALG1, p_init=3, k_s=0, total_steps=300, p_switch_step=150, p_after=7),
        "warmup_k3": _tiny(K=3, sizes=(5000, 77, 3), total_steps=90, period_mode=W.PERIOD_CONST, p_init=5,
                           sync_warmup_steps=12),
    }[key]


@pytest.mark.parametrize("key", ["quad_small", "vgg16_const8", "alg1_switch", "warmup_k3"])
def test_graph_replays_equal_eager_runs(A, key):
    """A constant-period run of a small problem is captured once as a HIP graph
    and replayed while the same run repeats.  Every replay, with the program's
    own eager work and synchronizations between them (single steps, separate
    syncs, a checkpoint restored), gives the bits of the eager launches of the
    same run (the host-waiting policy, which never captures)."""
    import torch
    w = _graph_case(key)
    _say(f"graph replays {key}: K={w.K} P={w.P} N={w.total_steps}")
    ref = gpu_run(w, policy=A.LAUNCH_HOST)
    with A.Adpsgd.from_workload(w) as eng:
        for rep in range(4):
            eng.reset()
            recs, var, n = eng.run(w.total_steps)
            assert recs.tobytes() == ref["recs"].tobytes() and np.array_equal(var, ref["var"]), rep
            assert np.array_equal(eng.x.double().cpu().numpy(), ref["x"]), rep
            assert np.array_equal(eng.m.double().cpu().numpy(), ref["m"]), rep
            st = eng.get_state()
            assert (st.t, st.cnt, st.p) == (ref["state"].t, ref["state"].cnt, ref["state"].p), rep
            eng.local_steps(3)                       # eager work between the replays
            eng.average()
            torch.cuda.synchronize()
        tm = eng.get_timing()
        assert (tm.graph_captures, tm.graph_replays) == (1, 4)
        # another start state is captured again, and matches the oracle
        eng.reset()
        eng.local_steps(5)
        r0 = eng.get_state()
        recs, var, n = eng.run(40)
        tm = eng.get_timing()
        assert (tm.graph_captures, tm.graph_replays) == (2, 5)
        x = eng.x.double().cpu().numpy()
    o = oracle.Oracle(w)
    h, xs = o.problem_data()
    xo, vo = np.zeros((w.K, w.P)), np.zeros((w.K, w.P))
    for t in range(5):
        o.local_step(t, xo, vo, h, xs)
    ost = OO._State(t=5, cnt=r0.cnt, nC2=0, C2=0.0, p=r0.p)
    r = o.run(n_steps=40, h=h, xs=xs, x=xo, v=vo, state=ost)
    assert_same_syncs(recs, r, w)
    assert max_rel_err(x, r.x, w.offsets()) < PARAM_TOL


@pytest.mark.parametrize("key,fused", [("resnet18_like", True), ("many_small", True),
                                       ("quad_small", True), ("resnet18_like", False)])
def test_manual_algorithm2_loop_equals_run(A, key, fused):
    """Algorithm 2 driven by hand through the primitive calls (p - 1 local steps,
    then the period's last step fused with the sync, or p local steps and a
    separate sync; then the host scheduler on the returned variances) takes the
    same syncs and computes the same replicas and momenta as adpsgd_run."""
    w = W.parity_workloads()[key]
    N = w.total_steps
    _say(f"manual loop {key} fused={fused}: K={w.K} P={w.P} N={N}")
    g = gpu_run(w)
    t_list, p_list, S_list, var_list = [], [], [], []
    with A.Adpsgd.from_workload(w) as eng:
        p, t = w.p_init, 0
        while t + p <= N:
            if fused:
                eng.local_steps(p - 1)
                var = eng.step_average()
            else:
                eng.local_steps(p)
                var = eng.average()
            t_list.append(t + p - 1); p_list.append(p)
            S_list.append(float(np.sum(var))); var_list.append(var)
            t += p
            p = eng.schedule(var)
        eng.local_steps(N - t)
        st = eng.get_state()
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
    recs = g["recs"]
    assert len(t_list) == g["n_syncs"]
    assert np.array_equal(recs["t"], t_list) and np.array_equal(recs["p"], p_list)
    assert np.array_equal(x, g["x"]) and np.array_equal(m, g["m"])
    assert np.allclose(np.asarray(var_list), g["var"], rtol=1e-12, atol=0.0)
    assert np.allclose(S_list, recs["S"], rtol=1e-12, atol=0.0)
    assert (st.t, st.cnt, st.p, st.nC2) == (g["state"].t, g["state"].cnt, g["state"].p, g["state"].nC2)
    assert st.C2 == pytest.approx(g["state"].C2, rel=1e-12)


STEP_SHAPES = [(64, 0, 1), (64, 8192, 1), (128, 0, 1), (256, 0, 1), (64, 8192, 16), (64, 8192, 32),
               (64, 8192, 64), (256, 65536, 1), (128, 0, 4096), (64, 0, 3)]
TIMED_SHAPES = STEP_SHAPES[:7]


@pytest.mark.parametrize("case", ["resnet18_like", "k5_packed_ragged"])
def test_step_launch_shapes_agree_bitwise(A, case):
    """The plain local step in every launch shape (the init-time choice among
    them depends on timing) computes the same bits; also with an odd K and
    rows packed at a P that is not a multiple of 4 (scalar accesses)."""
    w = W.parity_workloads()["resnet18_like"].replace(total_steps=200, k_s=50)
    pad = True
    if case == "k5_packed_ragged":
        w = w.replace(K=5, sizes=w.sizes[:-1] + (w.sizes[-1] + 3,))
        assert w.P % 4 != 0
        pad = False
    runs = {}
    for shape in STEP_SHAPES:
        with A.Adpsgd.from_workload(w, pad_rows=pad) as eng:
            eng.set_step_launch(*shape)
            assert eng.step_launch == shape
            recs, var, n = eng.run(w.total_steps)
            runs[shape] = (recs.tobytes(), var.tobytes(), eng.x.cpu().numpy().tobytes(),
                           eng.m.cpu().numpy().tobytes())
        with pytest.raises(A.AdpsgdError):
            A.adpsgd_set_step_launch(0, *shape)   # a NULL context is refused
    assert all(runs[s] == runs[STEP_SHAPES[0]] for s in STEP_SHAPES)
    if case != "resnet18_like":
        return
    with A.Adpsgd.from_workload(w) as eng:
        tuned = eng.step_launch
        assert tuned in TIMED_SHAPES
        for bad in [(96, 0, 1), (64, -1, 1), (64, 65537, 1), (64, 0, 0), (64, 0, 4097)]:
            with pytest.raises(A.AdpsgdError) as e:
                eng.set_step_launch(*bad)
            assert e.value.code == A.EINVAL
            assert eng.step_launch == tuned
        eng.set_step_launch(256, 4096, 2)
        eng.set_step_launch(0, 123, 0)             # back to the timed choice
        assert eng.step_launch == tuned


N_RANDOM_SMALL_K, N_RANDOM_LARGE_K = 128, 32


def _random_workload(i):
    """A seeded random small configuration: K (the first 128 cases up to 32,
    the next 32 from 25 to 65: two and four rows per wave with ragged last
    waves, and the loop kernel), 1-11 ragged tensors (empty ones included),
    period mode, LR schedule, warm-up prefix, period switch and momentum
    averaging."""
    rng = np.random.default_rng(7000 + i)
    ks = [1, 2, 3, 4, 5, 7, 8, 12, 16, 24, 32] if i < N_RANDOM_SMALL_K else [25, 31, 33, 48, 64, 65]
    K = int(rng.choice(ks))
    T = int(rng.integers(1, 12))
    sizes = [int(s) for s in rng.integers(0, 6000, size=T)]
    if sum(sizes) == 0:
        sizes[-1] = 17
    mode = int(rng.choice([W.PERIOD_CONST, W.PERIOD_ADAPTIVE, W.PERIOD_ALG1]))
    N = int(rng.integers(24, 90))
    kw = dict(name=f"random{i}", K=K, sizes=tuple(sizes), seed=100 + i,
              sigma=float(rng.uniform(0.01, 0.3)), momentum=float(rng.choice([0.0, 0.5, 0.9])),
              weight_decay=float(rng.choice([0.0, 1e-4, 5e-4])), h_lo=1e-2, h_hi=1.0,
              lr_kind=int(rng.choice([W.LR_CONST, W.LR_STEP, W.LR_COSINE, W.LR_WARMUP_STEP])),
              lr0=float(rng.uniform(0.01, 0.1)), total_steps=N, period_mode=mode,
              p_init=int(rng.integers(1, 7)),
              k_s=int(rng.integers(0, N // 2)) if mode == W.PERIOD_ADAPTIVE else 0,
              sync_warmup_steps=int(rng.choice([0, 0, 4])), avg_momentum=bool(rng.integers(0, 2)))
    if mode != W.PERIOD_ADAPTIVE and rng.integers(0, 2):
        kw.update(p_switch_step=N // 2, p_after=int(rng.integers(1, 7)))
    return W.Workload(**kw)


@pytest.mark.parametrize("i", range(N_RANDOM_SMALL_K + N_RANDOM_LARGE_K))
def test_random_workloads_match_oracle(A, i):
    """128 seeded random configurations against the oracle (x, m, the sync
    list, S and the per-tensor variances).  The closest decision of these seeds
    lies 5e-4 from a threshold (seed 50, where S is within 2.4e-7 of the
    oracle's); the others at least 1.7e-3."""
    w = _random_workload(i)
    _say(f"random {i}: K={w.K} P={w.P} T={w.T} mode={w.period_mode} N={w.total_steps}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    assert_same_syncs(g["recs"], r, w)
    assert rel_err(g["recs"]["S"], r.S, floor=1e-300) < VAR_TOL
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    assert max_rel_err(g["x"], r.x, w.offsets()) < PARAM_TOL
    assert max_rel_err(g["m"], r.v, w.offsets(), floor=MOM_FLOOR) < MOM_TOL
    assert g["state"].t == w.total_steps and g["state"].p == r.state.p


def test_package_imported_before_torch(A):
    """In a fresh process that imports this package before torch, the library
    binds to the same HIP runtime as torch (one runtime per process) and a run
    gives the same bits as here."""
    import hashlib
    import os
    import subprocess
    w = W.parity_workloads()["many_small"].replace(total_steps=40, k_s=10)
    g = gpu_run(w)
    want = hashlib.sha256(g["x"].tobytes() + g["m"].tobytes()).hexdigest()
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = (
        "import sys, hashlib\n"
        "import paper_2007_06134_amd\n"          # before torch, on purpose
        "sys.path.insert(0, 'tests')\n"
        "import workloads as W\n"
        "from helpers import gpu_run\n"
        "w = W.parity_workloads()['many_small'].replace(total_steps=40, k_s=10)\n"
        "g = gpu_run(w)\n"
        "print(hashlib.sha256(g['x'].tobytes() + g['m'].tobytes()).hexdigest())\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=240,
                       env=dict(os.environ, PYTHONPATH=root))
    assert r.returncode == 0, r.stderr[-3000:]
    assert r.stdout.strip().splitlines()[-1] == want


def _run_digest(A, w, stream=None):
    import hashlib
    import torch
    with A.Adpsgd.from_workload(w, stream=stream) as eng:
        recs, var, _ = eng.run(w.total_steps)
        eng.local_steps(3)
        v2 = eng.average()
        torch.cuda.synchronize()
        blob = eng.x.cpu().numpy().tobytes() + eng.m.cpu().numpy().tobytes() + recs.tobytes()
    return hashlib.sha256(blob + var.tobytes() + v2.tobytes()).hexdigest()


def test_side_streams_and_concurrent_contexts_agree_bitwise(A):
    """A context on a non-default stream (current, or passed while the default
    one is current), and several contexts on their own streams driven from as
    many host threads at once, give the bits of a default-stream run: all work
    of a context is ordered on its stream."""
    import threading
    import torch
    ws = [W.parity_workloads()[k].replace(total_steps=120, k_s=30)
          for k in ("resnet18_like", "many_small", "vgg16_adaptive")]
    base = [_run_digest(A, w) for w in ws]
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        assert [_run_digest(A, w, stream=side) for w in ws] == base
    assert [_run_digest(A, w, stream=side) for w in ws] == base
    for _ in range(2):
        out = {}

        def worker(j):
            out[j] = _run_digest(A, ws[j], stream=torch.cuda.Stream())

        threads = [threading.Thread(target=worker, args=(j,)) for j in range(len(ws))]
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        assert [out.get(j) for j in range(len(ws))] == base


@pytest.mark.parametrize("mode", [W.PERIOD_CONST, W.PERIOD_ADAPTIVE])
def test_last_steps_before_the_counter_limit(A, mode):
    """Steps up to t = 2^32 - 1 (the last value of the Philox counter word that
    holds the step) match the oracle from a restored state; one step more is
    refused and leaves the context unchanged."""
    import oracle.oracle as OO
    w = _tiny(K=4, sizes=(3001, 17), period_mode=mode, p_init=3, k_s=0, total_steps=1000)
    t0 = 2**32 - 20
    with A.Adpsgd.from_workload(w) as eng:
        st = eng.get_state()
        st.t, st.cnt, st.p, st.C2, st.nC2 = t0, 1, 3, 2e-4, 5
        eng.set_state(st)
        recs, var, n = eng.run(20)
        assert eng.get_state().t == 2**32
        with pytest.raises(A.AdpsgdError) as e:
            eng.local_steps(1)
        assert e.value.code == A.EINVAL and eng.get_state().t == 2**32
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
    o = oracle.Oracle(w)
    ost = OO._State(t=t0, cnt=1, nC2=5, C2=2e-4, p=3)
    r = o.run(n_steps=20, state=ost)
    assert_same_syncs(recs, r, w)
    assert n == r.n_syncs
    assert rel_err(var, r.var, floor=1e-300) < VAR_TOL
    assert max_rel_err(x, r.x, w.offsets()) < PARAM_TOL
    assert max_rel_err(m, r.v, w.offsets(), floor=MOM_FLOOR) < MOM_TOL


def test_checkpoint_resume_is_bit_exact(A):
    import torch
    w = W.parity_workloads()["resnet18_like"].replace(total_steps=700, k_s=150)
    full = gpu_run(w)
    with A.Adpsgd.from_workload(w) as eng:
        r1, v1, n1 = eng.run(350)
        st = eng.get_state()
        x_saved, m_saved = eng.x.clone(), eng.m.clone()
    with A.Adpsgd.from_workload(w) as eng:
        eng.x.copy_(x_saved); eng.m.copy_(m_saved)
        torch.cuda.synchronize()
        eng.set_state(st)
        r2, v2, n2 = eng.run(350)
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
    assert n1 + n2 == full["n_syncs"]
    assert np.concatenate([r1, r2]).tobytes() == full["recs"].tobytes()
    assert np.array_equal(x, full["x"]) and np.array_equal(m, full["m"])


def test_timing_counts_every_launch(A):
    w = W.parity_workloads()["vgg16_adaptive"].replace(total_steps=100, k_s=20)
    with A.Adpsgd.from_workload(w) as eng:
        eng.set_timing(True)
        recs, _, n = eng.run(100)
        tm = eng.get_timing()
    # every sync runs one fused kernel and one reduction; a step the host could
    # not plan (its sync decided on the device) also runs a reduction, and is
    # timed as a plain step when it turns out not to end a period
    assert tm.fused_launches == n and tm.segsum_launches >= n
    assert tm.step_launches == 100 - n and tm.average_launches == 0
    assert tm.step_ms > 0 and tm.fused_ms > 0
    # sampled: events around every 4th launch of each kind
    with A.Adpsgd.from_workload(w) as eng:
        eng.set_timing(4)
        eng.run(100)
        ts = eng.get_timing()
        with pytest.raises(A.AdpsgdError):
            eng.set_timing(-1)
    assert 0 < ts.step_launches <= (100 - n + 3) // 4 + 2 and 0 < ts.fused_launches <= (n + 3) // 4 + 2
    assert abs(ts.step_ms / ts.step_launches - tm.step_ms / tm.step_launches) < 0.5 * tm.step_ms / tm.step_launches


# ---------------------------------------------------------------- edge cases and errors

def test_maximum_worker_count(A):
    """K = 65536, the most the library accepts, on a ragged 12-element vector:
    the any-K sync kernel walks 65536 rows and the step grid has 524288 blocks."""
    w = W.Workload(name="kmax", K=65536, sizes=(3, 9), seed=5, sigma=0.1, momentum=0.9,
                   weight_decay=5e-4, h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.05,
                   total_steps=9, period_mode=W.PERIOD_CONST, p_init=4, k_s=0)
    _say(f"maximum K: K={w.K} P={w.P}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    assert np.array_equal(g["recs"]["t"], r.sync_t)
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    assert max_rel_err(g["x"], r.x, w.offsets()) < PARAM_TOL
    assert max_rel_err(g["m"], r.v, w.offsets(), floor=MOM_FLOOR) < MOM_TOL


def test_sync_log_as_json_lines(A, tmp_path):
    import json
    w = _tiny(K=4, sizes=(4096, 3), p_init=4, total_steps=20, period_mode=W.PERIOD_ADAPTIVE, k_s=8)
    with A.Adpsgd.from_workload(w) as eng:
        recs, var, n = eng.run(w.total_steps)
    path = tmp_path / "syncs.jsonl"
    assert A.write_sync_log(str(path), recs, var) == n == 5
    rows = [json.loads(line) for line in path.read_text().splitlines()]
    assert [r["t"] for r in rows] == list(recs["t"]) and rows[0]["margin"] is None
    assert np.allclose([sum(r["var"]) for r in rows], recs["S"], rtol=1e-12)


def test_destroyed_context_is_refused(A):
    """A call with a destroyed context returns EINVAL instead of touching freed
    memory, and a second destroy is refused."""
    w = _tiny(K=2, sizes=(1024,))
    eng = A.Adpsgd.from_workload(w)
    raw = eng.ctx
    eng.close()
    lib = A._native.lib
    assert lib.adpsgd_local_steps(raw, 1) == A.EINVAL
    assert "not a live context" in A.adpsgd_last_error()
    assert lib.adpsgd_destroy(raw) == A.EINVAL


def test_divergence_surfaces_through_a_separate_sync(A):
    """A diverging run: the separate sync reports non-finite variances and the
    controller refuses them with ENONFINITE, p unchanged."""
    w = _tiny(K=4, sizes=(4096,), lr0=50.0, p_init=5, total_steps=200,
              period_mode=W.PERIOD_ADAPTIVE, k_s=0)
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(60)
        var = eng.average()
        assert not np.all(np.isfinite(var))
        with pytest.raises(A.AdpsgdError) as e:
            eng.schedule(var)
        assert e.value.code == A.ENONFINITE and eng.get_state().p == 5


def test_empty_parameter_vector(A):
    w = _tiny(K=4, sizes=(0, 0), p_init=3, total_steps=10)
    with A.Adpsgd.from_workload(w) as eng:
        recs, var, n = eng.run(10)
    assert n == 3 and np.all(var == 0.0) and np.all(recs["S"] == 0.0)


def test_single_worker_has_zero_variance(A):
    w = _tiny(K=1, sizes=(777, 4096), p_init=4, total_steps=30,
              period_mode=W.PERIOD_ADAPTIVE, k_s=8)
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    assert np.all(g["var"] == 0.0)
    assert np.array_equal(g["recs"]["t"], r.sync_t)
    assert max_rel_err(g["x"], r.x, w.offsets()) < PARAM_TOL


def test_divergence_reports_non_finite_variance(A):
    w = _tiny(K=4, sizes=(4096,), lr0=50.0, p_init=40, total_steps=200,
              period_mode=W.PERIOD_ADAPTIVE, k_s=0)
    with A.Adpsgd.from_workload(w) as eng:
        with pytest.raises(A.AdpsgdError) as e:
            eng.run(200)
        assert e.value.code == A.ENONFINITE
        st = eng.get_state()
        assert st.p == 40 and st.t >= 40


@pytest.mark.parametrize("traced", [False, True])
@pytest.mark.parametrize("policy", ["hybrid", "device", "host"])
@pytest.mark.parametrize("mode", [W.PERIOD_CONST, W.PERIOD_ADAPTIVE, W.PERIOD_ALG1])
def test_divergence_under_every_policy(A, mode, policy, traced):
    """A diverging run (non-finite S) returns ENONFINITE, as the oracle does,
    under every launch policy, period mode and with tracing: the failing
    sync's update of p and C2 is withheld but its counter restarts, so the
    state stays consistent (cnt <= p), and the context stays usable."""
    pol = {"hybrid": A.LAUNCH_HYBRID, "device": A.LAUNCH_DEVICE, "host": A.LAUNCH_HOST}[policy]
    for K, p_init in ((3, 1), (8, 5)):
        w = _tiny(K=K, sizes=(3000, 5), lr0=50.0, p_init=p_init, total_steps=300, period_mode=mode, k_s=0)
        with pytest.raises(RuntimeError, match="-4"):
            oracle.Oracle(w).run()
        with A.Adpsgd.from_workload(w) as eng:
            eng.set_launch_policy(pol)
            with pytest.raises(A.AdpsgdError) as e:
                eng.run_traced(300) if traced else eng.run(300)
            assert e.value.code == A.ENONFINITE
            st = eng.get_state()
            assert 0 < st.t <= 300 and st.cnt <= st.p
            eng.reset()
            recs, _, n = eng.run(5)
            assert eng.get_state().t == 5


def test_invalid_calls_leave_context_unchanged(A):
    import torch
    w = _tiny(K=2, sizes=(1024,))
    with A.Adpsgd.from_workload(w) as eng:
        with pytest.raises(A.AdpsgdError) as e:
            eng.schedule(np.zeros(1))
        assert e.value.code == A.ESTATE
        for bad in (-1,):
            with pytest.raises(A.AdpsgdError):
                eng.local_steps(bad)
        with pytest.raises(A.AdpsgdError) as e:
            eng.set_launch_policy(7)
        assert e.value.code == A.EINVAL
        st = eng.get_state()
        bad_state = A.adpsgd_state(t=-1, cnt=0, nC2=0, C2=0.0, p=1)
        with pytest.raises(A.AdpsgdError):
            eng.set_state(bad_state)
        assert eng.get_state().t == st.t
        # a misaligned replica pointer is refused before anything runs
        buf = A.adpsgd_buffers(x=eng.x.data_ptr() + 4, m=eng.m.data_ptr(), h=eng.h.data_ptr(),
                               xstar=eng.xstar.data_ptr(), workspace=eng.workspace.data_ptr(),
                               workspace_bytes=eng.workspace.numel(),
                               stream=torch.cuda.current_stream().cuda_stream)
        with pytest.raises(A.AdpsgdError) as e:
            A.adpsgd_init(2, 1024, [0, 1024], eng.hp, buf)
        assert e.value.code == A.EINVAL


# ---------------------------------------------------------------- schedule and state variants

def _variant(name):
    base = W.parity_workloads()["resnet18_like"]      # K = 8, 62 ragged tensors, P = 40,000
    v = {
        # Section IV-C: gradual warm-up LR, p = 1 for the first 8 of 90 epochs, K_s = 0.2 N
        "imagenet_warmup": dict(total_steps=900, lr_kind=W.LR_WARMUP_STEP, lr0=0.1,
                                sync_warmup_steps=80, period_mode=W.PERIOD_ADAPTIVE, p_init=4, k_s=180),
        # Algorithm 1's sync test (after steps 0, p, 2p, ...)
        "alg1": dict(total_steps=300, period_mode=W.PERIOD_ALG1, p_init=6, k_s=0),
        # Section III-A strategy 1 (4, then 8) and Section V-B (20, then 5)
        "two_phase_up": dict(total_steps=400, period_mode=W.PERIOD_CONST, p_init=4, k_s=0,
                             p_switch_step=200, p_after=8),
        "two_phase_down": dict(total_steps=400, period_mode=W.PERIOD_CONST, p_init=20, k_s=0,
                               p_switch_step=200, p_after=5),
        "avg_momentum_adaptive": dict(total_steps=600, avg_momentum=True, k_s=150),
        "avg_momentum_k3": dict(K=3, total_steps=300, avg_momentum=True, period_mode=W.PERIOD_CONST,
                                p_init=5, k_s=0),
        "avg_momentum_k32": dict(K=32, total_steps=200, avg_momentum=True, period_mode=W.PERIOD_CONST,
                                 p_init=3, k_s=0),
        "avg_momentum_k24": dict(K=24, total_steps=200, avg_momentum=True, k_s=50),
        # an upper bound on p (p within [1, p_max]): p would reach 10 after the
        # LR decays of this run and is held at 3
        "p_max_cap": dict(p_max=3),
        "p_max_cap_k16": dict(K=16, p_init=4, p_max=6),
    }[name]
    return base.replace(name=name, **v)


@pytest.mark.parametrize("name", ["imagenet_warmup", "alg1", "two_phase_up", "two_phase_down",
                                  "avg_momentum_adaptive", "avg_momentum_k3", "avg_momentum_k32",
                                  "avg_momentum_k24", "p_max_cap", "p_max_cap_k16"])
def test_variant_run_matches_oracle(A, name):
    w = _variant(name)
    _say(f"variant {name}: K={w.K} P={w.P} N={w.total_steps}")
    g = gpu_run(w)
    r = oracle.Oracle(w).run()
    recs = g["recs"]
    assert_same_syncs(recs, r, w)
    assert rel_err(g["var"], r.var, floor=1e-300) < VAR_TOL
    off = w.offsets()
    ex, em = max_rel_err(g["x"], r.x, off), max_rel_err(g["m"], r.v, off, floor=MOM_FLOOR)
    _say(f"  {name}: {r.n_syncs} syncs, p {r.sync_p.min()}..{r.sync_p.max()}, err x {ex:.2e} m {em:.2e}")
    if w.p_max:
        assert r.sync_p.max() == w.p_max, "the cap must bind in this case"
    assert ex < PARAM_TOL and em < MOM_TOL
    assert g["state"].p == r.state.p and g["state"].cnt == r.state.cnt
    if w.avg_momentum and w.period_mode == W.PERIOD_CONST and w.total_steps % w.p_init == 0:
        m = g["m"]
        assert all(np.array_equal(m[k], m[0]) for k in range(w.K))   # synced at the last step


@pytest.mark.parametrize("K", [3, 5, 8, 12, 24, 25, 32, 33, 64, 65])
def test_separate_sync_averages_momentum(A, K):
    w = _tiny(K=K, sizes=(5000, 3, 0, 5001), avg_momentum=True)
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(6)
        var = eng.average()
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
    o = oracle.Oracle(w)
    r = o.run(n_steps=6)
    S_o, var_o = o.average(r.x, v=r.v)
    off = w.offsets()
    assert all(np.array_equal(m[k], m[0]) for k in range(K))
    assert max_rel_err(x, r.x, off) < PARAM_TOL
    assert max_rel_err(m, r.v, off, floor=MOM_FLOOR) < MOM_TOL
    nz = np.diff(off) > 0
    assert rel_err(var[nz], var_o[nz]) < VAR_TOL


# ---------------------------------------------------------------- traced runs

def _traced_cases():
    pw = W.parity_workloads()
    return {
        "resnet18_like": pw["resnet18_like"].replace(total_steps=1200, k_s=300),
        "many_small": pw["many_small"].replace(total_steps=800, k_s=200),
        "k3_const": _tiny(K=3, sizes=(5000, 3, 0, 5001), p_init=5, total_steps=60),
        "k24_adaptive": _tiny(K=24, sizes=(5000, 3, 0, 5001), p_init=2, total_steps=80,
                              period_mode=W.PERIOD_ADAPTIVE, k_s=20),
        "vgg16_adaptive": pw["vgg16_adaptive"],
    }


@pytest.mark.parametrize("key", list(_traced_cases()))
def test_traced_run_matches_oracle(A, key):
    w = _traced_cases()[key]
    _say(f"traced {key}: K={w.K} P={w.P} N={w.total_steps}")
    with A.Adpsgd.from_workload(w) as eng:
        recs, var, n, steps = eng.run_traced(w.total_steps)
    r = oracle.Oracle(w).run(trace=True)
    assert_same_syncs(recs, r, w)
    assert np.array_equal(steps["t"], np.arange(w.total_steps))
    assert np.array_equal(np.nonzero(steps["synced"])[0], r.sync_t)
    ev, eg = rel_err(steps["var"], r.trace_var), rel_err(steps["grad_norm2"], r.trace_grad_norm2)
    _say(f"  per-step variance err {ev:.2e}, gradient norm err {eg:.2e}")
    assert ev < VAR_TOL and eg < VAR_TOL
    np.testing.assert_array_equal(steps["var"][recs["t"]], recs["S"])


@pytest.mark.parametrize("key", ["resnet18_like", "k3_const"])
def test_traced_run_equals_plain_run(A, key):
    import torch
    w = _traced_cases()[key]
    with A.Adpsgd.from_workload(w) as a, A.Adpsgd.from_workload(w) as b:
        ra, va, na = a.run(w.total_steps)
        rb, vb, nb, _ = b.run_traced(w.total_steps)
        assert torch.equal(a.x, b.x) and torch.equal(a.m, b.m)
    assert na == nb and ra.tobytes() == rb.tobytes() and np.array_equal(va, vb)
