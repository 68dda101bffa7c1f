"""Full-size runs on cuda:0, in the launch configuration the bench times.

The oracle cannot replay a whole run of 1e11-1e12 element updates during a
test, so these tests check, at full size:

* against the oracle's own whole runs, stored offline
  (tests/golden/fullsize_<workload>.npz, written by make_fullsize_golden.py
  from the oracle alone): every sync's step, period, S, C2 and per-tensor
  variances, and the replicas and momenta at sampled elements;
* the replica mean at sampled elements.  Syncs preserve the mean of x and of
  m, and the dynamics are affine, so the mean follows one momentum-SGD run on
  the K-averaged noise whatever the sync schedule (adaptive runs included);
* with a constant period the schedule is known in advance, so the oracle
  replays any set of elements exactly: every tensor of up to 1e6 elements
  whole (x, m and its variance at every sync), and dense windows at every
  tensor boundary and at every multiple of 2^28 of the flat replica index, on
  every worker's row;
* the controller's decisions, recomputed from the reported S values.
"""
import os
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from helpers import MOM_FLOOR, MOM_TOL, PARAM_TOL, VAR_TOL, max_rel_err, rel_err, sync_mismatch

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
WHOLE_MAX = 1_000_000    # constant period: tensors up to this size are replayed whole
WINDOW = 64              # elements on each side of a boundary


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _sample(w, whole_max=0, row_stride=None, seed=0):
    """Sorted element indices and the tensors they cover whole.

    Tensors of at most whole_max elements are taken whole; of the others, both
    ends, WINDOW elements on each side of every tensor boundary and random
    interior elements.  With row_stride (the distance between rows of x and
    m in the device buffer), also WINDOW elements on each side of every
    element whose flat index k * row_stride + i is a multiple of 2^28 in some
    row k (byte offsets 2^30, 2^31, 2^32 ... of the replica buffer)."""
    rng = np.random.default_rng(seed)
    off = w.offsets()
    idx, whole = [], []
    per_tensor = max(4, 2048 // w.T)
    for tau in range(w.T):
        lo, hi = int(off[tau]), int(off[tau + 1])
        if hi - lo <= whole_max:
            idx.append(np.arange(lo, hi)); whole.append(tau)
        else:
            idx.append(np.arange(max(0, lo - WINDOW), min(w.P, lo + WINDOW)))
            idx.append(np.arange(max(0, hi - WINDOW), min(w.P, hi + WINDOW)))
            idx.append(rng.integers(lo, hi, size=min(per_tensor, hi - lo)))
    if row_stride:
        step = 1 << 28
        for k in range(w.K):
            first = (k * row_stride + step - 1) // step * step
            for f in range(first, k * row_stride + w.P, step):
                i = f - k * row_stride
                idx.append(np.arange(max(0, i - WINDOW), min(w.P, i + WINDOW)))
    idx = np.unique(np.concatenate(idx)).astype(np.int64)
    return idx, whole


def _check_controller(w, recs):
    t, p, S, gamma = recs["t"], recs["p"], recs["S"], recs["gamma"]
    assert len(t) > 0 and t[0] == w.p_init - 1 and p[0] == w.p_init
    assert np.all(np.diff(t) == p[1:]), "each period must last p steps"
    if w.period_mode == W.PERIOD_CONST:
        assert np.all(p == w.p_init)
        return
    C2, n = 0.0, 0
    for j in range(len(t) - 1):
        if t[j] < w.k_s:
            n += 1
            C2 += (S[j] / gamma[j] - C2) / n
            assert p[j + 1] == p[j]
            assert recs["C2"][j] == pytest.approx(C2, rel=1e-12)
        elif S[j] < w.thr_lo * gamma[j] * C2:
            assert p[j + 1] == p[j] + 1
        elif S[j] > w.thr_hi * gamma[j] * C2:
            assert p[j + 1] == max(p[j] - 1, 1)
        else:
            assert p[j + 1] == p[j]


@pytest.fixture(scope="module")
def A():
    import torch
    assert torch.cuda.is_available()
    import paper_2007_06134_amd as A
    return A


@pytest.mark.parametrize("key", list(W.full_workloads()))
def test_full_size_run(A, key):
    import torch
    w = W.full_workloads()[key]
    const = w.period_mode == W.PERIOD_CONST
    with A.Adpsgd.from_workload(w) as eng:
        # whole tensors and dense windows where the oracle can replay them (constant period)
        idx, whole = _sample(w, whole_max=WHOLE_MAX if const else 0, row_stride=eng.row_stride if const else None)
        _say(f"full size {key}: K={w.K} P={w.P} T={w.T} N={w.total_steps}; {len(idx)} sampled elements, "
             f"{len(whole)} whole tensors")
        it = torch.from_numpy(idx).cuda()
        recs, var, n = eng.run(w.total_steps)
        xs_sel = eng.x.index_select(1, it).double().cpu().numpy()
        ms_sel = eng.m.index_select(1, it).double().cpu().numpy()
    _say(f"  {n} syncs, p {recs['p'].min()}..{recs['p'].max()}")
    assert n == len(recs) and np.all(np.isfinite(recs["S"]))
    np.testing.assert_allclose(var.sum(axis=1), recs["S"], rtol=1e-12)
    _check_controller(w, recs)

    o = oracle.Oracle(w)
    xbar, vbar = o.mean_trajectory(w.total_steps, idx=idx)
    sub_off = np.searchsorted(idx, w.offsets())
    assert max_rel_err(xs_sel.mean(axis=0), xbar, sub_off) < PARAM_TOL
    # the mean of K momenta cancels most of their noise; its error comes from
    # the replicas, so it is judged on the replicas' rms
    assert max_rel_err(ms_sel.mean(axis=0), vbar, sub_off, floor=MOM_FLOOR, scale_of=ms_sel) < MOM_TOL

    if const:
        _say(f"  oracle replay of {len(idx)} elements x {w.K} workers x {w.total_steps} steps")
        r = o.run(idx=idx)
        assert np.array_equal(recs["t"], r.sync_t)
        ex = max_rel_err(xs_sel, r.x, sub_off)
        em = max_rel_err(ms_sel, r.v, sub_off, floor=MOM_FLOOR)
        ev = max((rel_err(var[:, tau], r.var[:, tau]) for tau in whole), default=0.0)
        _say(f"  every worker's row at {len(idx)} elements: err x {ex:.2e} m {em:.2e}; variance of the "
             f"{len(whole)} whole tensors at all {n} syncs: {ev:.2e}")
        assert ex < PARAM_TOL and em < MOM_TOL and ev < VAR_TOL


def _period_means(steps, sync_t, N):
    """V_t of eq. (vt): per period, the mean of Var[W_k] over its iterations
    (0 right after a sync, the traced variance of the previous step otherwise)."""
    syncs = set(int(t) for t in sync_t)
    out, cur, after_sync = [], [], True
    for t in range(N):
        cur.append(0.0 if after_sync else steps["var"][t - 1])
        after_sync = t in syncs
        if after_sync:
            out.append((t, float(np.mean(cur))))
            cur = []
    return out


def _mean_in(series, lo, hi):
    return float(np.mean([v for t, v in series if lo <= t < hi]))


def test_full_size_variance_behaviour(A):
    """The paper's Figs. 1-3 on the full ResNet18-shaped run (K = 8, P = 11.2M,
    62 tensors, 2000 steps, 10x rate decays at steps 1000 and 1500): V_t under a
    constant period 4 falls ~100x per decay (gamma^2, Section III-A); under
    ADPSGD (p_init 4, K_s 500) p rises after each decay (Fig. 3) and V_t falls
    ~10x (gamma, Section III-B), with fewer syncs."""
    w = W.full_workloads()["resnet18_like"]
    out = {}
    for name, ww in (("cpsgd4", w.replace(period_mode=W.PERIOD_CONST, p_init=4, k_s=0)),
                     ("adpsgd", w.replace(p_init=4))):
        _say(f"full-size traced {name}")
        with A.Adpsgd.from_workload(ww) as eng:
            recs, _, n, steps = eng.run_traced(ww.total_steps, with_var=False)
        out[name] = (recs, n, steps, _period_means(steps, recs["t"], ww.total_steps))
    (_, n_cp, _, v_cp), (rec_ad, n_ad, st_ad, v_ad) = out["cpsgd4"], out["adpsgd"]
    r_cp = _mean_in(v_cp, 600, 1000) / _mean_in(v_cp, 1100, 1500)
    r_ad = _mean_in(v_ad, 600, 1000) / _mean_in(v_ad, 1100, 1500)
    p = lambda lo, hi: rec_ad["p"][(rec_ad["t"] >= lo) & (rec_ad["t"] < hi)].mean()
    _say(f"  V_t drop at the first decay: CPSGD {r_cp:.1f}x, ADPSGD {r_ad:.1f}x; ADPSGD mean p "
         f"{p(500, 1000):.1f} / {p(1000, 1500):.1f} / {p(1500, 2000):.1f}; syncs {n_cp} vs {n_ad}")
    assert 30 < r_cp < 300 and 3 < r_ad < 30 and r_ad < r_cp / 3
    assert p(1000, 1500) > 2 * p(500, 1000) and p(1500, 2000) > p(1000, 1500)
    assert n_ad < n_cp
    gn = st_ad["grad_norm2"]
    assert gn[-1] < gn[999] < gn[100] < gn[0]


def test_full_size_launch_policies_agree(A):
    """The full ResNet18-shaped run (p = 1-2 for long stretches, so the default
    driver lets the device decide many steps) gives the same bits when every
    step is decided on the device and when the host waits for every decision."""
    import torch
    w = W.full_workloads()["resnet18_like"]
    out = {}
    for pol in (A.LAUNCH_HYBRID, A.LAUNCH_DEVICE, A.LAUNCH_HOST):
        _say(f"full-size resnet18_like, launch policy {pol}")
        with A.Adpsgd.from_workload(w) as eng:
            eng.set_launch_policy(pol)
            recs, var, n = eng.run(w.total_steps)
            out[pol] = (recs.tobytes(), var.tobytes(), eng.x.clone(), eng.m.clone())
    base = out[A.LAUNCH_HYBRID]
    for pol, o in out.items():
        assert o[0] == base[0] and o[1] == base[1], pol
        assert torch.equal(o[2], base[2]) and torch.equal(o[3], base[3]), pol


STORED = ["resnet18_like", "resnet50_like", "vgg16_adaptive", "many_small", "vgg16_const8", "vgg16_stepdecay"]


@pytest.mark.parametrize("key", STORED)
def test_full_size_run_matches_stored_oracle_run(A, key):
    """The whole run at full size, in the bench's launch configuration, against
    the oracle's own whole run (tests/golden/fullsize_<key>.npz, written by
    tests/golden/make_fullsize_golden.py from the oracle alone): the same
    sequence of sync steps and periods, S, C2 and every sync's per-tensor
    variances (the 102M, 16.8M and 4.1M-element tensors of the 138M runs
    included) within 1e-3, and the replicas and momenta at sampled elements.
    vgg16_stepdecay is the 138M workload under a step-decayed rate, whose
    controller moves p (the constant-rate runs keep it at p_init)."""
    import torch
    path = os.path.join(GOLDEN, f"fullsize_{key}.npz")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle run for {key} (tests/golden/make_fullsize_golden.py {key})")
    g = np.load(path)
    w = {**W.full_workloads(), **W.fullsize_variants()}[key]
    _say(f"full size {key} against the oracle's full run ({len(g['sync_t'])} syncs)")
    it = torch.from_numpy(g["idx"]).cuda()
    rows = torch.from_numpy(g["rows"]).cuda()
    with A.Adpsgd.from_workload(w) as eng:
        recs, var, n = eng.run(w.total_steps)
        xs_sel = eng.x.index_select(0, rows).index_select(1, it).double().cpu().numpy()
        ms_sel = eng.m.index_select(0, rows).index_select(1, it).double().cpu().numpy()
        st = eng.get_state()
    why = sync_mismatch(recs, g["sync_t"], g["sync_p"], g["S"], g["C2"], g["gamma"], w.thr_lo, w.thr_hi)
    assert why is None, why
    assert n == len(g["sync_t"])
    eS, eC2, ev = rel_err(recs["S"], g["S"]), rel_err(recs["C2"], g["C2"]), rel_err(var, g["var"])
    sub_off = np.searchsorted(g["idx"], w.offsets())
    ex = max_rel_err(xs_sel, g["x"], sub_off)
    em = max_rel_err(ms_sel, g["v"], sub_off, floor=MOM_FLOOR)
    margins = np.abs(recs["margin"][np.isfinite(recs["margin"])])
    _say(f"  {n} syncs identical, p {recs['p'].min()}..{recs['p'].max()}; err S {eS:.2e} C2 {eC2:.2e} "
         f"var ({var.shape[0]} syncs x {var.shape[1]} tensors) {ev:.2e} x {ex:.2e} m {em:.2e}; "
         f"closest decision {margins.min() if len(margins) else float('nan'):.2e}")
    assert eS < VAR_TOL and eC2 < VAR_TOL and ev < VAR_TOL
    assert ex < PARAM_TOL and em < MOM_TOL
    assert st.p == int(g["state_p"]) and st.nC2 == int(g["state_nC2"])


def _torch_variance(torch, x, offsets, chunk=1 << 25):
    """Per-tensor (1/K) sum_k sum_i (xbar_i - x_ki)^2 of the replicas in x [K, P],
    in fp64 on the device, chunk by chunk (an independent check at any size)."""
    K = x.shape[0]
    out = np.zeros(len(offsets) - 1)
    for tau in range(len(offsets) - 1):
        acc = 0.0
        for a in range(int(offsets[tau]), int(offsets[tau + 1]), chunk):
            b = min(a + chunk, int(offsets[tau + 1]))
            xc = x[:, a:b].double()
            acc += float(((xc - xc.mean(dim=0)) ** 2).sum())
            del xc
        out[tau] = acc / K
    return out


def test_largest_problem_in_hbm(A):
    """A problem sized to most of the GPU's memory (about 3.4e9 parameters of 8
    workers on a 288 GB MI355X): every grid is larger than one dispatch can
    hold, so the step and sync kernels run in several launches.  Checks the
    oracle at sampled elements (whole small tensors, the elements around every
    multiple of 2^28, where the launch pieces meet), the separate sync's
    variance of every tensor against an fp64 recomputation on the device, and
    that a fused sync leaves every replica equal."""
    import torch
    torch.cuda.empty_cache()
    free, _ = torch.cuda.mem_get_info()
    K = 8
    P = int(0.75 * free / (8 * K + 8.5)) // 4 * 4
    if K * P // 4 < 2 * (1 << 31):
        pytest.skip(f"{free / 2**30:.0f} GiB free: too little memory for a multi-launch grid")
    small = (1000, 7, 4093, 30001)
    big1 = P // 2 + 12345
    big2 = P - big1 - sum(small)
    sizes = (small[0], small[1], big1, small[2], big2, small[3])
    w = W.Workload(name=f"largest_k{K}", K=K, sizes=sizes, seed=11, sigma=0.02, momentum=0.9,
                   weight_decay=5e-4, h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.01, total_steps=8,
                   period_mode=W.PERIOD_CONST, p_init=3, k_s=0)
    off = w.offsets()
    assert w.P == P
    _say(f"largest problem: K={K} P={P} ({8 * K * P / 2**30:.0f} GiB of x and m, "
         f"{free / 2**30:.0f} GiB free)")
    rng = np.random.default_rng(5)
    idx = [np.arange(off[0], off[2]), np.arange(off[3], off[4]), np.arange(off[5], off[6])]
    for b in range(1 << 28, P, 1 << 28):
        idx.append(np.arange(b - 300, min(b + 300, P)))
    idx.append(rng.integers(0, P, size=4000))
    idx = np.unique(np.concatenate(idx)).astype(np.int64)
    whole = [0, 1, 3, 5]
    it = torch.from_numpy(idx).cuda()

    eng = A.Adpsgd.from_workload(w)
    try:
        eng.local_steps(2)                                   # steps 0, 1
        torch.cuda.synchronize()
        _say("  two steps done; fp64 variance on the device")
        var_ref = _torch_variance(torch, eng.x, off)
        var1 = eng.average()                                 # separate sync after step 1
        _say("  separate sync done")
        var2 = eng.step_average()                            # step 2 fused with its sync
        torch.cuda.synchronize()
        for a in range(0, P, 1 << 26):                       # every replica equals the mean
            b = min(a + (1 << 26), P)
            assert bool((eng.x[:, a:b] == eng.x[0:1, a:b]).all()), f"replicas differ in [{a}, {b})"
        eng.local_steps(1)                                   # step 3
        xs_sel = eng.x.index_select(1, it).double().cpu().numpy()
        ms_sel = eng.m.index_select(1, it).double().cpu().numpy()
    finally:
        eng.close()
        del eng
        torch.cuda.empty_cache()
    _say("  GPU part done; oracle replay of the sampled elements")
    assert rel_err(var1, var_ref) < 1e-6

    o = oracle.Oracle(w)
    h, xs = o.problem_data(idx)
    x = np.zeros((K, len(idx)))
    v = np.zeros((K, len(idx)))
    o.local_step(0, x, v, h, xs, idx)
    o.local_step(1, x, v, h, xs, idx)
    _, ov1 = o.average(x, idx)
    o.local_step(2, x, v, h, xs, idx)
    _, ov2 = o.average(x, idx)
    o.local_step(3, x, v, h, xs, idx)
    sub_off = np.searchsorted(idx, off)
    assert max_rel_err(xs_sel, x, sub_off) < PARAM_TOL
    assert max_rel_err(ms_sel, v, sub_off, floor=MOM_FLOOR) < MOM_TOL
    for tau in whole:
        assert rel_err(var1[tau], ov1[tau]) < VAR_TOL, tau
        assert rel_err(var2[tau], ov2[tau]) < VAR_TOL, tau
