"""Random sequences of the primitive calls against the oracle driven the same way.

Each case draws a small workload and 25 calls among adpsgd_local_steps,
adpsgd_step_average, adpsgd_average, adpsgd_schedule (on the variances the last
sync returned), adpsgd_run, and checkpoints (adpsgd_get_state with copies of x
and m, restored later through adpsgd_set_state).  The oracle is driven through
its own primitives in the same order.  After every call the controller state
(t, cnt, p, nC2, C2) must agree, every sync's per-tensor variances and every
run's sync list too, and at the end x and m.
"""
import sys

import numpy as np
import pytest

import oracle
import oracle.oracle as OO
import workloads as W
from helpers import MOM_FLOOR, MOM_TOL, PARAM_TOL, max_rel_err, rel_err

pytestmark = pytest.mark.gpu

# A sync right after a sync gives exactly 0 on the GPU (the pairwise mean of
# equal rows is exact) and ~1e-32 in the oracle's sequential fp64 sum, so
# variances, and C2 sampled from them, are compared with an absolute floor.
ZERO_FLOOR = 1e-20


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def A():
    import torch
    assert torch.cuda.is_available()
    import paper_2007_06134_amd as A
    return A


def _case(i):
    rng = np.random.default_rng(50000 + i)
    K = int(rng.choice([1, 2, 3, 4, 8, 16, 32]))
    T = int(rng.integers(1, 6))
    sizes = [int(s) for s in rng.integers(0, 3000, size=T)]
    if sum(sizes) == 0:
        sizes[-1] = 9
    mode = int(rng.choice([W.PERIOD_CONST, W.PERIOD_ADAPTIVE, W.PERIOD_ADAPTIVE, W.PERIOD_ALG1]))
    kw = dict(name=f"calls{i}", K=K, sizes=tuple(sizes), seed=int(rng.integers(0, 2**31)),
              sigma=float(rng.uniform(0.02, 0.2)), momentum=float(rng.choice([0.0, 0.9])),
              weight_decay=float(rng.choice([0.0, 5e-4])), h_lo=1e-2, h_hi=1.0,
              lr_kind=int(rng.choice([W.LR_CONST, W.LR_STEP, W.LR_COSINE])), lr0=float(rng.uniform(0.01, 0.1)),
              total_steps=200, period_mode=mode, p_init=int(rng.integers(1, 6)),
              k_s=int(rng.integers(0, 40)) if mode == W.PERIOD_ADAPTIVE else 0,
              sync_warmup_steps=int(rng.choice([0, 0, 5])), avg_momentum=bool(rng.integers(0, 2)))
    if mode != W.PERIOD_ADAPTIVE and rng.integers(0, 2):
        kw.update(p_switch_step=int(rng.integers(1, 120)), p_after=int(rng.integers(1, 6)))
    return W.Workload(**kw), rng


class _OracleSide:
    """The oracle's replicas, momenta and controller state, moved by the same calls."""

    def __init__(self, w):
        self.w, self.o = w, oracle.Oracle(w)
        self.h, self.xs = self.o.problem_data()
        self.x = np.zeros((w.K, w.P))
        self.v = np.zeros((w.K, w.P))
        self.st = self.o.new_state()

    def _switch(self, t):
        w = self.w
        if w.period_mode != W.PERIOD_ADAPTIVE and w.p_switch_step > 0 and t >= w.p_switch_step:
            self.st.p = w.p_after

    def local_steps(self, n):
        for t in range(self.st.t, self.st.t + n):
            self.o.local_step(t, self.x, self.v, self.h, self.xs)
        self.st.t += n
        self.st.cnt += n
        self._switch(self.st.t - 1)

    def sync(self, fused):
        if fused:
            self.o.local_step(self.st.t, self.x, self.v, self.h, self.xs)
            self._switch(self.st.t)
            self.st.t += 1
        _, var = self.o.average(self.x, None, self.v if self.w.avg_momentum else None)
        self.st.cnt = 0
        return var

    def schedule(self, var):
        self.st.cnt = 0
        self.o.controller(self.st, self.st.t - 1, float(np.sum(var)))
        return self.st.p

    def run(self, n):
        return self.o.run(n_steps=n, h=self.h, xs=self.xs, x=self.x, v=self.v, state=self.st)

    def save(self):
        s = self.st
        return (OO._State(t=s.t, cnt=s.cnt, nC2=s.nC2, C2=s.C2, p=s.p), self.x.copy(), self.v.copy())

    def restore(self, saved):
        s = saved[0]
        self.st = OO._State(t=s.t, cnt=s.cnt, nC2=s.nC2, C2=s.C2, p=s.p)
        self.x, self.v = saved[1].copy(), saved[2].copy()


@pytest.mark.parametrize("i", range(64))
def test_random_call_sequence_matches_oracle(A, i):
    import torch
    w, rng = _case(i)
    ref = _OracleSide(w)
    ops = []
    saved = None
    var_gpu = var_ref = None
    with A.Adpsgd.from_workload(w) as eng:
        for _ in range(25):
            t = int(eng.get_state().t)
            room = w.total_steps - 1 - t
            if room < 2:
                break
            op = str(rng.choice(["local", "local", "stepavg", "avg", "sched", "run", "run", "save", "restore"]))
            if op == "local":
                n = int(rng.integers(1, min(6, room)))
                eng.local_steps(n)
                ref.local_steps(n)
                ops.append(f"local({n})")
            elif op in ("stepavg", "avg"):
                var_gpu = eng.step_average() if op == "stepavg" else eng.average()
                var_ref = ref.sync(op == "stepavg")
                ops.append(op)
                assert rel_err(var_gpu, var_ref, floor=ZERO_FLOOR) < 1e-3, ops
            elif op == "sched":
                if t < 1 or var_gpu is None:
                    continue
                p = eng.schedule(var_gpu)
                ops.append(f"schedule->{p}")
                assert p == ref.schedule(var_ref), ops
            elif op == "run":
                n = int(rng.integers(1, min(25, room)))
                recs, _, ns = eng.run(n)
                r = ref.run(n)
                ops.append(f"run({n})->{ns}")
                assert ns == r.n_syncs and np.array_equal(recs["t"], r.sync_t), ops
                assert np.array_equal(recs["p"], r.sync_p), ops
            elif op == "save":
                saved = (eng.get_state(), eng.x.clone(), eng.m.clone(), ref.save())
                ops.append("save")
            elif saved is not None:
                eng.set_state(saved[0])
                eng.x.copy_(saved[1])
                eng.m.copy_(saved[2])
                torch.cuda.synchronize()
                ref.restore(saved[3])
                ops.append("restore")
            st = eng.get_state()
            assert (st.t, st.cnt, st.p, st.nC2) == (ref.st.t, ref.st.cnt, ref.st.p, ref.st.nC2), ops
            assert rel_err([st.C2], [ref.st.C2], floor=ZERO_FLOOR) < 1e-3, ops
        x = eng.x.double().cpu().numpy()
        m = eng.m.double().cpu().numpy()
    _say(f"calls {i}: K={w.K} P={w.P} mode={w.period_mode}: {' '.join(ops)}")
    assert max_rel_err(x, ref.x, w.offsets()) < PARAM_TOL
    assert max_rel_err(m, ref.v, w.offsets(), floor=MOM_FLOOR) < MOM_TOL


def test_period_switch_applies_to_the_state_of_manual_calls(A):
    """A constant period that switches at p_switch_step does so for the state
    that adpsgd_local_steps and adpsgd_step_average leave, as it does in a run;
    adpsgd_schedule then reports the new period."""
    w = W.Workload(name="switch", K=4, sizes=(1000,), seed=5, sigma=0.1, momentum=0.9, weight_decay=0.0,
                   h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.05, total_steps=100,
                   period_mode=W.PERIOD_CONST, p_init=4, k_s=0, p_switch_step=10, p_after=2)
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(10)                      # steps 0..9: before the switch
        assert eng.get_state().p == 4
        var = eng.step_average()                 # step 10: the switch
        assert eng.get_state().p == 2 and eng.schedule(var) == 2
    with A.Adpsgd.from_workload(w) as eng:
        eng.local_steps(11)                      # steps 0..10
        assert eng.get_state().p == 2
        recs, _, n = eng.run(6)                  # cnt = 11 >= 2: a sync after step 11, then 13, 15
        assert list(recs["t"]) == [11, 13, 15] and list(recs["p"]) == [2, 2, 2]
