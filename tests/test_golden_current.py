"""The stored full-size oracle runs (tests/golden/fullsize_<workload>.npz) still
equal what the oracle computes now (CPU).

The full-size GPU tests compare against these files, which the oracle wrote
offline (make_fullsize_golden.py): an edit of the oracle's arithmetic would
leave them comparing against stale numbers.  Each test recomputes the first
sync of a stored run with the current oracle: its step, its S and every
per-tensor variance (Algorithm 2's steps and sync).  For the three 138M-parameter runs
(4.4e9 updates to their first sync) the oracle replays the 26 tensors of at
most 1e6 elements: the first sync follows step p_init - 1 before any decision,
so its schedule does not depend on the data and a subset replay is exact.
"""
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _stored(key):
    path = os.path.join(GOLDEN, f"fullsize_{key}.npz")
    if not os.path.exists(path):
        pytest.skip(f"no stored run for {key}")
    return np.load(path)


@pytest.mark.parametrize("key", ["resnet18_like", "many_small", "resnet50_like"])
def test_first_sync_of_stored_run_is_current(key):
    g = _stored(key)
    w = W.full_workloads()[key]
    t0 = int(g["sync_t"][0])
    r = oracle.Oracle(w).run(n_steps=t0 + 1, log_cap=1)
    assert r.n_syncs == 1 and int(r.sync_t[0]) == t0 and int(r.sync_p[0]) == int(g["sync_p"][0])
    np.testing.assert_allclose(r.S[0], g["S"][0], rtol=1e-13, atol=0)
    np.testing.assert_allclose(r.var[0], g["var"][0], rtol=1e-13, atol=0)
    assert r.C2[0] == pytest.approx(float(g["C2"][0]), rel=1e-13)


@pytest.mark.parametrize("key", ["vgg16_adaptive", "vgg16_const8", "vgg16_stepdecay"])
def test_first_sync_of_stored_138m_run_is_current_on_small_tensors(key):
    g = _stored(key)
    w = {**W.full_workloads(), **W.fullsize_variants()}[key]
    t0 = int(g["sync_t"][0])
    assert t0 == w.p_init - 1
    wc = w.replace(period_mode=W.PERIOD_CONST, k_s=0)       # the same first sync, no decision
    off = w.offsets()
    small = [tau for tau in range(w.T) if 0 < off[tau + 1] - off[tau] <= 1_000_000]
    idx = np.concatenate([np.arange(off[tau], off[tau + 1]) for tau in small]).astype(np.int64)
    r = oracle.Oracle(wc).run(n_steps=t0 + 1, idx=idx, log_cap=1)
    assert r.n_syncs == 1 and int(r.sync_t[0]) == t0
    np.testing.assert_allclose(r.var[0][small], g["var"][0][small], rtol=1e-13, atol=0)
