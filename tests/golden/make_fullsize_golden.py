"""Writes tests/golden/fullsize_<workload>.npz from whole full-size runs of the
oracle: the adaptive workloads, whose sync schedule depends on every element
(with the 138M workload also under a step-decayed rate, which makes its
controller move p), and the constant-period 138M workload, whose three large
tensors (102M, 16.8M and 4.1M elements) are too large for the oracle to replay
during a test:

    sync_t, sync_p, S, C2, gamma   every sync of the run
    var                            per-tensor variances of every sync [n_syncs, T]
    idx, rows, x, v                replicas and momenta at sampled elements after the
                                   run: every worker for K <= 8, else workers
                                   0, 1, K/2 and K-1
    state_p, state_C2, state_nC2   the controller's final state
    oracle_source_sha256           digest of the oracle source the run came from

Calls only the oracle (oracle/) and the seeded inputs (workloads/).  CPU only;
a run takes minutes to tens of minutes on 8 cores and up to ~25 GB of memory
(the 138M workloads' fp64 replicas and momenta).

    python tests/golden/make_fullsize_golden.py [workload ...]
"""
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workloads as W  # noqa: E402

STORED = ("resnet18_like", "resnet50_like", "vgg16_adaptive", "many_small", "vgg16_const8", "vgg16_stepdecay")


def workload(key):
    return {**W.full_workloads(), **W.fullsize_variants()}[key]


def sample_indices(w, seed=0):
    """About 1024 sorted element indices: both ends of every tensor and random
    interior ones."""
    rng = np.random.default_rng(seed)
    ends = 4 if w.T <= 64 else 2
    per_tensor = max(2, 1024 // w.T)
    off = w.offsets()
    idx = []
    for tau in range(w.T):
        lo, hi = int(off[tau]), int(off[tau + 1])
        if hi == lo:
            continue
        idx.append(np.arange(lo, min(hi, lo + ends)))
        idx.append(np.arange(max(lo, hi - ends), hi))
        idx.append(rng.integers(lo, hi, size=min(per_tensor, hi - lo)))
    return np.unique(np.concatenate(idx)).astype(np.int64)


def main(keys):
    for key in keys:
        w = workload(key)
        t0 = time.time()
        print(f"{key}: K={w.K} P={w.P} T={w.T} N={w.total_steps}, oracle on "
              f"{oracle.num_threads()} threads ...", flush=True)
        r = oracle.Oracle(w).run()
        idx = sample_indices(w)
        rows = np.arange(w.K) if w.K <= 8 else np.array([0, 1, w.K // 2, w.K - 1])
        path = os.path.join(HERE, f"fullsize_{key}.npz")
        with open(oracle.oracle._SRC, "rb") as f:
            digest = hashlib.sha256(f.read()).hexdigest()
        np.savez_compressed(path, sync_t=r.sync_t, sync_p=r.sync_p, S=r.S, C2=r.C2, gamma=r.gamma,
                            var=r.var, idx=idx, rows=rows,
                            x=r.x[np.ix_(rows, idx)], v=r.v[np.ix_(rows, idx)], state_p=np.int64(r.state.p),
                            state_C2=np.float64(r.state.C2), state_nC2=np.int64(r.state.nC2),
                            oracle_source_sha256=np.array(digest))
        print(f"  {r.n_syncs} syncs, p {r.sync_p.min()}..{r.sync_p.max()}, {time.time() - t0:.0f} s -> {path}",
              flush=True)
        del r


if __name__ == "__main__":
    main(sys.argv[1:] or STORED)
