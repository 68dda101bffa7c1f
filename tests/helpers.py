"""Shared helpers of the test suite: error metrics and GPU run wrappers."""
from __future__ import annotations

import numpy as np


def max_rel_err(a: np.ndarray, b: np.ndarray, offsets, floor: float = 1e-2, scale_of=None) -> float:
    """Largest |a - b| / max(|b|, floor * rms_tau(b)) over all rows and tensors.

    a, b: [K, P] (or [P]); the rms floor is taken per tensor so elements that
    happen to sit near zero are judged against the tensor's own scale.  If
    scale_of ([*, P]) is given, the rms is taken over it instead of b.
    """
    a = np.atleast_2d(np.asarray(a, dtype=np.float64))
    b = np.atleast_2d(np.asarray(b, dtype=np.float64))
    ref = b if scale_of is None else np.atleast_2d(np.asarray(scale_of, dtype=np.float64))
    worst = 0.0
    for lo, hi in zip(offsets[:-1], offsets[1:]):
        if hi == lo:
            continue
        bb = b[:, lo:hi]
        rr = ref[:, lo:hi]
        rms = float(np.sqrt(np.mean(rr * rr)))
        den = np.maximum(np.abs(bb), max(floor * rms, 1e-30))
        worst = max(worst, float(np.max(np.abs(a[:, lo:hi] - bb) / den)))
    return worst


def rel_err(a, b, floor: float = 1e-300) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.size == 0:
        return 0.0
    return float(np.max(np.abs(a - b) / np.maximum(np.abs(b), floor)))


def gpu_run(w, n_steps=None, fetch=True, policy=None, pad_rows=True):
    """Run workload w on cuda:0 through the C ABI; returns a dict of host results."""
    import paper_2007_06134_amd as A
    n = w.total_steps if n_steps is None else n_steps
    with A.Adpsgd.from_workload(w, pad_rows=pad_rows) as eng:
        if policy is not None:
            eng.set_launch_policy(policy)
        recs, var, n_syncs = eng.run(n)
        out = dict(recs=recs, var=var, n_syncs=n_syncs, state=eng.get_state())
        if fetch:
            out["x"] = eng.x.double().cpu().numpy()
            out["m"] = eng.m.double().cpu().numpy()
            out["h"] = eng.h.double().cpu().numpy()
            out["xs"] = eng.xstar.double().cpu().numpy()
    return out
