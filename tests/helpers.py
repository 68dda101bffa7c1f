"""Shared helpers of the test suite: error metrics, tolerances and GPU run wrappers."""
from __future__ import annotations

import numpy as np

# Parity bars of the HIP path against the oracle.  Parameters: max relative
# error per tensor against max(|oracle|, 1e-2 rms of the tensor).  Per-tensor
# variances and S: relative error.
PARAM_TOL = 1e-4
VAR_TOL = 1e-3
# Momentum buffers are zero-mean, noise-driven state, so an element's error is
# judged against max(|m|, rms of its tensor) (MOM_FLOOR = 1), not a 1e-2 rms
# floor.  m integrates each step's fp32 gradient error with gain 1 / (1 - mu)
# = 10 and sees the parameter error through h, so its error runs above the
# parameters'; the largest seen over every parity run is 1.6e-4 (K = 3 with
# averaged momentum), the others at most 7e-5.  The bar is twice the largest.
MOM_FLOOR = 1.0
MOM_TOL = 3e-4


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


def _margin(S, gamma, C2, thr_lo, thr_hi):
    """Signed relative distance of S to the nearer threshold (Algorithm 2, lines
    16-19): S / (thr gamma C2) - 1; NaN when no decision is possible."""
    lo, hi = thr_lo * gamma * C2, thr_hi * gamma * C2
    if not (lo > 0):
        return float("nan")
    m_lo, m_hi = S / lo - 1.0, S / hi - 1.0
    return m_lo if abs(m_lo) < abs(m_hi) else m_hi


def sync_mismatch(recs, o_t, o_p, o_S, o_C2, o_gamma, thr_lo=0.7, thr_hi=1.3):
    """None if the GPU's sync list (recs: fields t, p, S, C2, margin) equals the
    oracle's, else a message naming the first differing sync and the decision
    behind it: the sync before it, with both sides' S, their relative gap and
    each side's margin to the nearer threshold.  A gap comparable to the
    margin marks a near-tie (two correct roundings on either side of a
    threshold) rather than a wrong controller."""
    t, p = np.asarray(recs["t"]), np.asarray(recs["p"])
    o_t, o_p = np.asarray(o_t), np.asarray(o_p)
    n = min(len(t), len(o_t))
    diff = np.nonzero((t[:n] != o_t[:n]) | (p[:n] != o_p[:n]))[0]
    if len(diff) == 0 and len(t) == len(o_t):
        return None
    j = int(diff[0]) if len(diff) else n
    msg = [f"sync lists differ at sync {j} of {len(o_t)} (GPU {len(t)} syncs)"]
    if j < n:
        msg.append(f"GPU (t={t[j]}, p={p[j]}) vs oracle (t={o_t[j]}, p={o_p[j]})")
    if j == 0:
        msg.append("the first sync already differs: no decision precedes it")
        return "; ".join(msg)
    d = j - 1
    gap = abs(recs["S"][d] - o_S[d]) / abs(o_S[d]) if o_S[d] != 0 else float("inf")
    # C2 is unchanged by a decisive sync, so the record's C2 is the one decided on
    m_o = _margin(o_S[d], o_gamma[d], o_C2[d], thr_lo, thr_hi)
    msg.append(f"decision at sync {d} (t={o_t[d]}): S GPU {recs['S'][d]:.17g} oracle {o_S[d]:.17g} "
               f"(relative gap {gap:.2e}); margin GPU {recs['margin'][d]:.3e} oracle {m_o:.3e}")
    if np.isfinite(m_o) and gap >= 0.5 * abs(m_o):
        msg.append("near-tie: the S gap reaches the margin")
    return "; ".join(msg)


def assert_same_syncs(recs, r, w):
    """Identical sync lists (steps and periods) between a GPU run's records and
    an oracle run r, with the near-tie diagnosis of sync_mismatch on failure."""
    why = sync_mismatch(recs, r.sync_t, r.sync_p, r.S, r.C2, r.gamma, w.thr_lo, w.thr_hi)
    assert why is None, why
