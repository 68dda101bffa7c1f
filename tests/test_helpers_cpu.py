"""The test suite's own diagnostics (CPU): the sync-list mismatch report names
the first differing sync and tells a near-tie from a wrong decision."""
import numpy as np

from helpers import sync_mismatch


def _recs(t, p, S, margin):
    r = np.zeros(len(t), dtype=[("t", np.int64), ("p", np.int32), ("S", np.float64), ("margin", np.float64)])
    r["t"], r["p"], r["S"], r["margin"] = t, p, S, margin
    return r


def test_identical_lists_give_no_report():
    t, p = [3, 7, 12], [4, 4, 5]
    assert sync_mismatch(_recs(t, p, [1.0, 1.0, 1.0], [np.nan] * 3), t, p, [1.0] * 3, [1.0] * 3,
                         [0.1] * 3) is None


def test_near_tie_is_named():
    # oracle: S at t = 7 sits 1e-7 below 0.7 gamma C2, so p grows; the GPU's S
    # is 3e-7 above it, so p stays: the next sync differs
    gamma, C2 = 0.1, 10.0
    thr = 0.7 * gamma * C2
    o_S = [1.0, thr * (1 - 1e-7), 1.0]
    g_S = [1.0, thr * (1 + 3e-7), 1.0]
    o_t, o_p = [3, 7, 12], [4, 4, 5]
    g_t, g_p = [3, 7, 11], [4, 4, 4]
    msg = sync_mismatch(_recs(g_t, g_p, g_S, [np.nan, 3e-7, np.nan]), o_t, o_p, o_S, [C2] * 3, [gamma] * 3)
    assert "at sync 2" in msg and "decision at sync 1 (t=7)" in msg and "near-tie" in msg


def test_wrong_decision_is_not_a_near_tie():
    gamma, C2 = 0.1, 10.0
    thr = 0.7 * gamma * C2
    o_S = g_S = [1.0, thr * 0.5, 1.0]            # far below the band: p must grow
    msg = sync_mismatch(_recs([3, 7, 11], [4, 4, 4], g_S, [np.nan, -0.5, np.nan]), [3, 7, 12], [4, 4, 5],
                        o_S, [C2] * 3, [gamma] * 3)
    assert "decision at sync 1" in msg and "near-tie" not in msg


def test_length_difference_and_first_sync():
    msg = sync_mismatch(_recs([3, 7], [4, 4], [1.0, 1.0], [np.nan] * 2), [3, 7, 11], [4, 4, 4],
                        [1.0] * 3, [1.0] * 3, [0.1] * 3)
    assert "at sync 2" in msg
    msg = sync_mismatch(_recs([2], [3], [1.0], [np.nan]), [3], [4], [1.0], [1.0], [0.1])
    assert "first sync already differs" in msg
