"""adpsgd_average_noalloc, the entry point that allocates nothing, against
adpsgd_average on the same replicas (GPU).

Three calls in a row on one GPU, each on a smaller problem than the one
before (the scratch array keeps the previous call's contents): the replicas
must come out bitwise equal to those adpsgd_average leaves, and the
per-tensor variances equal to its variances within the parity bar (and to
rounding).  A problem beyond the scratch array is refused before anything
runs."""
import sys

import numpy as np
import pytest

import workloads as W
from helpers import VAR_TOL, rel_err

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def A():
    import torch
    assert torch.cuda.is_available()
    import paper_2007_06134_amd as A
    return A


def _cases():
    pw = W.parity_workloads()
    return [
        ("K=32, 400 tensors, rows padded", pw["many_small"].replace(sizes=W.log_uniform_sizes(11, 400, 16, 4096, 90_000, minimum=1, multiple=1)), True),
        ("K=8, 62 ragged tensors, rows padded", pw["resnet18_like"], True),
        ("K=3, an empty tensor, rows packed (P odd)", W.Workload(
            name="k3", K=3, sizes=(1001, 0, 2046, 7, 3), seed=5, sigma=0.1, momentum=0.9, weight_decay=5e-4,
            h_lo=1e-2, h_hi=1.0, lr_kind=W.LR_CONST, lr0=0.05, total_steps=10, period_mode=W.PERIOD_CONST,
            p_init=100, k_s=0), False),
    ]


def test_noalloc_sync_equals_context_sync(A):
    import torch
    sizes_seen = []
    for name, w, pad in _cases():
        _say(f"no-alloc sync, {name}: K={w.K} P={w.P} T={w.T}")
        with A.Adpsgd.from_workload(w, pad_rows=pad) as eng:
            eng.local_steps(5)
            rows = eng._x_rows.clone()                      # the same replicas, same layout
            var_ctx = eng.average()                          # adpsgd_average on the context
            torch.cuda.synchronize()
            var_na = A.adpsgd_average_noalloc(w.K, w.P, eng.row_stride, w.offsets(), rows.data_ptr(),
                                              torch.cuda.current_stream().cuda_stream)
            x_ctx = eng.x.clone()
        x_na = rows[:, :w.P]
        assert torch.equal(x_na, x_ctx), name
        assert bool((x_na == x_na[0:1]).all()), name       # every row holds the mean
        assert rel_err(var_na, var_ctx) < VAR_TOL, name
        assert rel_err(var_na, var_ctx) < 1e-12, name
        nz = np.diff(w.offsets()) > 0
        assert np.all(var_na[nz] > 0) and np.all(var_na[~nz] == 0), name
        sizes_seen.append(w.K * w.P)
    assert sizes_seen == sorted(sizes_seen, reverse=True)


def test_noalloc_refuses_beyond_scratch(A):
    import torch
    P = 1 << 30                                   # 4M sync tiles: more than the scratch array holds
    with pytest.raises(A.AdpsgdError) as e:
        A.adpsgd_average_noalloc(2, P, 0, [0, P], 256, 0)
    assert e.value.code == A.EINVAL and "scratch" in A.adpsgd_last_error()
    with pytest.raises(A.AdpsgdError) as e:
        A.adpsgd_average_noalloc(0, 8, 0, [0, 8], 256, 0)
    assert e.value.code == A.EINVAL
