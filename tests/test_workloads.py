"""The seeded input generator (workloads/): shapes and hyper-parameters of the
six runs, exact tensor-size sums, alignment, fixed tensors, determinism, and
the reduced parity copies.  Inputs only: nothing here computes the method."""
import numpy as np
import pytest

import workloads as W

# K, P, T, N, period mode, p_init, K_s, sigma, momentum, weight decay, LR kind, lr0, h_lo
EXPECTED = {
    "quad_small": (4, 65_536, 1, 200, W.PERIOD_CONST, 4, 0, 0.1, 0.9, 0.0, W.LR_CONST, 0.05, 1e-2),
    "resnet18_like": (8, 11_200_000, 62, 2000, W.PERIOD_ADAPTIVE, 1, 500, 0.05, 0.9, 5e-4, W.LR_STEP, 0.1, 1e-2),
    "resnet50_like": (16, 25_600_000, 161, 1000, W.PERIOD_ADAPTIVE, 4, 250, 0.1, 0.9, 1e-4, W.LR_COSINE, 0.1, 1e-3),
    "vgg16_const8": (8, 138_000_000, 32, 500, W.PERIOD_CONST, 8, 0, 0.02, 0.9, 5e-4, W.LR_CONST, 0.01, 1e-2),
    "vgg16_adaptive": (8, 138_000_000, 32, 500, W.PERIOD_ADAPTIVE, 4, 125, 0.02, 0.9, 5e-4, W.LR_CONST, 0.01, 1e-2),
    "many_small": (32, 1_200_000, 400, 5000, W.PERIOD_ADAPTIVE, 4, 1250, 0.2, 0.9, 0.0, W.LR_CONST, 0.05, 1e-2),
}


@pytest.mark.parametrize("key", list(EXPECTED))
def test_full_workload_shapes_and_hyperparameters(key):
    w = W.full_workloads()[key]
    K, P, T, N, mode, p_init, k_s, sigma, mu, wd, lr_kind, lr0, h_lo = EXPECTED[key]
    assert (w.K, w.P, w.T, w.total_steps, w.period_mode, w.p_init, w.k_s) == (K, P, T, N, mode, p_init, k_s)
    assert (w.sigma, w.momentum, w.weight_decay, w.lr_kind, w.lr0, w.h_lo, w.h_hi) == \
        (sigma, mu, wd, lr_kind, lr0, h_lo, 1.0)
    assert (w.thr_lo, w.thr_hi) == (0.7, 1.3)
    if mode == W.PERIOD_ADAPTIVE:
        assert w.k_s == N // 4                      # K_s = 0.25 of the run
    off = w.offsets()
    assert off[0] == 0 and off[-1] == P and np.all(np.diff(off) == np.asarray(w.sizes))


@pytest.mark.parametrize("key", list(EXPECTED))
def test_full_workload_sizes_are_aligned(key):
    w = W.full_workloads()[key]
    sizes = np.asarray(w.sizes)
    assert np.all(sizes % 4 == 0)                  # 16-byte float4 groups never straddle tensors
    assert sizes.min() >= (16 if key == "many_small" else 4)
    if key.startswith("vgg16"):
        assert w.sizes[:3] == (102_000_000, 16_800_000, 4_100_000)
        assert sum(w.sizes[3:]) == 15_100_000


def test_drawn_sizes_follow_the_log_uniform_law():
    """Many draws: the log of the drawn sizes is roughly uniform over [ln lo, ln hi]
    before rescaling, so the rescaled sizes span several decades."""
    sizes = np.asarray(W.log_uniform_sizes(77, 4000, 64, 2.4e6, 4000 * 50_000))
    ls = np.log(sizes)
    assert ls.max() - ls.min() > 0.8 * (np.log(2.4e6) - np.log(64))
    assert sum(sizes) == 4000 * 50_000


def test_generator_is_deterministic_and_exact():
    a = W.full_workloads()
    b = W.full_workloads()
    assert all(a[k].sizes == b[k].sizes for k in a)
    for stream in range(5):
        s = W.log_uniform_sizes(stream, 37, 3, 9000, 123_457, multiple=1, minimum=1)
        assert len(s) == 37 and sum(s) == 123_457 and min(s) >= 1
    with pytest.raises(ValueError):
        W.log_uniform_sizes(0, 10, 64, 100, 39)     # cannot place 10 tensors of >= 4


def test_parity_copies_keep_the_schedule_and_are_ragged():
    full, par = W.full_workloads(), W.parity_workloads()
    assert set(par) == set(full)
    for key, w in par.items():
        f = full[key]
        assert (w.K, w.period_mode, w.p_init, w.lr_kind, w.lr0, w.sigma) == \
            (f.K, f.period_mode, f.p_init, f.lr_kind, f.lr0, f.sigma)
        assert w.P <= 120_000 and w.T == f.T
        if key != "quad_small":
            assert any(s % 4 for s in w.sizes), key   # some tensors straddle float4 groups
