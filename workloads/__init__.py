"""Seeded synthetic workloads shared by the HIP path, the oracle, the tests and the bench.

This module holds inputs only: problem sizes, hyper-parameters and the tensor
partition of the flat parameter vector.  It contains none of the method's
arithmetic (no gradient, no averaging, no variance, no period control), so both
the GPU library and the CPU oracle can take their inputs from it without sharing
any computation.

The method is ADPSGD, adaptive periodic parameter averaging SGD (Jiang and
Agrawal, arXiv 2007.06134).  The paper trains CNNs on CIFAR-10 and ImageNet
(Section IV-A); those datasets and networks are not used here.  They are
replaced by a separable noisy diagonal quadratic

    f(x) = 1/2 * sum_i h_i (x_i - x*_i)^2,  stochastic gradient h*(x - x*) + sigma*z,

with the tensor partitions below shaped after real models (a ResNet18-sized,
a ResNet50-sized and a VGG16-ImageNet-sized parameter vector, and a many-small-
tensor stress case).  h, x* and z are drawn inside the method from a
counter-based generator keyed by the seed; only the seed is an input.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

LR_CONST, LR_STEP, LR_COSINE, LR_WARMUP_STEP = 0, 1, 2, 3
PERIOD_CONST, PERIOD_ADAPTIVE, PERIOD_ALG1 = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic ADPSGD run.  Field names follow the C ABI's hparams."""

    name: str
    K: int                    # simulated workers (the paper's n nodes)
    sizes: tuple              # element count of each tensor, in order; sum == P
    seed: int
    sigma: float              # std of the additive gradient noise
    momentum: float           # heavy-ball coefficient (0.9 throughout the paper)
    weight_decay: float       # coupled L2 coefficient
    h_lo: float               # curvatures h_i ~ LogUniform[h_lo, h_hi]
    h_hi: float
    lr_kind: int
    lr0: float
    total_steps: int          # N, the number of local steps (the paper's K)
    period_mode: int
    p_init: int
    k_s: int                  # end of the C2 sampling phase (step index)
    thr_lo: float = 0.7       # Algorithm 2 thresholds
    thr_hi: float = 1.3
    sync_warmup_steps: int = 0   # steps synced every step before Algorithm 2 starts
    p_switch_step: int = 0       # constant modes: the period becomes p_after from this step
    p_after: int = 0
    avg_momentum: bool = False   # average the momentum buffers at a sync as well
    p_max: int = 0               # upper bound on the adaptive period (0: none)

    @property
    def P(self) -> int:
        return int(sum(self.sizes))

    @property
    def T(self) -> int:
        return len(self.sizes)

    def offsets(self) -> np.ndarray:
        off = np.zeros(self.T + 1, dtype=np.int64)
        off[1:] = np.cumsum(np.asarray(self.sizes, dtype=np.int64))
        return off

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def updates_per_run(self) -> int:
        return self.K * self.P * self.total_steps


def log_uniform_sizes(stream: int, T: int, lo: float, hi: float, total: int,
                      multiple: int = 4, minimum: int = 4,
                      fixed: Optional[List[int]] = None) -> tuple:
    """Tensor sizes drawn log-uniformly in [lo, hi], rescaled to sum to `total`.

    `fixed` sizes come first, unchanged; the T - len(fixed) drawn sizes share
    the remainder.  Each drawn size is rounded to a multiple of `multiple`
    (at least `minimum`) and the rounding residue goes to the largest drawn
    tensor, so the sum is exact.  The generator is numpy's PCG64 seeded with
    `stream`, so the partition is reproducible.
    """
    fixed = list(fixed or [])
    n = T - len(fixed)
    rest = total - sum(fixed)
    spare = rest - n * minimum
    if n < 1 or spare < 0 or spare % multiple or minimum < 1:
        raise ValueError("cannot place the drawn tensors")
    rng = np.random.default_rng(stream)
    s = np.exp(rng.uniform(np.log(lo), np.log(hi), n))
    # Each tensor gets `minimum` plus a share of the spare elements, in units of
    # `multiple`, proportional to its drawn size; leftover units go to the largest.
    units = spare // multiple
    share = np.floor(s * (units / s.sum())).astype(np.int64)
    share[int(np.argmax(s))] += units - int(share.sum())
    out = minimum + multiple * share
    assert int(out.sum()) == rest and out.min() >= minimum
    return tuple(int(v) for v in fixed) + tuple(int(v) for v in out)


def _cfg_quadratic_small() -> Workload:
    return Workload(
        name="k4_p65536_t1_const4", K=4, sizes=(65_536,), seed=1,
        sigma=0.1, momentum=0.9, weight_decay=0.0, h_lo=1e-2, h_hi=1.0,
        lr_kind=LR_CONST, lr0=0.05, total_steps=200,
        period_mode=PERIOD_CONST, p_init=4, k_s=0)


def _cfg_resnet18_like() -> Workload:
    return Workload(
        name="k8_p11.2m_t62_stepdecay_adaptive", K=8,
        sizes=log_uniform_sizes(1002, 62, 64, 2.4e6, 11_200_000), seed=2,
        sigma=0.05, momentum=0.9, weight_decay=5e-4, h_lo=1e-2, h_hi=1.0,
        lr_kind=LR_STEP, lr0=0.1, total_steps=2000,
        period_mode=PERIOD_ADAPTIVE, p_init=1, k_s=500)


def _cfg_resnet50_like() -> Workload:
    return Workload(
        name="k16_p25.6m_t161_cosine_adaptive", K=16,
        sizes=log_uniform_sizes(1003, 161, 64, 2.4e6, 25_600_000), seed=3,
        sigma=0.1, momentum=0.9, weight_decay=1e-4, h_lo=1e-3, h_hi=1.0,
        lr_kind=LR_COSINE, lr0=0.1, total_steps=1000,
        period_mode=PERIOD_ADAPTIVE, p_init=4, k_s=250)


def _vgg16_sizes() -> tuple:
    return log_uniform_sizes(1004, 32, 64, 2.4e6, 138_000_000,
                             fixed=[102_000_000, 16_800_000, 4_100_000])


def _cfg_vgg16_like(adaptive: bool) -> Workload:
    return Workload(
        name="k8_p138m_t32_" + ("adaptive" if adaptive else "const8"), K=8,
        sizes=_vgg16_sizes(), seed=4,
        sigma=0.02, momentum=0.9, weight_decay=5e-4, h_lo=1e-2, h_hi=1.0,
        lr_kind=LR_CONST, lr0=0.01, total_steps=500,
        period_mode=PERIOD_ADAPTIVE if adaptive else PERIOD_CONST,
        p_init=4 if adaptive else 8, k_s=125 if adaptive else 0)


def _cfg_many_small() -> Workload:
    return Workload(
        name="k32_p1.2m_t400_adaptive", K=32,
        sizes=log_uniform_sizes(1005, 400, 16, 65_536, 1_200_000, minimum=16),
        seed=5, sigma=0.2, momentum=0.9, weight_decay=0.0, h_lo=1e-2, h_hi=1.0,
        lr_kind=LR_CONST, lr0=0.05, total_steps=5000,
        period_mode=PERIOD_ADAPTIVE, p_init=4, k_s=1250)


def full_workloads() -> dict:
    """The six full-size runs, keyed by a short id."""
    return {
        "quad_small": _cfg_quadratic_small(),
        "resnet18_like": _cfg_resnet18_like(),
        "resnet50_like": _cfg_resnet50_like(),
        "vgg16_const8": _cfg_vgg16_like(False),
        "vgg16_adaptive": _cfg_vgg16_like(True),
        "many_small": _cfg_many_small(),
    }


def fullsize_variants() -> dict:
    """Full-size variants used only by the tests: the 138M-parameter adaptive
    workload with the step-decayed rate of the ResNet-shaped runs (x0.1 at steps
    250 and 375), so that the controller moves p at that size (with the
    constant rate it keeps p = 4)."""
    w = _cfg_vgg16_like(True)
    return {"vgg16_stepdecay": w.replace(name="k8_p138m_t32_stepdecay_adaptive", lr_kind=LR_STEP)}


def reduced(w: Workload, P: int, T: Optional[int] = None, steps: Optional[int] = None,
            minimum: int = 1, multiple: int = 1, stream: int = 7) -> Workload:
    """A smaller copy of `w` for element-by-element parity against the oracle.

    K, the hyper-parameters, the period mode and the learning-rate schedule are
    kept; P shrinks, the tensor sizes are redrawn log-uniformly (ragged: any
    size >= `minimum`, multiple of `multiple`), and optionally fewer steps are
    run with the schedule's boundaries scaled to the new step count.
    """
    T = w.T if T is None else T
    lo = max(1, min(w.sizes))
    hi = max(lo + 1, min(max(w.sizes), P))
    sizes = log_uniform_sizes(stream, T, lo, hi, P, multiple=multiple, minimum=minimum)
    kw = dict(name=w.name + f"_reduced_p{P}", sizes=sizes)
    if steps is not None:
        kw["total_steps"] = steps
        kw["k_s"] = int(w.k_s * steps // w.total_steps)
    return w.replace(**kw)


def parity_workloads() -> dict:
    """Reduced copies of every full run, sized so the oracle takes seconds.

    They keep each run's K, N, schedule and controller, and use ragged tensor
    sizes (not multiples of 4), so tiles straddle float4 groups.
    """
    f = full_workloads()
    return {
        "quad_small": f["quad_small"],
        "resnet18_like": reduced(f["resnet18_like"], 40_000, steps=2000),
        "resnet50_like": reduced(f["resnet50_like"], 36_000, steps=1000),
        "vgg16_const8": reduced(f["vgg16_const8"], 120_000),
        "vgg16_adaptive": reduced(f["vgg16_adaptive"], 120_000),
        "many_small": reduced(f["many_small"], 6_000, steps=5000),
    }
