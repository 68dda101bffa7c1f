"""ADPSGD hot path on MI355X: Python side of the C ABI in ``include/adpsgd.h``.

``_native`` holds the ctypes binding (functions named as in C).  ``Adpsgd``
below owns one context together with its torch-allocated device buffers;
torch supplies only device memory and the HIP stream.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from ._native import (  # noqa: F401
    AdpsgdError, EDEVICE, EINVAL, ENONFINITE, ESTATE, EXPORTED, LAUNCH_DEVICE, LAUNCH_HOST, LAUNCH_HYBRID,
    LIB_PATH, LR_CONST, LR_COSINE, adpsgd_average_noalloc,
    LR_STEP, LR_WARMUP_STEP, OK, PERIOD_ADAPTIVE, PERIOD_ALG1, PERIOD_CONST, adpsgd_average, adpsgd_buffers, adpsgd_destroy,
    adpsgd_get_state, adpsgd_get_timing, adpsgd_hparams, adpsgd_init, adpsgd_last_error,
    adpsgd_local_steps, adpsgd_lr, adpsgd_normal_dump, adpsgd_philox_dump, adpsgd_reset, adpsgd_run,
    adpsgd_run_traced, adpsgd_step_rec,
    adpsgd_sched_init, adpsgd_sched_on_sync, adpsgd_sched_step, adpsgd_schedule, adpsgd_set_launch_policy, adpsgd_set_state, adpsgd_set_timing,
    adpsgd_get_step_launch, adpsgd_set_step_launch,
    adpsgd_padded_row_stride, adpsgd_state, adpsgd_step_average, adpsgd_sync_rec, adpsgd_timing,
    adpsgd_workspace_bytes, make_hparams,
)


def hparams_of(w) -> adpsgd_hparams:
    """hparams from any object with the fields of the C struct (e.g. a workload)."""
    return make_hparams(seed=w.seed, sigma=w.sigma, momentum=w.momentum, weight_decay=w.weight_decay,
                        h_lo=w.h_lo, h_hi=w.h_hi, lr_kind=w.lr_kind, lr0=w.lr0,
                        total_steps=w.total_steps, period_mode=w.period_mode, p_init=w.p_init,
                        k_s=w.k_s, thr_lo=w.thr_lo, thr_hi=w.thr_hi,
                        sync_warmup_steps=getattr(w, "sync_warmup_steps", 0),
                        p_switch_step=getattr(w, "p_switch_step", 0), p_after=getattr(w, "p_after", 0),
                        avg_momentum=getattr(w, "avg_momentum", False), p_max=getattr(w, "p_max", 0))


class Adpsgd:
    """One ADPSGD context with its device buffers on a torch device.

    x, m: float32 [K, P]; h, xstar: float32 [P]; workspace: uint8 sized by
    adpsgd_workspace_bytes.  The stream is the torch stream current at
    construction (or the one passed in).  With pad_rows (default), x, m, h and
    xstar are views of the rows of ONE [2K + 2, row_stride] buffer (x rows,
    then m rows, then h, then xstar), row_stride = adpsgd_padded_row_stride(P):
    256 n floats with n odd.  Every row then starts on a 1 KB boundary (the
    kernels move whole float4 groups, and each 64-lane wave's 1 KB of a row is
    one aligned kilobyte), and the rows that a kernel streams together start an
    odd number of kilobytes apart, which measures fastest on MI355X.
    pad_rows=False allocates x and m as packed [K, P] buffers and h and xstar
    on their own.
    """

    def __init__(self, K: int, offsets, hp: adpsgd_hparams, device="cuda", stream=None, pad_rows: bool = True):
        import torch
        self.torch = torch
        off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
        self.K, self.P, self.T = int(K), int(off[-1]), len(off) - 1
        self.offsets = off
        self.hp = hp
        self.device = torch.device(device)
        if self.device.type != "cuda":
            raise ValueError("the ADPSGD library runs on a GPU device only")
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = adpsgd_workspace_bytes(self.K, self.P, off)
        if nbytes == 0:
            raise ValueError("invalid K, P or tensor offsets")
        alloc = dict(device=self.device, dtype=torch.float32)
        K = self.K
        if pad_rows:
            self.row_stride = adpsgd_padded_row_stride(self.P)
            self._rows = torch.empty((2 * K + 2, self.row_stride), **alloc)
            self._x_rows, self._m_rows = self._rows[:K], self._rows[K:2 * K]
            self.h, self.xstar = self._rows[2 * K, :self.P], self._rows[2 * K + 1, :self.P]
        else:
            self.row_stride = self.P
            self._x_rows = torch.empty((K, self.P), **alloc)
            self._m_rows = torch.empty((K, self.P), **alloc)
            self.h = torch.empty((self.P,), **alloc)
            self.xstar = torch.empty((self.P,), **alloc)
        self.x = self._x_rows[:, :self.P]
        self.m = self._m_rows[:, :self.P]
        self.workspace = torch.empty((nbytes,), device=self.device, dtype=torch.uint8)
        self.buf = adpsgd_buffers(x=self._x_rows.data_ptr(), m=self._m_rows.data_ptr(), h=self.h.data_ptr(),
                                  xstar=self.xstar.data_ptr(), workspace=self.workspace.data_ptr(),
                                  workspace_bytes=nbytes, stream=self.stream.cuda_stream,
                                  row_stride=self.row_stride)
        with torch.cuda.device(self.device):
            self.ctx = adpsgd_init(self.K, self.P, off, hp, self.buf)

    @classmethod
    def from_workload(cls, w, device="cuda", stream=None, pad_rows: bool = True) -> "Adpsgd":
        return cls(w.K, w.offsets(), hparams_of(w), device=device, stream=stream, pad_rows=pad_rows)

    # -- the hot path
    def local_steps(self, n: int) -> None:
        adpsgd_local_steps(self.ctx, n)

    def average(self) -> np.ndarray:
        return adpsgd_average(self.ctx, self.T)

    def step_average(self) -> np.ndarray:
        return adpsgd_step_average(self.ctx, self.T)

    def schedule(self, var: np.ndarray) -> int:
        return adpsgd_schedule(self.ctx, var)

    def run(self, n_steps: int, log_cap: Optional[int] = None, with_var: bool = True):
        return adpsgd_run(self.ctx, n_steps, self.T, log_cap=log_cap, with_var=with_var)

    def run_traced(self, n_steps: int, log_cap: Optional[int] = None, with_var: bool = True):
        return adpsgd_run_traced(self.ctx, n_steps, self.T, log_cap=log_cap, with_var=with_var)

    def reset(self) -> None:
        adpsgd_reset(self.ctx)

    # -- state, timing
    def get_state(self) -> adpsgd_state:
        return adpsgd_get_state(self.ctx)

    def set_state(self, st: adpsgd_state) -> None:
        adpsgd_set_state(self.ctx, st)

    @property
    def step_launch(self) -> tuple:
        """(threads per block, LDS bytes reserved per block, chunks of a row an
        XCD takes in a run) of the plain local step."""
        return adpsgd_get_step_launch(self.ctx)

    def set_step_launch(self, block: int, lds_bytes: int = 0, row_chunks: int = 1) -> None:
        adpsgd_set_step_launch(self.ctx, block, lds_bytes, row_chunks)

    def set_launch_policy(self, policy: int) -> None:
        adpsgd_set_launch_policy(self.ctx, policy)

    def set_timing(self, every=True) -> None:
        adpsgd_set_timing(self.ctx, every)

    def get_timing(self) -> adpsgd_timing:
        return adpsgd_get_timing(self.ctx)

    def close(self) -> None:
        if getattr(self, "ctx", None):
            adpsgd_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def write_sync_log(path: str, recs: np.ndarray, var: Optional[np.ndarray] = None) -> int:
    """Append one JSON line per sync record (t, p, S, C2, gamma, margin and, when
    given, the per-tensor variances) to `path`; returns the number written."""
    import json
    with open(path, "a") as f:
        for j, r in enumerate(recs):
            row = {"t": int(r["t"]), "p": int(r["p"]), "S": float(r["S"]), "C2": float(r["C2"]),
                   "gamma": float(r["gamma"]),
                   "margin": None if np.isnan(r["margin"]) else float(r["margin"])}
            if var is not None:
                row["var"] = [float(v) for v in var[j]]
            f.write(json.dumps(row) + "\n")
    return len(recs)
