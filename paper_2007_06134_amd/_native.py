"""ctypes binding of ``libadpsgd.so`` (the C ABI in ``include/adpsgd.h``).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  Functions keep the C names; a failing status raises
``AdpsgdError`` carrying the library's message.  If the library has not been
built, or was built from other sources than those in the tree (a digest
recorded at build time), importing this module builds it (hipcc, gfx950); if
that fails, or ADPSGD_NO_REBUILD is set, it raises ImportError (there is no
fallback).
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libadpsgd.so")

OK, EINVAL, ESTATE, EDEVICE, ENONFINITE = 0, -1, -2, -3, -4
LR_CONST, LR_STEP, LR_COSINE, LR_WARMUP_STEP = 0, 1, 2, 3
PERIOD_CONST, PERIOD_ADAPTIVE, PERIOD_ALG1 = 0, 1, 2
LAUNCH_HYBRID, LAUNCH_DEVICE, LAUNCH_HOST = 0, 1, 2


class AdpsgdError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"adpsgd error {code}: {message}")
        self.code = code


class adpsgd_hparams(C.Structure):
    _fields_ = [
        ("seed", C.c_uint64), ("sigma", C.c_double), ("momentum", C.c_double),
        ("weight_decay", C.c_double), ("h_lo", C.c_double), ("h_hi", C.c_double),
        ("lr_kind", C.c_int32), ("period_mode", C.c_int32), ("lr0", C.c_double),
        ("total_steps", C.c_int64), ("p_init", C.c_int32), ("p_max", C.c_int32),
        ("k_s", C.c_int64), ("thr_lo", C.c_double), ("thr_hi", C.c_double),
        ("sync_warmup_steps", C.c_int64), ("p_switch_step", C.c_int64), ("p_after", C.c_int32),
        ("avg_momentum", C.c_int32),
    ]


class adpsgd_buffers(C.Structure):
    _fields_ = [
        ("x", C.c_void_p), ("m", C.c_void_p), ("h", C.c_void_p), ("xstar", C.c_void_p),
        ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t), ("stream", C.c_void_p),
        ("row_stride", C.c_int64),
    ]


class adpsgd_state(C.Structure):
    _fields_ = [("t", C.c_int64), ("cnt", C.c_int64), ("nC2", C.c_int64), ("C2", C.c_double),
                ("p", C.c_int32), ("reserved", C.c_int32)]


class adpsgd_sync_rec(C.Structure):
    _fields_ = [("t", C.c_int64), ("p", C.c_int32), ("reserved", C.c_int32), ("S", C.c_double),
                ("C2", C.c_double), ("gamma", C.c_double), ("margin", C.c_double)]


class adpsgd_step_rec(C.Structure):
    _fields_ = [("t", C.c_int64), ("synced", C.c_int32), ("p", C.c_int32), ("var", C.c_double),
                ("grad_norm2", C.c_double), ("gamma", C.c_double)]


class adpsgd_timing(C.Structure):
    _fields_ = [("step_ms", C.c_double), ("step_launches", C.c_int64),
                ("fused_ms", C.c_double), ("fused_launches", C.c_int64),
                ("average_ms", C.c_double), ("average_launches", C.c_int64),
                ("segsum_ms", C.c_double), ("segsum_launches", C.c_int64),
                ("trace_ms", C.c_double), ("trace_launches", C.c_int64),
                ("graph_captures", C.c_int64), ("graph_replays", C.c_int64)]


from . import build as _build  # noqa: E402

if not _build.is_current():
    # nothing built yet, or built from other sources than the ones here (the
    # digest written next to the library at build time differs): build it now
    # with hipcc (gfx950).  ADPSGD_NO_REBUILD=1 refuses instead.  There is no
    # fallback either way.
    _why = "is not built" if not os.path.exists(LIB_PATH) else "was built from other sources"
    if os.environ.get("ADPSGD_NO_REBUILD"):
        raise ImportError(f"{LIB_PATH} {_why} (source digest differs) and ADPSGD_NO_REBUILD is set; "
                          "run `python -m paper_2007_06134_amd.build`")
    import sys as _sys
    print(f"paper_2007_06134_amd: {LIB_PATH} {_why}; building it", file=_sys.stderr, flush=True)
    try:
        _build.build()
    except Exception as e:  # noqa: BLE001
        raise ImportError(f"{LIB_PATH} {_why} and building it failed ({e}); "
                          "run `python -m paper_2007_06134_amd.build`") from e

# One HIP runtime per process.  torch ships its own libamdhip64 and finds it
# next to its libraries; this library asks for libamdhip64.so.7, which the
# loader resolves to whatever is already loaded under that name.  Importing
# torch first makes that torch's copy.  Loaded the other way round, the
# process would hold two runtimes and this library's would see no device.
import torch  # noqa: E402,F401

lib = C.CDLL(LIB_PATH)

_CTX = C.c_void_p
_I64P = C.POINTER(C.c_int64)
_DP = C.POINTER(C.c_double)

_SIGS = {
    "adpsgd_workspace_bytes": (C.c_size_t, [C.c_int32, C.c_int64, C.c_int32, _I64P]),
    "adpsgd_padded_row_stride": (C.c_int64, [C.c_int64]),
    "adpsgd_init": (C.c_int, [C.c_int32, C.c_int64, _I64P, C.c_int32, C.POINTER(adpsgd_hparams),
                              C.POINTER(adpsgd_buffers), C.POINTER(_CTX)]),
    "adpsgd_reset": (C.c_int, [_CTX]),
    "adpsgd_local_steps": (C.c_int, [_CTX, C.c_int32]),
    "adpsgd_average": (C.c_int, [_CTX, _DP]),
    "adpsgd_step_average": (C.c_int, [_CTX, _DP]),
    "adpsgd_schedule": (C.c_int, [_CTX, _DP, C.POINTER(C.c_int32)]),
    "adpsgd_run": (C.c_int, [_CTX, C.c_int64, C.POINTER(adpsgd_sync_rec), C.c_int64, _DP, _I64P]),
    "adpsgd_run_traced": (C.c_int, [_CTX, C.c_int64, C.POINTER(adpsgd_sync_rec), C.c_int64, _DP,
                                    C.POINTER(adpsgd_step_rec), C.c_int64, _I64P]),
    "adpsgd_get_state": (C.c_int, [_CTX, C.POINTER(adpsgd_state)]),
    "adpsgd_set_state": (C.c_int, [_CTX, C.POINTER(adpsgd_state)]),
    "adpsgd_set_launch_policy": (C.c_int, [_CTX, C.c_int32]),
    "adpsgd_set_step_launch": (C.c_int, [_CTX, C.c_int32, C.c_int32, C.c_int32]),
    "adpsgd_get_step_launch": (C.c_int, [_CTX, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32)]),
    "adpsgd_set_timing": (C.c_int, [_CTX, C.c_int32]),
    "adpsgd_get_timing": (C.c_int, [_CTX, C.POINTER(adpsgd_timing)]),
    "adpsgd_destroy": (C.c_int, [_CTX]),
    "adpsgd_last_error": (C.c_char_p, []),
    "adpsgd_average_noalloc": (C.c_int, [C.c_int32, C.c_int64, C.c_int64, _I64P, C.c_int32, C.c_void_p, _DP,
                                         C.c_void_p]),
    "adpsgd_philox_dump": (C.c_int, [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_int64,
                                     C.c_int64, C.c_void_p, C.c_void_p]),
    "adpsgd_normal_dump": (C.c_int, [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_int64,
                                     C.c_int64, C.c_void_p, C.c_void_p]),
    "adpsgd_lr": (C.c_double, [C.POINTER(adpsgd_hparams), C.c_int64]),
    "adpsgd_sched_init": (C.c_int, [C.POINTER(adpsgd_hparams), C.POINTER(adpsgd_state)]),
    "adpsgd_sched_step": (C.c_int, [C.POINTER(adpsgd_hparams), C.POINTER(adpsgd_state), C.POINTER(C.c_int32)]),
    "adpsgd_sched_on_sync": (C.c_int, [C.POINTER(adpsgd_hparams), C.POINTER(adpsgd_state), C.c_int64,
                                       C.c_double, _DP]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


def _check(code: int) -> int:
    if code != OK:
        raise AdpsgdError(code, lib.adpsgd_last_error().decode())
    return code


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def adpsgd_last_error() -> str:
    return lib.adpsgd_last_error().decode()


def make_hparams(seed, sigma, momentum, weight_decay, h_lo, h_hi, lr_kind, lr0, total_steps,
                 period_mode, p_init, k_s, thr_lo=0.7, thr_hi=1.3, p_max=0, sync_warmup_steps=0,
                 p_switch_step=0, p_after=0, avg_momentum=False) -> adpsgd_hparams:
    return adpsgd_hparams(seed=seed, sigma=sigma, momentum=momentum, weight_decay=weight_decay,
                          h_lo=h_lo, h_hi=h_hi, lr_kind=lr_kind, period_mode=period_mode, lr0=lr0,
                          total_steps=total_steps, p_init=p_init, p_max=p_max, k_s=k_s,
                          thr_lo=thr_lo, thr_hi=thr_hi, sync_warmup_steps=sync_warmup_steps,
                          p_switch_step=p_switch_step, p_after=p_after,
                          avg_momentum=1 if avg_momentum else 0)


def adpsgd_workspace_bytes(K: int, P: int, offsets: Sequence[int]) -> int:
    off = _i64(offsets)
    return int(lib.adpsgd_workspace_bytes(K, P, len(off) - 1, off.ctypes.data_as(_I64P)))


def adpsgd_padded_row_stride(P: int) -> int:
    return int(lib.adpsgd_padded_row_stride(P))


def adpsgd_init(K: int, P: int, offsets: Sequence[int], hp: adpsgd_hparams, buf: adpsgd_buffers) -> int:
    off = _i64(offsets)
    ctx = _CTX()
    _check(lib.adpsgd_init(K, P, off.ctypes.data_as(_I64P), len(off) - 1, C.byref(hp), C.byref(buf),
                           C.byref(ctx)))
    return ctx.value


def adpsgd_reset(ctx: int) -> None:
    _check(lib.adpsgd_reset(ctx))


def adpsgd_local_steps(ctx: int, n: int) -> None:
    _check(lib.adpsgd_local_steps(ctx, n))


def adpsgd_average(ctx: int, T: int) -> np.ndarray:
    var = np.zeros(T)
    _check(lib.adpsgd_average(ctx, var.ctypes.data_as(_DP)))
    return var


def adpsgd_step_average(ctx: int, T: int) -> np.ndarray:
    var = np.zeros(T)
    _check(lib.adpsgd_step_average(ctx, var.ctypes.data_as(_DP)))
    return var


def adpsgd_average_noalloc(K: int, P: int, row_stride: int, offsets: Sequence[int], x_ptr: int,
                           stream: int) -> np.ndarray:
    """The separate sync of a [K, row_stride] device buffer with no context and no
    allocation on the device; returns the per-tensor variances."""
    off = _i64(offsets)
    var = np.zeros(len(off) - 1)
    _check(lib.adpsgd_average_noalloc(K, P, row_stride, off.ctypes.data_as(_I64P), len(off) - 1, x_ptr,
                                      var.ctypes.data_as(_DP), stream))
    return var


def adpsgd_schedule(ctx: int, var: np.ndarray) -> int:
    v = np.ascontiguousarray(var, dtype=np.float64)
    p = C.c_int32()
    _check(lib.adpsgd_schedule(ctx, v.ctypes.data_as(_DP), C.byref(p)))
    return p.value


def adpsgd_run(ctx: int, n_steps: int, T: int, log_cap: Optional[int] = None, with_var: bool = True):
    """Returns (records [n_logged] as a structured array, var_log [n_logged, T] or None, n_syncs)."""
    cap = n_steps if log_cap is None else log_cap
    log = (adpsgd_sync_rec * max(cap, 1))()
    var_log = np.zeros((max(cap, 1), T)) if with_var else None
    n = C.c_int64()
    _check(lib.adpsgd_run(ctx, n_steps, log, cap, None if var_log is None else var_log.ctypes.data_as(_DP),
                          C.byref(n)))
    k = min(n.value, cap)
    recs = np.zeros(k, dtype=[("t", np.int64), ("p", np.int32), ("S", np.float64), ("C2", np.float64),
                              ("gamma", np.float64), ("margin", np.float64)])
    for i in range(k):
        r = log[i]
        recs[i] = (r.t, r.p, r.S, r.C2, r.gamma, r.margin)
    return recs, (None if var_log is None else var_log[:k].copy()), n.value


def adpsgd_run_traced(ctx: int, n_steps: int, T: int, log_cap: Optional[int] = None, with_var: bool = True):
    """adpsgd_run plus one record per step; returns (records, var_log, n_syncs, steps).

    steps is a structured array with fields t, synced, p, var, grad_norm2, gamma."""
    cap = n_steps if log_cap is None else log_cap
    log = (adpsgd_sync_rec * max(cap, 1))()
    var_log = np.zeros((max(cap, 1), T)) if with_var else None
    trace = (adpsgd_step_rec * max(n_steps, 1))()
    n = C.c_int64()
    _check(lib.adpsgd_run_traced(ctx, n_steps, log, cap,
                                 None if var_log is None else var_log.ctypes.data_as(_DP),
                                 trace, n_steps, C.byref(n)))
    k = min(n.value, cap)
    recs = np.zeros(k, dtype=[("t", np.int64), ("p", np.int32), ("S", np.float64), ("C2", np.float64),
                              ("gamma", np.float64), ("margin", np.float64)])
    for i in range(k):
        r = log[i]
        recs[i] = (r.t, r.p, r.S, r.C2, r.gamma, r.margin)
    steps = np.zeros(n_steps, dtype=[("t", np.int64), ("synced", np.int32), ("p", np.int32),
                                     ("var", np.float64), ("grad_norm2", np.float64), ("gamma", np.float64)])
    for i in range(n_steps):
        r = trace[i]
        steps[i] = (r.t, r.synced, r.p, r.var, r.grad_norm2, r.gamma)
    return recs, (None if var_log is None else var_log[:k].copy()), n.value, steps


def adpsgd_get_state(ctx: int) -> adpsgd_state:
    st = adpsgd_state()
    _check(lib.adpsgd_get_state(ctx, C.byref(st)))
    return st


def adpsgd_set_state(ctx: int, st: adpsgd_state) -> None:
    _check(lib.adpsgd_set_state(ctx, C.byref(st)))


def adpsgd_set_step_launch(ctx: int, block: int, lds_bytes: int = 0, row_chunks: int = 1) -> None:
    _check(lib.adpsgd_set_step_launch(ctx, block, lds_bytes, row_chunks))


def adpsgd_get_step_launch(ctx: int) -> tuple:
    """(threads per block, LDS bytes reserved per block, chunks per row run)."""
    b, s, r = C.c_int32(), C.c_int32(), C.c_int32()
    _check(lib.adpsgd_get_step_launch(ctx, C.byref(b), C.byref(s), C.byref(r)))
    return b.value, s.value, r.value


def adpsgd_set_launch_policy(ctx: int, policy: int) -> None:
    _check(lib.adpsgd_set_launch_policy(ctx, policy))


def adpsgd_set_timing(ctx: int, every) -> None:
    """every: False/0 off, True/1 every launch, n > 1 every n-th launch of each kind."""
    _check(lib.adpsgd_set_timing(ctx, int(every)))


def adpsgd_get_timing(ctx: int) -> adpsgd_timing:
    t = adpsgd_timing()
    _check(lib.adpsgd_get_timing(ctx, C.byref(t)))
    return t


def adpsgd_destroy(ctx: int) -> None:
    _check(lib.adpsgd_destroy(ctx))


def adpsgd_philox_dump(seed: int, c1: int, c2: int, c3: int, g0: int, n_groups: int, dev_out_ptr: int,
                       stream: int) -> None:
    _check(lib.adpsgd_philox_dump(seed, c1, c2, c3, g0, n_groups, dev_out_ptr, stream))


def adpsgd_normal_dump(seed: int, c1: int, c2: int, c3: int, g0: int, n_groups: int, dev_out_ptr: int,
                       stream: int) -> None:
    _check(lib.adpsgd_normal_dump(seed, c1, c2, c3, g0, n_groups, dev_out_ptr, stream))


def adpsgd_lr(hp: adpsgd_hparams, t: int) -> float:
    return float(lib.adpsgd_lr(C.byref(hp), t))


def adpsgd_sched_init(hp: adpsgd_hparams) -> adpsgd_state:
    st = adpsgd_state()
    _check(lib.adpsgd_sched_init(C.byref(hp), C.byref(st)))
    return st


def adpsgd_sched_step(hp: adpsgd_hparams, st: adpsgd_state) -> bool:
    """Begins step st.t (updates st in place); True if a sync follows it."""
    due = C.c_int32()
    _check(lib.adpsgd_sched_step(C.byref(hp), C.byref(st), C.byref(due)))
    return bool(due.value)


def adpsgd_sched_on_sync(hp: adpsgd_hparams, st: adpsgd_state, t: int, S: float) -> float:
    """Updates st in place; returns the decision margin (NaN if no decision)."""
    margin = C.c_double()
    _check(lib.adpsgd_sched_on_sync(C.byref(hp), C.byref(st), t, S, C.byref(margin)))
    return margin.value
