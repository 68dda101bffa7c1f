"""ORACLE -- test infrastructure, not product code.

ctypes binding of the fp64 CPU reference (``adpsgd_oracle.c``).  The shared
library is compiled with gcc from that one file; nothing here touches a GPU.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "adpsgd_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def lib_path() -> str:
    return _LIB


def build_oracle(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with plain IEEE fp64 (no fast-math, no FMA contraction)."""
    tmp = out + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
           src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class _Problem(C.Structure):
    _fields_ = [
        ("K", C.c_int32), ("T", C.c_int32), ("P", C.c_int64),
        ("offsets", C.POINTER(C.c_int64)), ("seed", C.c_uint64),
        ("sigma", C.c_double), ("momentum", C.c_double), ("weight_decay", C.c_double),
        ("h_lo", C.c_double), ("h_hi", C.c_double),
        ("lr_kind", C.c_int32), ("period_mode", C.c_int32),
        ("lr0", C.c_double), ("total_steps", C.c_int64), ("k_s", C.c_int64),
        ("thr_lo", C.c_double), ("thr_hi", C.c_double),
        ("p_init", C.c_int32), ("avg_momentum", C.c_int32),
        ("sync_warmup_steps", C.c_int64), ("p_switch_step", C.c_int64),
        ("p_after", C.c_int32), ("p_max", C.c_int32),
    ]


class _State(C.Structure):
    _fields_ = [("t", C.c_int64), ("cnt", C.c_int64), ("nC2", C.c_int64),
                ("C2", C.c_double), ("p", C.c_int32), ("pad_", C.c_int32)]


class _Sync(C.Structure):
    _fields_ = [("t", C.c_int64), ("p", C.c_int32), ("pad_", C.c_int32),
                ("S", C.c_double), ("C2", C.c_double), ("gamma", C.c_double)]


_D = C.POINTER(C.c_double)
_I64 = C.POINTER(C.c_int64)
_U32 = C.POINTER(C.c_uint32)


def _load():
    """The compiled oracle; ADPSGD_ORACLE_LIB names another build of the same
    source to load instead (the mutation test points the pins at copies with a
    planted mistake)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        path = os.environ.get("ADPSGD_ORACLE_LIB")
        if not path:
            path = _LIB
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build_oracle()
        lib = C.CDLL(path)
        lib.orc_philox4x32_10.argtypes = [_U32, _U32, _U32]
        lib.orc_normals4.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32, _D]
        lib.orc_lr.argtypes = [C.POINTER(_Problem), C.c_int64]
        lib.orc_lr.restype = C.c_double
        lib.orc_problem_data.argtypes = [C.POINTER(_Problem), _I64, C.c_int64, _D, _D]
        lib.orc_local_step.argtypes = [C.POINTER(_Problem), _I64, C.c_int64, C.c_int64, _D, _D, _D, _D]
        lib.orc_average.argtypes = [C.POINTER(_Problem), _I64, C.c_int64, _D, _D, _D]
        lib.orc_average.restype = C.c_double
        lib.orc_schedule_trace.argtypes = [C.POINTER(_Problem), C.POINTER(_State), C.c_int64, _D,
                                           _I64, C.POINTER(C.c_int32), C.c_int64]
        lib.orc_schedule_trace.restype = C.c_int64
        lib.orc_controller.argtypes = [C.POINTER(_Problem), C.POINTER(_State), C.c_int64, C.c_double]
        lib.orc_controller.restype = C.c_int
        lib.orc_state_init.argtypes = [C.POINTER(_Problem), C.POINTER(_State)]
        lib.orc_run.argtypes = [C.POINTER(_Problem), _I64, C.c_int64, C.POINTER(_State), C.c_int64,
                                _D, _D, _D, _D, C.POINTER(_Sync), C.c_int64, _D, _D, _D]
        lib.orc_variance.argtypes = [C.POINTER(_Problem), _I64, C.c_int64, _D, _D]
        lib.orc_variance.restype = C.c_double
        lib.orc_grad_norm2.argtypes = [C.POINTER(_Problem), C.c_int64, _D, _D, _D]
        lib.orc_grad_norm2.restype = C.c_double
        lib.orc_run.restype = C.c_int64
        lib.orc_mean_trajectory.argtypes = [C.POINTER(_Problem), _I64, C.c_int64, C.c_int64,
                                            C.c_int64, _D, _D, _D, _D]
        lib.orc_num_threads.restype = C.c_int
        lib.orc_box_muller.argtypes = [C.c_uint32, C.c_uint32, _D]
        lib.orc_philox_groups.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32,
                                          C.c_int64, C.c_int64, _U32]
        lib.orc_normals_groups.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_uint32,
                                           C.c_int64, C.c_int64, _D]
        _lib = lib
        return lib


def _dp(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(_D)


def _ip(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.int64 and a.flags.c_contiguous
    return a.ctypes.data_as(_I64)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def philox4x32_10(ctr, key) -> np.ndarray:
    lib = _load()
    c = (C.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (C.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (C.c_uint32 * 4)()
    lib.orc_philox4x32_10(c, k, o)
    return np.array(list(o), dtype=np.uint32)


def normals4(seed: int, c0: int, c1: int, c2: int, c3: int) -> np.ndarray:
    z = np.zeros(4, dtype=np.float64)
    _load().orc_normals4(seed, c0, c1, c2, c3, _dp(z))
    return z


def box_muller(ra: int, rb: int) -> np.ndarray:
    z = np.zeros(2)
    _load().orc_box_muller(ra & 0xFFFFFFFF, rb & 0xFFFFFFFF, _dp(z))
    return z


def philox_groups(seed: int, c1: int, c2: int, c3: int, g0: int, n: int) -> np.ndarray:
    """Raw Philox words of groups g0..g0+n-1, shape [n, 4] uint32."""
    out = np.zeros((n, 4), dtype=np.uint32)
    _load().orc_philox_groups(seed, c1, c2, c3, g0, n, out.ctypes.data_as(_U32))
    return out


def normals_groups(seed: int, c1: int, c2: int, c3: int, g0: int, n: int) -> np.ndarray:
    """Box-Muller normals of groups g0..g0+n-1, flat [4n] fp64."""
    z = np.zeros(4 * n)
    _load().orc_normals_groups(seed, c1, c2, c3, g0, n, _dp(z))
    return z


class Oracle:
    """One workload's problem, as the oracle sees it."""

    def __init__(self, w):
        self.w = w
        self._off = np.ascontiguousarray(w.offsets(), dtype=np.int64)
        self.pb = _Problem(
            K=w.K, T=w.T, P=w.P, offsets=self._off.ctypes.data_as(_I64), seed=w.seed,
            sigma=w.sigma, momentum=w.momentum, weight_decay=w.weight_decay,
            h_lo=w.h_lo, h_hi=w.h_hi, lr_kind=w.lr_kind, period_mode=w.period_mode,
            lr0=w.lr0, total_steps=w.total_steps, k_s=w.k_s, thr_lo=w.thr_lo,
            thr_hi=w.thr_hi, p_init=w.p_init, avg_momentum=1 if w.avg_momentum else 0,
            sync_warmup_steps=w.sync_warmup_steps, p_switch_step=w.p_switch_step,
            p_after=w.p_after, p_max=w.p_max)
        self.lib = _load()

    def lr(self, t: int) -> float:
        return float(self.lib.orc_lr(C.byref(self.pb), t))

    def problem_data(self, idx: Optional[np.ndarray] = None):
        n = self.w.P if idx is None else len(idx)
        h = np.zeros(n); xs = np.zeros(n)
        self.lib.orc_problem_data(C.byref(self.pb), _ip(idx), n, _dp(h), _dp(xs))
        return h, xs

    def local_step(self, t, x, v, h, xs, idx=None):
        n = x.shape[1]
        self.lib.orc_local_step(C.byref(self.pb), _ip(idx), n, t, _dp(h), _dp(xs), _dp(x), _dp(v))

    def average(self, x, idx=None, v=None):
        """Sync x (and v when the workload averages momentum); returns (S, var[T])."""
        var = np.zeros(self.w.T)
        S = self.lib.orc_average(C.byref(self.pb), _ip(idx), x.shape[1], _dp(x), _dp(v), _dp(var))
        return float(S), var

    def new_state(self):
        st = _State()
        self.lib.orc_state_init(C.byref(self.pb), C.byref(st))
        return st

    def controller(self, st, t: int, S: float) -> int:
        return int(self.lib.orc_controller(C.byref(self.pb), C.byref(st), t, S))

    def run(self, n_steps: Optional[int] = None, idx: Optional[np.ndarray] = None,
            h=None, xs=None, x=None, v=None, state=None, log_cap: Optional[int] = None,
            trace: bool = False):
        """Algorithm 2 for n_steps steps.  trace=True also records, per step, the
        replicas' variance before any sync and |grad F|^2 at their mean."""
        w = self.w
        n_steps = w.total_steps if n_steps is None else n_steps
        n = w.P if idx is None else len(idx)
        if idx is not None:
            idx = np.ascontiguousarray(idx, dtype=np.int64)
            assert np.all(np.diff(idx) > 0)
        if h is None or xs is None:
            h0, xs0 = self.problem_data(idx)
            h = h0 if h is None else h
            xs = xs0 if xs is None else xs
        x = np.zeros((w.K, n)) if x is None else x
        v = np.zeros((w.K, n)) if v is None else v
        st = self.new_state() if state is None else state
        cap = n_steps if log_cap is None else log_cap
        log = (_Sync * max(cap, 1))()
        var_log = np.zeros((max(cap, 1), w.T))
        tv = np.zeros(max(n_steps, 1)) if trace else None
        tg = np.zeros(max(n_steps, 1)) if trace else None
        rc = self.lib.orc_run(C.byref(self.pb), _ip(idx), n, C.byref(st), n_steps,
                              _dp(h), _dp(xs), _dp(x), _dp(v), log, cap, _dp(var_log), _dp(tv), _dp(tg))
        if rc < 0:
            raise RuntimeError(f"oracle run failed: {rc}")
        k = min(int(rc), cap)
        recs = [(log[i].t, log[i].p, log[i].S, log[i].C2, log[i].gamma) for i in range(k)]
        return OracleRun(x=x, v=v, h=h, xs=xs, state=st, n_syncs=int(rc),
                         sync_t=np.array([r[0] for r in recs], dtype=np.int64),
                         sync_p=np.array([r[1] for r in recs], dtype=np.int64),
                         S=np.array([r[2] for r in recs]), C2=np.array([r[3] for r in recs]),
                         gamma=np.array([r[4] for r in recs]), var=var_log[:k].copy(),
                         trace_var=None if tv is None else tv[:n_steps].copy(),
                         trace_grad_norm2=None if tg is None else tg[:n_steps].copy())

    def variance(self, x, idx=None):
        """The replicas' variance without averaging them: (Var[W], per-tensor terms)."""
        var = np.zeros(self.w.T)
        S = self.lib.orc_variance(C.byref(self.pb), _ip(idx), x.shape[1], _dp(x), _dp(var))
        return float(S), var

    def grad_norm2(self, x, h, xs):
        return float(self.lib.orc_grad_norm2(C.byref(self.pb), x.shape[1], _dp(x), _dp(h), _dp(xs)))

    def mean_trajectory(self, n_steps, idx=None, h=None, xs=None, t0=0, xbar=None, vbar=None):
        n = self.w.P if idx is None else len(idx)
        if idx is not None:
            idx = np.ascontiguousarray(idx, dtype=np.int64)
        if h is None or xs is None:
            h, xs = self.problem_data(idx)
        xbar = np.zeros(n) if xbar is None else xbar
        vbar = np.zeros(n) if vbar is None else vbar
        self.lib.orc_mean_trajectory(C.byref(self.pb), _ip(idx), n, t0, n_steps,
                                     _dp(h), _dp(xs), _dp(xbar), _dp(vbar))
        return xbar, vbar


@dataclass
class OracleRun:
    x: np.ndarray
    v: np.ndarray
    h: np.ndarray
    xs: np.ndarray
    state: object
    n_syncs: int
    sync_t: np.ndarray
    sync_p: np.ndarray
    S: np.ndarray
    C2: np.ndarray
    gamma: np.ndarray
    var: np.ndarray
    trace_var: Optional[np.ndarray] = None
    trace_grad_norm2: Optional[np.ndarray] = None


def problem_data(w, idx=None):
    return Oracle(w).problem_data(idx)


def lr(w, t: int) -> float:
    return Oracle(w).lr(t)


def controller_trace(w, S_of_sync, through_nonfinite: bool = False):
    """Drive the oracle's schedule with scripted variances.

    S_of_sync(t, gamma) gives S for a sync after step t.  Returns the list of
    (t, p in force) syncs over w.total_steps steps and the final state.  A
    non-finite S stops the oracle's schedule at that sync (with its counter
    restarted); through_nonfinite=True then resumes it from the state it left,
    else FloatingPointError is raised.
    """
    o = Oracle(w)
    st = o.new_state()
    N = w.total_steps
    S = np.array([float(S_of_sync(t, o.lr(t))) for t in range(N)])
    out = []
    while st.t < N:
        left = N - st.t
        sync_t = np.full(left, -1, dtype=np.int64)
        sync_p = np.zeros(left, dtype=np.int32)
        n = o.lib.orc_schedule_trace(C.byref(o.pb), C.byref(st), left, _dp(S), _ip(sync_t),
                                     sync_p.ctypes.data_as(C.POINTER(C.c_int32)), left)
        if n >= 0:
            out += [(int(a), int(b)) for a, b in zip(sync_t[:n], sync_p[:n])]
            break
        if not through_nonfinite:
            raise FloatingPointError(n)
        k = int(np.count_nonzero(sync_t >= 0))   # syncs recorded up to the failing one
        out += [(int(a), int(b)) for a, b in zip(sync_t[:k], sync_p[:k])]
    return out, st
