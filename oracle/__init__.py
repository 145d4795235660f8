"""CPU oracle for StageFrontier frontier accounting -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never calls it;
the GPU path and the oracle share no code.

Two independent statements of the same definitions (Sec. 3, Eq. (1) and
Eq. (2); top-2 routing, the routing candidate set, the lag and the
localization evidence of Sec. 4; the direct-exposure gain of Eq. (4); the per-stage
baselines of Props. 1-2; the closure of Appendix A):

* ``frontier`` / ``window_summary`` -- plain C nested loops in
  ``sf_oracle.c`` (fast enough for the full workloads on sampled steps),
  called through ctypes on numpy arrays;
* ``pyref`` -- the same definitions as pure-Python loops for tiny inputs.

Both follow the readings documented in ``sf_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sf_oracle.c")
_LIB = os.path.join(_HERE, "libsforacle.so")


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the C oracle with gcc (plain -O2, single thread)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared",
             src, "-o", tmp])
        os.replace(tmp, out)
    return out


class COracle:
    """ctypes view of one compiled copy of ``sf_oracle.c``."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        lib.sfo_frontier.argtypes = [vp, i64, i32, i32, vp, vp]
        lib.sfo_frontier.restype = ctypes.c_int
        lib.sfo_window_summary.argtypes = [vp, vp, i64, i32, i32, i64, vp, vp, vp]
        lib.sfo_window_summary.restype = None
        lib.sfo_window_lead_exposed.argtypes = [vp, vp, i64, i32, i32, i64, vp, vp]
        lib.sfo_window_lead_exposed.restype = None
        lib.sfo_window_leader_switches.argtypes = [vp, vp, vp, i64, i32, i64, i64, vp, vp]
        lib.sfo_window_leader_switches.restype = None
        lib.sfo_frontier_evidence.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp]
        lib.sfo_frontier_evidence.restype = ctypes.c_int
        lib.sfo_ingest.argtypes = [vp, vp, i64, i32, i32, vp, vp]
        lib.sfo_ingest.restype = None
        lib.sfo_route.argtypes = [vp, i64, i32, i64, i64, vp, vp]
        lib.sfo_route.restype = None
        lib.sfo_exposure_gain.argtypes = [vp, vp, i64, i32, i32, i64, vp, vp, vp, vp]
        lib.sfo_exposure_gain.restype = ctypes.c_int
        lib.sfo_frontier_lag.argtypes = [vp, i64, i32, i32, vp, vp]
        lib.sfo_frontier_lag.restype = ctypes.c_int
        lib.sfo_rank_spread.argtypes = [vp, i64, i32, i32, i64, vp, vp]
        lib.sfo_rank_spread.restype = ctypes.c_int
        lib.sfo_window_median.argtypes = [vp, i64, i32, i32, i64, vp]
        lib.sfo_window_median.restype = ctypes.c_int
        lib.sfo_range_status.argtypes = [vp, i64, i32, i32]
        lib.sfo_range_status.restype = ctypes.c_int
        self.lib = lib
        self.path = path

    def frontier(self, d: np.ndarray):
        """Eq. (1) for every step.

        ``d``: int64 array of shape [T, S, R] (ns).  Returns ``(inc, lead)``
        with shapes [T, S] (int64 ns and int32 rank).
        """
        d = np.ascontiguousarray(d, dtype=np.int64)
        if d.ndim != 3:
            raise ValueError("durations must be [T, S, R]")
        T, S, R = d.shape
        inc = np.empty((T, S), dtype=np.int64)
        lead = np.empty((T, S), dtype=np.int32)
        if T and S and R:
            rc = self.lib.sfo_frontier(d.ctypes.data, T, R, S,
                                       inc.ctypes.data, lead.ctypes.data)
            if rc != 0:
                raise MemoryError("oracle prefix scratch allocation failed")
        return inc, lead

    def frontier_evidence(self, d: np.ndarray):
        """Eq. (1) plus the localization evidence of Sec. 4 and the
        per-stage baselines of Props. 1-2, for every boundary.

        Returns a dict of [T, S] arrays: ``inc``, ``lead``, ``gap`` (int64),
        ``ties`` (int32), ``stage_max``, ``stage_sum`` (int64).
        """
        d = np.ascontiguousarray(d, dtype=np.int64)
        if d.ndim != 3:
            raise ValueError("durations must be [T, S, R]")
        T, S, R = d.shape
        out = {k: np.empty((T, S), dtype=np.int32 if k in ("lead", "ties") else np.int64)
               for k in ("inc", "lead", "gap", "ties", "stage_max", "stage_sum")}
        if T and S and R:
            rc = self.lib.sfo_frontier_evidence(
                d.ctypes.data, T, R, S, *(out[k].ctypes.data for k in
                                          ("inc", "lead", "gap", "ties", "stage_max", "stage_sum")))
            if rc != 0:
                raise MemoryError("oracle prefix scratch allocation failed")
        return out

    def window_leader_switches(self, lead: np.ndarray, gap: np.ndarray, ties: np.ndarray,
                               window: int, min_gap: int = 0):
        """Leader switches between confident unique leaders per window and
        stage (Sec. 4 localization evidence).  ``lead``, ``ties`` int32 and
        ``gap`` int64, all [T, S] (as from ``frontier_evidence``).

        Returns ``(switches [W,S] int32, eligible [W,S] int32)``.
        """
        lead = np.ascontiguousarray(lead, dtype=np.int32)
        gap = np.ascontiguousarray(gap, dtype=np.int64)
        ties = np.ascontiguousarray(ties, dtype=np.int32)
        T, S = lead.shape
        assert gap.shape == (T, S) and ties.shape == (T, S)
        W = num_windows(T, window)
        sw = np.empty((W, S), dtype=np.int32)
        el = np.empty((W, S), dtype=np.int32)
        if W:
            self.lib.sfo_window_leader_switches(lead.ctypes.data, gap.ctypes.data, ties.ctypes.data,
                                                T, S, window, min_gap, sw.ctypes.data, el.ctypes.data)
        return sw, el

    def ingest(self, x: np.ndarray, w: np.ndarray):
        """Appendix A closure and the transpose to [T][S][R].

        ``x``: int64 [R, T, K] explicit stage durations per rank; ``w``: int64
        [R, T] step wall times.  Returns ``(d [T, K+1, R], o [T, R])``.
        """
        x = np.ascontiguousarray(x, dtype=np.int64)
        w = np.ascontiguousarray(w, dtype=np.int64)
        R, T, K = x.shape
        assert w.shape == (R, T)
        d = np.empty((T, K + 1, R), dtype=np.int64)
        o = np.empty((T, R), dtype=np.int64)
        if R and T:
            self.lib.sfo_ingest(x.ctypes.data, w.ctypes.data, T, R, K, d.ctypes.data, o.ctypes.data)
        return d, o

    def route(self, exposed: np.ndarray, tau_num: int = 4, tau_den: int = 5):
        """Routing candidate set per window: ``(order [W, S], size [W])``."""
        exposed = np.ascontiguousarray(exposed, dtype=np.int64)
        W, S = exposed.shape
        order = np.empty((W, S), dtype=np.int32)
        size = np.empty((W,), dtype=np.int32)
        if W and S:
            self.lib.sfo_route(exposed.ctypes.data, W, S, tau_num, tau_den,
                               order.ctypes.data, size.ctypes.data)
        return order, size

    def frontier_lag(self, d: np.ndarray):
        """Lag of the frontier over the (lower) median rank and its
        increment, [T, S] int64 each (Sec. 4)."""
        d = np.ascontiguousarray(d, dtype=np.int64)
        T, S, R = d.shape
        lag = np.empty((T, S), dtype=np.int64)
        inc = np.empty((T, S), dtype=np.int64)
        if T and S and R:
            if self.lib.sfo_frontier_lag(d.ctypes.data, T, R, S, lag.ctypes.data, inc.ctypes.data):
                raise MemoryError("oracle scratch allocation failed")
        return lag, inc

    def rank_spread(self, d: np.ndarray, window: int):
        """Raw rank spread of Sec. 6.2: max_r d - (lower) median_r d per
        step and stage, [T, S], and its window sums, [W, S] (int64)."""
        d = np.ascontiguousarray(d, dtype=np.int64)
        T, S, R = d.shape
        W = num_windows(T, window)
        spread = np.empty((T, S), dtype=np.int64)
        wspread = np.zeros((W, S), dtype=np.int64)
        if T and S and R:
            if self.lib.sfo_rank_spread(d.ctypes.data, T, R, S, window, spread.ctypes.data,
                                        wspread.ctypes.data):
                raise MemoryError("oracle scratch allocation failed")
        return spread, wspread

    def window_median(self, d: np.ndarray, window: int):
        """Per-rank window median (a baseline btilde of Eq. (4)): the lower
        median over each window's steps, [W, S, R] int64."""
        d = np.ascontiguousarray(d, dtype=np.int64)
        T, S, R = d.shape
        W = num_windows(T, window)
        med = np.empty((W, S, R), dtype=np.int64)
        if T and S and R:
            if self.lib.sfo_window_median(d.ctypes.data, T, R, S, window, med.ctypes.data):
                raise MemoryError("oracle scratch allocation failed")
        return med

    def range_status(self, d: np.ndarray) -> int:
        """2 (SF_ERANGE) if some duration is negative or some prefix reaches
        2^47 ns, else 0 (the data contract of Sec. 3 with the library's
        prefix bound)."""
        d = np.ascontiguousarray(d, dtype=np.int64)
        T, S, R = d.shape
        if not (T and S and R):
            return 0
        st = self.lib.sfo_range_status(d.ctypes.data, T, R, S)
        if st < 0:
            raise MemoryError("oracle scratch allocation failed")
        return st

    def exposure_gain(self, d: np.ndarray, btilde: np.ndarray, window: int):
        """Eq. (4) numerators and denominators.

        ``d``: int64 [T, S, R]; ``btilde``: int64 [W, S, R] baseline per
        window.  Returns a dict: ``gain`` [T, S], ``makespan`` [T],
        ``window_gain`` [W, S], ``window_makespan`` [W] (all int64).
        """
        d = np.ascontiguousarray(d, dtype=np.int64)
        btilde = np.ascontiguousarray(btilde, dtype=np.int64)
        T, S, R = d.shape
        W = num_windows(T, window)
        assert btilde.shape == (W, S, R)
        out = {"gain": np.empty((T, S), np.int64), "makespan": np.empty((T,), np.int64),
               "window_gain": np.empty((W, S), np.int64),
               "window_makespan": np.empty((W,), np.int64)}
        if T:
            rc = self.lib.sfo_exposure_gain(
                d.ctypes.data, btilde.ctypes.data, T, R, S, window,
                *(out[k].ctypes.data for k in ("gain", "makespan", "window_gain",
                                               "window_makespan")))
            if rc != 0:
                raise MemoryError("oracle scratch allocation failed")
        return out

    def window_summary(self, inc: np.ndarray, lead: np.ndarray, R: int, window: int):
        """Window reduction of per-step results.

        Returns ``(exposed [W,S] int64, counts [W,S,R] int32,
        top2 [W,2,2] int32)``.
        """
        inc = np.ascontiguousarray(inc, dtype=np.int64)
        lead = np.ascontiguousarray(lead, dtype=np.int32)
        T, S = inc.shape
        W = num_windows(T, window)
        exposed = np.empty((W, S), dtype=np.int64)
        counts = np.empty((W, S, R), dtype=np.int32)
        top2 = np.empty((W, 2, 2), dtype=np.int32)
        if W:
            self.lib.sfo_window_summary(
                inc.ctypes.data, lead.ctypes.data, T, R, S, window,
                exposed.ctypes.data, counts.ctypes.data, top2.ctypes.data)
        return exposed, counts, top2

    def window_lead_exposed(self, inc: np.ndarray, lead: np.ndarray, R: int, window: int):
        """Exposed time each rank led, per window and stage: the sum of the
        window's advances of the stage whose leader is that rank.

        Returns ``(lead_exposed [W,S,R] int64, top2 [W,2,2] int32)``: the
        top-2 stages of the window summary, each with the rank that led the
        most exposed time of it (lowest rank on ties, -1 if none led any).
        """
        inc = np.ascontiguousarray(inc, dtype=np.int64)
        lead = np.ascontiguousarray(lead, dtype=np.int32)
        T, S = inc.shape
        W = num_windows(T, window)
        out = np.empty((W, S, R), dtype=np.int64)
        top2 = np.empty((W, 2, 2), dtype=np.int32)
        if W:
            self.lib.sfo_window_lead_exposed(inc.ctypes.data, lead.ctypes.data, T, R, S, window,
                                             out.ctypes.data, top2.ctypes.data)
        return out, top2


def num_windows(T: int, window: int) -> int:
    return (T + window - 1) // window


_default = None


def _get() -> COracle:
    global _default
    if _default is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _default = COracle(_LIB)
    return _default


def frontier(d: np.ndarray):
    return _get().frontier(d)


def window_leader_switches(lead, gap, ties, window: int, min_gap: int = 0):
    return _get().window_leader_switches(lead, gap, ties, window, min_gap)


def window_lead_exposed(inc: np.ndarray, lead: np.ndarray, R: int, window: int):
    return _get().window_lead_exposed(inc, lead, R, window)


def window_summary(inc: np.ndarray, lead: np.ndarray, R: int, window: int):
    return _get().window_summary(inc, lead, R, window)


def frontier_evidence(d: np.ndarray):
    return _get().frontier_evidence(d)


def ingest(x: np.ndarray, w: np.ndarray):
    return _get().ingest(x, w)


def route(exposed: np.ndarray, tau_num: int = 4, tau_den: int = 5):
    return _get().route(exposed, tau_num, tau_den)


def exposure_gain(d: np.ndarray, btilde: np.ndarray, window: int):
    return _get().exposure_gain(d, btilde, window)


def frontier_lag(d: np.ndarray):
    return _get().frontier_lag(d)


def rank_spread(d: np.ndarray, window: int):
    return _get().rank_spread(d, window)


def window_median(d: np.ndarray, window: int):
    return _get().window_median(d, window)


def range_status(d: np.ndarray) -> int:
    return _get().range_status(d)


from . import pyref  # noqa: E402  (pure-Python twin, no compiled code)

__all__ = ["build", "COracle", "frontier", "frontier_evidence", "frontier_lag", "rank_spread",
           "window_median", "range_status", "ingest", "route",
           "exposure_gain",
           "window_summary", "num_windows", "pyref"]
