"""Seeded synthetic stage-duration workloads (int64 ns, layout [T][S][R]).

The generator is shared by the GPU tests, the benchmark and the oracle
tests, and holds no part of the accounting method.  The heavy sampling runs
in ``sfsynth.c`` (counter-based, OpenMP over steps); the few sparse
injections (faults, stalls, ties) are applied here with numpy.

Workload recipes stand in for the paper's private training runs: six broad
stages in the default order of the stage taxonomy (Appendix A), a step of
about 220 ms at the default stage bases, hidden-rank host delays of tens of
milliseconds injected into one rank's span (Sec. 6), and windows of hundreds
of steps.
"""
from __future__ import annotations

import ctypes
import math
import os
import statistics
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sfsynth.c")
_LIB = os.path.join(_HERE, "libsfsynth.so")

MS = 1_000_000  # ns per ms
QBITS = 12      # 4096 interpolation intervals per stage table

# stream ids for independent SplitMix64 keys
_ST_BASE, _ST_TAIL, _ST_FAULT, _ST_ROLE, _ST_TIE, _ST_STRAG = 1, 2, 3, 4, 5, 6

_lib = None


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O3", "-std=gnu11", "-fopenmp", "-fPIC", "-shared",
             _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        i64, i32, u64, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_void_p
        lib.sfs_generate.argtypes = [i64, i64, i32, i32, vp, i32, u64, u64, u64,
                                     i64, i32, i64, i64, i32, vp, vp, i32]
        lib.sfs_generate.restype = None
        lib.sfs_splitmix64_at.argtypes = [u64, u64]
        lib.sfs_splitmix64_at.restype = u64
        _lib = lib
    return _lib


def splitmix64_at(key: int, i: int) -> int:
    return int(_load().sfs_splitmix64_at(key, i))


def _key(seed: int, stream: int) -> int:
    """Independent SplitMix64 key per (seed, stream)."""
    return splitmix64_at(seed & 0xFFFFFFFFFFFFFFFF, stream)


class _Stream:
    """Sequential draws from one SplitMix64 sequence (host-side choices)."""

    def __init__(self, seed: int, stream: int):
        self.k = _key(seed, stream)
        self.i = 0

    def u64(self) -> int:
        v = splitmix64_at(self.k, self.i)
        self.i += 1
        return v

    def below(self, n: int) -> int:
        """Uniform integer in [0, n) (rejection-free multiply-shift)."""
        return (self.u64() * n) >> 64

    def between(self, lo: int, hi: int) -> int:
        """Uniform integer in [lo, hi] inclusive."""
        return lo + self.below(hi - lo + 1)

    def distinct(self, n: int, k: int) -> list[int]:
        """k distinct integers from [0, n), in draw order."""
        seen, out = set(), []
        while len(out) < k:
            v = self.below(n)
            if v not in seen:
                seen.add(v)
                out.append(v)
        return out


def lognormal_table(base_ns: float, sigma: float, qbits: int = QBITS) -> np.ndarray:
    """Quantile nodes of lognormal(mu=ln(base), sigma) at probabilities
    (k + 1/2) / (2^qbits + 1), k = 0 .. 2^qbits, rounded to integer ns."""
    n = (1 << qbits) + 1
    nd = statistics.NormalDist()
    return np.array([round(base_ns * math.exp(sigma * nd.inv_cdf((k + 0.5) / n)))
                     for k in range(n)], dtype=np.int64)


@dataclass(frozen=True)
class Workload:
    name: str
    R: int
    S: int
    T: int
    window: int
    stages: tuple
    base_ms: tuple
    sigma: float
    seed: int
    chunks: int = 1                 # step-axis chunks the benchmark streams
    tail_prob: float = 0.0          # per-sample probability of x tail_mult
    tail_mult: int = 1
    straggler_pct: int = 0          # persistent straggler: + pct % on all stages
    role_groups: int = 0            # rank role groups with additive offsets
    role_off_ms: tuple = (0, 0)     # offset range per (group, stage), ms
    stall_frac: float = 0.0         # steps with a data stall on one rank, seen as bwd wait elsewhere
    stall_ms: int = 0
    fault_frac: float = 0.0         # single (stage, rank) delays
    fault_ms: tuple = (0, 0)
    tie_frac: float = 0.0           # fraction of (t, s) boundaries made exact ties
    tie_ms: int = 0
    note: str = field(default="", compare=False)

    @property
    def samples(self) -> int:
        return self.T * self.S * self.R

    @property
    def input_bytes(self) -> int:
        return 8 * self.samples

    @property
    def num_windows(self) -> int:
        return (self.T + self.window - 1) // self.window

    def chunk_bounds(self):
        step = (self.T + self.chunks - 1) // self.chunks
        return [(t0, min(t0 + step, self.T)) for t0 in range(0, self.T, step)]


_S6 = ("data", "fwd", "bwd", "callback", "optim", "other")
_B6 = (20, 60, 120, 2, 15, 3)
_S8 = ("data", "all_gather", "fwd", "bwd", "reduce_scatter", "callback", "optim", "other")
_B8 = (20, 8, 60, 120, 6, 2, 15, 3)
_S12 = ("data", "fwd_mb0", "fwd_mb1", "fwd_mb2", "fwd_mb3",
        "bwd_mb0", "bwd_mb1", "bwd_mb2", "bwd_mb3", "callback", "optim", "other")
_B12 = (10, 20, 20, 20, 20, 40, 40, 40, 40, 5, 15, 5)

WORKLOADS = {
    "r8_s6_t1k": Workload(
        "r8_s6_t1k", R=8, S=6, T=1000, window=100, stages=_S6, base_ms=_B6,
        sigma=0.05, seed=1001, stall_frac=0.05, stall_ms=30,
        note="5% of steps: one seeded rank +30 ms data, others +30 ms bwd wait"),
    "r128_s6_t100k": Workload(
        "r128_s6_t100k", R=128, S=6, T=100_000, window=1000, stages=_S6,
        base_ms=_B6, sigma=0.1, seed=1002, fault_frac=0.01, fault_ms=(10, 50),
        note="1% of steps: one (stage, rank) +U[10,50] ms"),
    "r1024_s8_t50k": Workload(
        "r1024_s8_t50k", R=1024, S=8, T=50_000, window=500, stages=_S8,
        base_ms=_B8, sigma=0.15, seed=1003, tail_prob=0.001, tail_mult=10,
        straggler_pct=3, note="heavy tail x10 at p=0.001; straggler +3%"),
    "r4096_s12_t20k": Workload(
        "r4096_s12_t20k", R=4096, S=12, T=20_000, window=250, stages=_S12,
        base_ms=_B12, sigma=0.1, seed=1004, role_groups=4, role_off_ms=(0, 5),
        tie_frac=0.01, tie_ms=200,
        note="4 role groups, offsets U[0,5] ms; exact ties on 1% of boundaries"),
    "r16384_s12_t20k": Workload(
        "r16384_s12_t20k", R=16384, S=12, T=20_000, window=1000, stages=_S12,
        base_ms=_B12, sigma=0.1, seed=1005, chunks=2, fault_frac=0.005,
        fault_ms=(5, 100), note="0.5% of steps: one (stage, rank) +U[5,100] ms"),
}
# order from smallest to largest
WORKLOAD_ORDER = ["r8_s6_t1k", "r128_s6_t100k", "r1024_s8_t50k",
                  "r4096_s12_t20k", "r16384_s12_t20k"]


def straggler_rank(wl: Workload) -> int:
    """The seeded persistent straggler rank, or -1."""
    return _Stream(wl.seed, _ST_STRAG).below(wl.R) if wl.straggler_pct else -1


def _tables(wl: Workload) -> np.ndarray:
    return np.stack([lognormal_table(b * MS, wl.sigma) for b in wl.base_ms])


_TABLE_CACHE: dict = {}


def injections(wl: Workload):
    """The sparse, seeded edits of a workload, as a list of
    (t, kind, args) tuples sorted by t (host-side, deterministic)."""
    out = []
    st = _Stream(wl.seed, _ST_FAULT)
    if wl.stall_frac:
        n = round(wl.stall_frac * wl.T)
        rank = st.below(wl.R)
        for t in sorted(st.distinct(wl.T, n)):
            out.append((t, "stall", (rank, wl.stall_ms * MS)))
    if wl.fault_frac:
        n = round(wl.fault_frac * wl.T)
        for t in st.distinct(wl.T, n):
            s = st.below(wl.S)
            r = st.below(wl.R)
            delay = st.between(wl.fault_ms[0] * MS, wl.fault_ms[1] * MS)
            out.append((t, "fault", (s, r, delay)))
    if wl.tie_frac:
        ts = _Stream(wl.seed, _ST_TIE)
        n = round(wl.tie_frac * wl.T * wl.S)
        for b in sorted(ts.distinct(wl.T * wl.S, n)):
            t, s = divmod(b, wl.S)
            r1 = ts.below(wl.R)
            r2 = (r1 + 1 + ts.below(wl.R - 1)) % wl.R
            out.append((t, "tie", (s, r1, r2, wl.tie_ms * MS)))
    out.sort(key=lambda e: e[0])
    return out


def _apply(buf: np.ndarray, wl: Workload, t0: int, t1: int, inj):
    data = wl.stages.index("data") if "data" in wl.stages else 0
    bwd = [i for i, n in enumerate(wl.stages) if n.startswith("bwd")]
    for t, kind, args in inj:
        if t < t0 or t >= t1:
            continue
        x = buf[t - t0]
        if kind == "stall":
            # one rank's data stage is late; the others observe the same
            # group delay as wait in their backward stage (Sec. 2 pattern)
            rank, delay = args
            x[data, rank] += delay
            others = np.arange(wl.R) != rank
            x[bwd[0], others] += delay
        elif kind == "fault":
            s, r, delay = args
            x[s, r] += delay
        elif kind == "tie":
            # rank r2 repeats rank r1's stages 0..s, then both get the same
            # extra delay at s: their prefixes at s are equal by construction
            s, r1, r2, delay = args
            x[: s + 1, r2] = x[: s + 1, r1]
            x[s, r1] += delay
            x[s, r2] += delay


def generate(wl: Workload, t0: int = 0, t1: int | None = None,
             out: np.ndarray | None = None, threads: int | None = None) -> np.ndarray:
    """Steps [t0, t1) of workload ``wl`` as an int64 [t1-t0, S, R] array."""
    if t1 is None:
        t1 = wl.T
    n = t1 - t0
    if out is None:
        out = np.empty((n, wl.S, wl.R), dtype=np.int64)
    assert out.shape == (n, wl.S, wl.R) and out.dtype == np.int64 and out.flags.c_contiguous
    if n == 0:
        return out
    key = wl.name
    if key not in _TABLE_CACHE:
        _TABLE_CACHE[key] = (np.ascontiguousarray(_tables(wl)), injections(wl))
    tables, inj = _TABLE_CACHE[key]
    groups = wl.role_groups
    if groups:
        rs = _Stream(wl.seed, _ST_ROLE)
        goff = np.array([[rs.between(wl.role_off_ms[0] * MS, wl.role_off_ms[1] * MS)
                          for _ in range(wl.S)] for _ in range(groups)], dtype=np.int64)
    else:
        goff = np.zeros((1, wl.S), dtype=np.int64)
    thresh = int(wl.tail_prob * 2.0 ** 64) if wl.tail_prob else 0
    if threads is None:
        threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or (os.cpu_count() or 1)
    _load().sfs_generate(
        t0, t1, wl.R, wl.S, tables.ctypes.data, QBITS,
        _key(wl.seed, _ST_BASE), _key(wl.seed, _ST_TAIL), thresh, wl.tail_mult,
        straggler_rank(wl), wl.straggler_pct, 100,
        groups, goff.ctypes.data, out.ctypes.data, threads)
    _apply(out, wl, t0, t1, inj)
    return out


def random_durations(T: int, S: int, R: int, seed: int, lo: int = 0, hi: int = 1000) -> np.ndarray:
    """Small uniform int64 [T, S, R] matrix in [lo, hi] for shape sweeps.
    A narrow range (e.g. hi=3) makes exact prefix ties frequent."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(lo, hi + 1, size=(T, S, R), dtype=np.int64)
