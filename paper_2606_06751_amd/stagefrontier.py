"""Python binding of libstagefrontier (ctypes; argument marshalling only).

Every function has the name of the C entry point it wraps (declared in
``include/stagefrontier.h``).  Arrays are torch tensors on the GPU; torch is
used for device memory and streams only, and every step of the computation
runs in the library's HIP kernels.  There is no fallback: if the library is
missing, importing this module raises.
"""
from __future__ import annotations

import ctypes
import functools
import os

import torch  # loaded first so that the library binds to torch's HIP runtime

from . import build as _build

SF_OK, SF_EINVAL, SF_ERANGE, SF_EHIP = 0, 1, 2, 3
SF_MAX_R = 65536
SF_MAX_PREFIX_NS = 1 << 47
SF_XOR_PIECE_BYTES = 262144

LIB_PATH = _build.LIB


class StageFrontierError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, sf_strerror(status), status))


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "libstagefrontier.so is not built (expected at %s); run "
            "`python -c 'import __graft_entry__ as g; g.build()'` first" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    lib.sf_frontier.argtypes = [vp, i64, i32, i32, vp, vp, vp]
    lib.sf_frontier.restype = ctypes.c_int
    lib.sf_frontier_checked.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp]
    lib.sf_frontier_checked.restype = ctypes.c_int
    lib.sf_frontier_evidence.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    lib.sf_frontier_evidence.restype = ctypes.c_int
    lib.sf_ingest.argtypes = [vp, vp, i64, i32, i32, vp, vp, vp]
    lib.sf_ingest.restype = ctypes.c_int
    lib.sf_route.argtypes = [vp, i64, i32, i64, i64, vp, vp, vp]
    lib.sf_route.restype = ctypes.c_int
    lib.sf_exposure_gain.argtypes = [vp, vp, i64, i32, i32, i64, vp, vp, vp, vp, vp]
    lib.sf_exposure_gain.restype = ctypes.c_int
    lib.sf_frontier_lag.argtypes = [vp, i64, i32, i32, vp, vp, vp]
    lib.sf_frontier_lag.restype = ctypes.c_int
    lib.sf_rank_spread.argtypes = [vp, i64, i32, i32, i64, vp, vp, vp]
    lib.sf_rank_spread.restype = ctypes.c_int
    lib.sf_window_median.argtypes = [vp, i64, i32, i32, i64, vp, vp]
    lib.sf_window_median.restype = ctypes.c_int
    lib.sf_read_xor.argtypes = [vp, i64, vp, vp]
    lib.sf_read_xor.restype = ctypes.c_int
    lib.sf_read_xor_pieces.argtypes = [i64]
    lib.sf_read_xor_pieces.restype = i64
    lib.sf_num_windows.argtypes = [i64, i64]
    lib.sf_num_windows.restype = i64
    lib.sf_window_summary.argtypes = [vp, vp, i64, i32, i32, i64, vp, vp, vp, vp]
    lib.sf_window_summary.restype = ctypes.c_int
    lib.sf_frontier_summary.argtypes = [vp, i64, i32, i32, i64, vp, vp, vp, vp, vp, vp]
    lib.sf_frontier_summary.restype = ctypes.c_int
    lib.sf_window_lead_exposed.argtypes = [vp, vp, i64, i32, i32, i64, vp, vp, vp]
    lib.sf_window_lead_exposed.restype = ctypes.c_int
    lib.sf_window_leader_switches.argtypes = [vp, vp, vp, i64, i32, i64, i64, vp, vp, vp]
    lib.sf_window_leader_switches.restype = ctypes.c_int
    lib.sf_strerror.argtypes = [ctypes.c_int]
    lib.sf_strerror.restype = ctypes.c_char_p
    lib.sf_version.argtypes = []
    lib.sf_version.restype = ctypes.c_char_p
    return lib


_lib = _load()


def sf_strerror(status: int) -> str:
    return _lib.sf_strerror(status).decode()


def sf_version() -> str:
    return _lib.sf_version().decode()


def sf_num_windows(T: int, window: int) -> int:
    return int(_lib.sf_num_windows(T, window))


@functools.lru_cache(maxsize=64)
def _num_windows(T: int, window: int) -> int:
    """sf_num_windows, remembered for the (T, window) pairs a caller repeats."""
    return int(_lib.sf_num_windows(T, window))


def _stream(stream, device):
    """The torch stream a call runs on: ``stream`` (a torch stream or a raw
    hipStream_t handle), else the current stream of ``device``."""
    if stream is None:
        return torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=device)


def _stream_handle(stream, device) -> int:
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(_stream(stream, device).cuda_stream)


def _new(shape, dtype, device, stream, zero: bool = False) -> torch.Tensor:
    """An output the binding allocates for a call on ``stream``.  It is
    allocated (and, with ``zero``, cleared) on that stream, so the clear is
    ordered before the call's kernels and the caching allocator does not hand
    the block to other work while they may still use it."""
    with torch.cuda.stream(_stream(stream, device)):
        if zero:
            return torch.zeros(shape, dtype=dtype, device=device)
        return torch.empty(shape, dtype=dtype, device=device)


def _check(t: torch.Tensor, name: str, dtype, shape, like: torch.Tensor | None = None):
    """Type, device, layout and shape of one argument; ``like``: the call's
    first array, whose device every other array must share.  (One chained
    test of cheap attribute reads on the good path: launch-bound callers pay
    for it per call; the reason is worked out only on failure.)"""
    try:
        if (t.dtype is dtype and t.is_cuda and t.shape == shape and t.is_contiguous()
                and (like is None or t.get_device() == like.get_device())):
            return
    except AttributeError:
        raise TypeError("%s must be a torch.Tensor" % name) from None
    if t.dtype is not dtype or not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a %s torch.Tensor, got %r" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if t.shape != shape:
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    raise ValueError("%s is on %s, the call's other arrays on %s" % (name, t.device, like.device))


def sf_frontier(durations: torch.Tensor, out_increment: torch.Tensor | None = None,
                out_leader: torch.Tensor | None = None, stream=None):
    """Frontier advances and leaders of every step (``sf_frontier``).

    ``durations``: int64 GPU tensor [T, S, R] (ns).  Returns
    ``(out_increment [T, S] int64, out_leader [T, S] int32)``, allocated
    here when not given.  Asynchronous on ``stream`` (default: the current
    torch stream of the tensor's device).
    """
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    _check(durations, "durations", torch.int64, (T, S, R))
    dev = durations.device
    if out_increment is None:
        out_increment = _new((T, S), torch.int64, dev, stream)
    if out_leader is None:
        out_leader = _new((T, S), torch.int32, dev, stream)
    _check(out_increment, "out_increment", torch.int64, (T, S), like=durations)
    _check(out_leader, "out_leader", torch.int32, (T, S), like=durations)
    rc = _lib.sf_frontier(durations.data_ptr(), T, R, S, out_increment.data_ptr(),
                          out_leader.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_frontier")
    return out_increment, out_leader


EVIDENCE_FIELDS = ("increment", "leader", "gap", "ties", "stage_max", "stage_sum")


def sf_frontier_checked(durations: torch.Tensor, out_increment: torch.Tensor | None = None,
                        out_leader: torch.Tensor | None = None, status: torch.Tensor | None = None,
                        stream=None):
    """``sf_frontier`` plus the data-contract check (``sf_frontier_checked``).

    ``status`` is a one-element int32 tensor on the device (the bits of the
    C ABI's uint32 word); a new zeroed one is made when none is given.  The
    library only ORs ``SF_ERANGE`` into it.  Returns ``(out_increment,
    out_leader, status)``.
    """
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    _check(durations, "durations", torch.int64, (T, S, R))
    dev = durations.device
    if out_increment is None:
        out_increment = _new((T, S), torch.int64, dev, stream)
    if out_leader is None:
        out_leader = _new((T, S), torch.int32, dev, stream)
    if status is None:
        status = _new((1,), torch.int32, dev, stream, zero=True)
    _check(out_increment, "out_increment", torch.int64, (T, S), like=durations)
    _check(out_leader, "out_leader", torch.int32, (T, S), like=durations)
    _check(status, "status", torch.int32, (1,), like=durations)
    rc = _lib.sf_frontier_checked(durations.data_ptr(), T, R, S, out_increment.data_ptr(),
                                  out_leader.data_ptr(), status.data_ptr(),
                                  _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_frontier_checked")
    return out_increment, out_leader, status


def sf_frontier_evidence(durations: torch.Tensor, out: dict | None = None, stream=None) -> dict:
    """The frontier pass plus localization evidence and per-stage baselines
    (``sf_frontier_evidence``).

    ``durations``: int64 GPU tensor [T, S, R].  Returns a dict of [T, S]
    tensors keyed by ``EVIDENCE_FIELDS`` (``leader`` and ``ties`` int32,
    the others int64); ``out`` may supply any of them.
    """
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    _check(durations, "durations", torch.int64, (T, S, R))
    out = dict(out or {})
    for k in EVIDENCE_FIELDS:
        dt = torch.int32 if k in ("leader", "ties") else torch.int64
        if k not in out:
            out[k] = _new((T, S), dt, durations.device, stream)
        _check(out[k], k, dt, (T, S), like=durations)
    rc = _lib.sf_frontier_evidence(durations.data_ptr(), T, R, S,
                                   *(out[k].data_ptr() for k in EVIDENCE_FIELDS),
                                   _stream_handle(stream, durations.device))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_frontier_evidence")
    return out


def sf_window_summary(increment: torch.Tensor, leader: torch.Tensor, R: int, window: int,
                      out_stage_exposed: torch.Tensor | None = None,
                      out_lead_counts: torch.Tensor | None = None,
                      out_top2: torch.Tensor | None = None, stream=None):
    """Window reduction of per-step results (``sf_window_summary``).

    Returns ``(out_stage_exposed [W, S] int64, out_lead_counts [W, S, R]
    int32, out_top2 [W, 2, 2] int32)``.
    """
    if increment.dim() != 2:
        raise ValueError("increment must be [T, S]")
    T, S = increment.shape
    _check(increment, "increment", torch.int64, (T, S))
    _check(leader, "leader", torch.int32, (T, S), like=increment)
    W = sf_num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_window_summary")
    dev = increment.device
    if out_stage_exposed is None:
        out_stage_exposed = _new((W, S), torch.int64, dev, stream)
    if out_lead_counts is None:
        out_lead_counts = _new((W, S, R), torch.int32, dev, stream)
    if out_top2 is None:
        out_top2 = _new((W, 2, 2), torch.int32, dev, stream)
    _check(out_stage_exposed, "out_stage_exposed", torch.int64, (W, S), like=increment)
    _check(out_lead_counts, "out_lead_counts", torch.int32, (W, S, R), like=increment)
    _check(out_top2, "out_top2", torch.int32, (W, 2, 2), like=increment)
    rc = _lib.sf_window_summary(increment.data_ptr(), leader.data_ptr(), T, R, S, window,
                                out_stage_exposed.data_ptr(), out_lead_counts.data_ptr(),
                                out_top2.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_window_summary")
    return out_stage_exposed, out_lead_counts, out_top2


def sf_frontier_summary(durations: torch.Tensor, window: int, out_increment: torch.Tensor | None = None,
                        out_leader: torch.Tensor | None = None,
                        out_stage_exposed: torch.Tensor | None = None,
                        out_lead_counts: torch.Tensor | None = None,
                        out_top2: torch.Tensor | None = None, stream=None):
    """``sf_frontier`` and ``sf_window_summary`` in one call
    (``sf_frontier_summary``; one kernel launch for small inputs).

    Returns ``(out_increment [T, S], out_leader [T, S], out_stage_exposed
    [W, S], out_lead_counts [W, S, R], out_top2 [W, 2, 2])``.  Written out
    argument by argument: callers of this entry point are bound by its
    per-call cost.
    """
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    _check(durations, "durations", torch.int64, (T, S, R))
    W = _num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_frontier_summary")
    if out_increment is None:
        out_increment = _new((T, S), torch.int64, durations.device, stream)
    if out_leader is None:
        out_leader = _new((T, S), torch.int32, durations.device, stream)
    if out_stage_exposed is None:
        out_stage_exposed = _new((W, S), torch.int64, durations.device, stream)
    if out_lead_counts is None:
        out_lead_counts = _new((W, S, R), torch.int32, durations.device, stream)
    if out_top2 is None:
        out_top2 = _new((W, 2, 2), torch.int32, durations.device, stream)
    _check(out_increment, "out_increment", torch.int64, (T, S), durations)
    _check(out_leader, "out_leader", torch.int32, (T, S), durations)
    _check(out_stage_exposed, "out_stage_exposed", torch.int64, (W, S), durations)
    _check(out_lead_counts, "out_lead_counts", torch.int32, (W, S, R), durations)
    _check(out_top2, "out_top2", torch.int32, (W, 2, 2), durations)
    rc = _lib.sf_frontier_summary(durations.data_ptr(), T, R, S, window, out_increment.data_ptr(),
                                  out_leader.data_ptr(), out_stage_exposed.data_ptr(),
                                  out_lead_counts.data_ptr(), out_top2.data_ptr(),
                                  _stream_handle(stream, durations.device))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_frontier_summary")
    return out_increment, out_leader, out_stage_exposed, out_lead_counts, out_top2


def sf_window_lead_exposed(increment: torch.Tensor, leader: torch.Tensor, R: int, window: int,
                           out_lead_exposed: torch.Tensor | None = None,
                           out_top2: torch.Tensor | None = None, stream=None):
    """Exposed time each rank led, per window and stage, and the top-2
    weighted by it (``sf_window_lead_exposed``).

    Returns ``(out_lead_exposed [W, S, R] int64, out_top2 [W, 2, 2] int32)``.
    """
    if increment.dim() != 2:
        raise ValueError("increment must be [T, S]")
    T, S = increment.shape
    _check(increment, "increment", torch.int64, (T, S))
    _check(leader, "leader", torch.int32, (T, S), like=increment)
    W = sf_num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_window_lead_exposed")
    dev = increment.device
    if out_lead_exposed is None:
        out_lead_exposed = _new((W, S, R), torch.int64, dev, stream)
    if out_top2 is None:
        out_top2 = _new((W, 2, 2), torch.int32, dev, stream)
    _check(out_lead_exposed, "out_lead_exposed", torch.int64, (W, S, R), like=increment)
    _check(out_top2, "out_top2", torch.int32, (W, 2, 2), like=increment)
    rc = _lib.sf_window_lead_exposed(increment.data_ptr(), leader.data_ptr(), T, R, S, window,
                                     out_lead_exposed.data_ptr(), out_top2.data_ptr(),
                                     _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_window_lead_exposed")
    return out_lead_exposed, out_top2


def sf_window_leader_switches(leader: torch.Tensor, gap: torch.Tensor, ties: torch.Tensor,
                              window: int, min_gap: int = 0,
                              out_switches: torch.Tensor | None = None,
                              out_eligible: torch.Tensor | None = None, stream=None):
    """Leader switches between confident unique leaders, per window and
    stage (``sf_window_leader_switches``); the inputs are the ``leader``,
    ``gap`` and ``ties`` outputs of ``sf_frontier_evidence``.

    Returns ``(out_switches [W, S] int32, out_eligible [W, S] int32)``.
    """
    if leader.dim() != 2:
        raise ValueError("leader must be [T, S]")
    T, S = leader.shape
    _check(leader, "leader", torch.int32, (T, S))
    _check(gap, "gap", torch.int64, (T, S), like=leader)
    _check(ties, "ties", torch.int32, (T, S), like=leader)
    W = sf_num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_window_leader_switches")
    dev = leader.device
    if out_switches is None:
        out_switches = _new((W, S), torch.int32, dev, stream)
    if out_eligible is None:
        out_eligible = _new((W, S), torch.int32, dev, stream)
    _check(out_switches, "out_switches", torch.int32, (W, S), like=leader)
    _check(out_eligible, "out_eligible", torch.int32, (W, S), like=leader)
    rc = _lib.sf_window_leader_switches(leader.data_ptr(), gap.data_ptr(), ties.data_ptr(), T, S,
                                        window, min_gap, out_switches.data_ptr(),
                                        out_eligible.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_window_leader_switches")
    return out_switches, out_eligible


def sf_ingest(stages: torch.Tensor, wall: torch.Tensor, out_durations: torch.Tensor | None = None,
              out_overlap: torch.Tensor | None = None, stream=None):
    """Gathered per-rank buffers to [T][K+1][R] with the Appendix A closure
    (``sf_ingest``).

    ``stages``: int64 GPU tensor [R, T, K]; ``wall``: int64 [R, T].  Returns
    ``(out_durations [T, K+1, R], out_overlap [T, R])``.
    """
    if stages.dim() != 3:
        raise ValueError("stages must be [R, T, K]")
    R, T, K = stages.shape
    _check(stages, "stages", torch.int64, (R, T, K))
    _check(wall, "wall", torch.int64, (R, T), like=stages)
    dev = stages.device
    if out_durations is None:
        out_durations = _new((T, K + 1, R), torch.int64, dev, stream)
    if out_overlap is None:
        out_overlap = _new((T, R), torch.int64, dev, stream)
    _check(out_durations, "out_durations", torch.int64, (T, K + 1, R), like=stages)
    _check(out_overlap, "out_overlap", torch.int64, (T, R), like=stages)
    rc = _lib.sf_ingest(stages.data_ptr(), wall.data_ptr(), T, R, K, out_durations.data_ptr(),
                        out_overlap.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_ingest")
    return out_durations, out_overlap


def sf_route(stage_exposed: torch.Tensor, tau_num: int = 4, tau_den: int = 5,
             out_order: torch.Tensor | None = None, out_size: torch.Tensor | None = None,
             stream=None):
    """Routing candidate set per window (``sf_route``); tau = num / den
    (default 4/5 = 0.80).  Returns ``(out_order [W, S], out_size [W])``."""
    if stage_exposed.dim() != 2:
        raise ValueError("stage_exposed must be [W, S]")
    W, S = stage_exposed.shape
    _check(stage_exposed, "stage_exposed", torch.int64, (W, S))
    dev = stage_exposed.device
    if out_order is None:
        out_order = _new((W, S), torch.int32, dev, stream)
    if out_size is None:
        out_size = _new((W,), torch.int32, dev, stream)
    _check(out_order, "out_order", torch.int32, (W, S), like=stage_exposed)
    _check(out_size, "out_size", torch.int32, (W,), like=stage_exposed)
    rc = _lib.sf_route(stage_exposed.data_ptr(), W, S, tau_num, tau_den, out_order.data_ptr(),
                       out_size.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_route")
    return out_order, out_size


GAIN_FIELDS = ("gain", "makespan", "window_gain", "window_makespan")


def sf_exposure_gain(durations: torch.Tensor, baseline: torch.Tensor, window: int,
                     out: dict | None = None, stream=None) -> dict:
    """Direct-exposure gain of Eq. (4) (``sf_exposure_gain``).

    ``durations``: int64 GPU tensor [T, S, R]; ``baseline``: int64 [W, S, R]
    (btilde per window).  Returns a dict keyed by ``GAIN_FIELDS``: ``gain``
    [T, S], ``makespan`` [T], ``window_gain`` [W, S], ``window_makespan`` [W].
    G_s of window w is window_gain[w, s] / window_makespan[w].
    """
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    W = sf_num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_exposure_gain")
    _check(durations, "durations", torch.int64, (T, S, R))
    _check(baseline, "baseline", torch.int64, (W, S, R), like=durations)
    shapes = {"gain": (T, S), "makespan": (T,), "window_gain": (W, S), "window_makespan": (W,)}
    out = dict(out or {})
    for k, shp in shapes.items():
        if k not in out:
            out[k] = _new(shp, torch.int64, durations.device, stream)
        _check(out[k], k, torch.int64, shp, like=durations)
    rc = _lib.sf_exposure_gain(durations.data_ptr(), baseline.data_ptr(), T, R, S, window,
                               *(out[k].data_ptr() for k in GAIN_FIELDS),
                               _stream_handle(stream, durations.device))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_exposure_gain")
    return out


def sf_frontier_lag(durations: torch.Tensor, out_lag: torch.Tensor | None = None,
                    out_lag_inc: torch.Tensor | None = None, stream=None):
    """Lag of the frontier over the (lower) median rank and its increment
    (``sf_frontier_lag``).  Returns ``(out_lag [T, S], out_lag_inc [T, S])``."""
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    _check(durations, "durations", torch.int64, (T, S, R))
    dev = durations.device
    if out_lag is None:
        out_lag = _new((T, S), torch.int64, dev, stream)
    if out_lag_inc is None:
        out_lag_inc = _new((T, S), torch.int64, dev, stream)
    _check(out_lag, "out_lag", torch.int64, (T, S), like=durations)
    _check(out_lag_inc, "out_lag_inc", torch.int64, (T, S), like=durations)
    rc = _lib.sf_frontier_lag(durations.data_ptr(), T, R, S, out_lag.data_ptr(),
                              out_lag_inc.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_frontier_lag")
    return out_lag, out_lag_inc


def sf_rank_spread(durations: torch.Tensor, window: int, out_spread: torch.Tensor | None = None,
                   out_window_spread: torch.Tensor | None = None, stream=None):
    """Raw rank spread, max_r d - (lower) median_r d, and its window sums
    (``sf_rank_spread``).  Returns ``(out_spread [T, S], out_window_spread
    [W, S])``."""
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    W = sf_num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_rank_spread")
    _check(durations, "durations", torch.int64, (T, S, R))
    dev = durations.device
    if out_spread is None:
        out_spread = _new((T, S), torch.int64, dev, stream)
    if out_window_spread is None:
        out_window_spread = _new((W, S), torch.int64, dev, stream)
    _check(out_spread, "out_spread", torch.int64, (T, S), like=durations)
    _check(out_window_spread, "out_window_spread", torch.int64, (W, S), like=durations)
    rc = _lib.sf_rank_spread(durations.data_ptr(), T, R, S, window, out_spread.data_ptr(),
                             out_window_spread.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_rank_spread")
    return out_spread, out_window_spread


def sf_window_median(durations: torch.Tensor, window: int, out_median: torch.Tensor | None = None,
                     stream=None) -> torch.Tensor:
    """Per-rank window median (``sf_window_median``), the baseline argument
    of ``sf_exposure_gain``.  Returns ``out_median [W, S, R]``."""
    if durations.dim() != 3:
        raise ValueError("durations must be [T, S, R]")
    T, S, R = durations.shape
    W = sf_num_windows(T, window)
    if W < 0:
        raise StageFrontierError(SF_EINVAL, "sf_window_median")
    _check(durations, "durations", torch.int64, (T, S, R))
    dev = durations.device
    if out_median is None:
        out_median = _new((W, S, R), torch.int64, dev, stream)
    _check(out_median, "out_median", torch.int64, (W, S, R), like=durations)
    rc = _lib.sf_window_median(durations.data_ptr(), T, R, S, window, out_median.data_ptr(),
                               _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_window_median")
    return out_median


def sf_read_xor_pieces(nbytes: int) -> int:
    """Words ``sf_read_xor`` writes for a buffer of ``nbytes`` bytes."""
    return int(_lib.sf_read_xor_pieces(nbytes))


def sf_read_xor(buf: torch.Tensor, out_xor: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Plain-read calibration (``sf_read_xor``): the XOR of the 64-bit words
    of every ``SF_XOR_PIECE_BYTES`` piece of a contiguous GPU tensor whose
    size in bytes is a multiple of 8.

    ``out_xor`` is an int64 tensor of ``sf_read_xor_pieces(nbytes)``
    elements on the same device (the bits of the C ABI's uint64 words); a
    new one is made when none is given.  Returns ``out_xor``.
    """
    if not isinstance(buf, torch.Tensor):
        raise TypeError("buf must be a torch.Tensor")
    if buf.device.type != "cuda":
        raise ValueError("buf must be a GPU tensor")
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    dev = buf.device
    nbytes = buf.numel() * buf.element_size()
    if nbytes % 8:
        raise StageFrontierError(SF_EINVAL, "sf_read_xor")
    pieces = sf_read_xor_pieces(nbytes)
    if out_xor is None:
        out_xor = _new((pieces,), torch.int64, dev, stream)
    _check(out_xor, "out_xor", torch.int64, (pieces,), like=buf)
    if nbytes == 0:
        return out_xor
    rc = _lib.sf_read_xor(buf.data_ptr(), nbytes, out_xor.data_ptr(), _stream_handle(stream, dev))
    if rc != SF_OK:
        raise StageFrontierError(rc, "sf_read_xor")
    return out_xor


def raw_library() -> ctypes.CDLL:
    """The loaded ctypes library, for callers that pass raw device pointers."""
    return _lib
