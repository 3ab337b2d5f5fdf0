"""ctypes binding of the schedule model in include/vpp_sched.h (argument marshalling only).

The model runs in the native library libvpp_sched.so (host C++, built in-tree by
build.build_sched); this module raises if it is missing. ``simulate`` takes the
per-chunk stage times of one or more requests and returns the timeline summary;
``SCHEMES`` names the four schedules of sections 2.4 and 5.1-5.3 of the paper.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvpp_sched.so")

LAYOUT_CPP, LAYOUT_VPP = 0, 1
COMM_SYNC, COMM_ASYNC = 0, 1

# name -> (layout, comm, entry_first, packing)
SCHEMES = {
    "cpp": (LAYOUT_CPP, COMM_SYNC, 0, 0),
    "vpp": (LAYOUT_VPP, COMM_SYNC, 0, 0),
    "vpp_async": (LAYOUT_VPP, COMM_ASYNC, 1, 0),
    "vpp_async_packed": (LAYOUT_VPP, COMM_ASYNC, 1, 1),
}

EXPORTED = ["vpp_sched_event_count", "vpp_sched_simulate"]


class Problem(ctypes.Structure):
    _fields_ = [
        ("layout", ctypes.c_int32),
        ("comm", ctypes.c_int32),
        ("entry_first", ctypes.c_int32),
        ("packing", ctypes.c_int32),
        ("num_requests", ctypes.c_int32),
        ("num_chunks", ctypes.c_void_p),
        ("stage_time", ctypes.c_void_p),
        ("comm_time", ctypes.c_double),
    ]


class Summary(ctypes.Structure):
    _fields_ = [
        ("makespan", ctypes.c_double),
        ("compute", ctypes.c_double * 2),
        ("exposed_comm", ctypes.c_double * 2),
        ("idle", ctypes.c_double * 2),
        ("bubble_ratio", ctypes.c_double),
    ]


class Event(ctypes.Structure):
    _fields_ = [
        ("request", ctypes.c_int32),
        ("chunk", ctypes.c_int32),
        ("stage", ctypes.c_int32),
        ("rank", ctypes.c_int32),
        ("start", ctypes.c_double),
        ("end", ctypes.c_double),
    ]


_lib = None


def load():
    """Load the in-tree schedule library (raises OSError if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OSError("%s is missing: run __graft_entry__.build()" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        lib.vpp_sched_event_count.restype = ctypes.c_int
        lib.vpp_sched_event_count.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(ctypes.c_int64)]
        lib.vpp_sched_simulate.restype = ctypes.c_int
        lib.vpp_sched_simulate.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Summary),
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        _lib = lib
    return _lib


class SchedError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed with status %d" % (where, status))


def _problem(stage_times: Sequence[Sequence[float]], comm_time: float, layout: int, comm: int,
             entry_first: int, packing: int):
    counts = np.ascontiguousarray([len(r) for r in stage_times], dtype=np.int32)
    flat = np.ascontiguousarray(np.concatenate([np.asarray(r, dtype=np.float64).ravel()
                                                for r in stage_times]) if len(stage_times) else
                                np.zeros(0, np.float64))
    p = Problem(layout, comm, entry_first, packing, len(stage_times),
                counts.ctypes.data, flat.ctypes.data, float(comm_time))
    return p, (counts, flat)


def vpp_sched_event_count(stage_times: Sequence[Sequence[float]], *, scheme: Optional[str] = None,
                          layout: int = LAYOUT_VPP, comm: int = COMM_SYNC, entry_first: int = 0,
                          packing: int = 0) -> int:
    """Number of timeline intervals the model writes for these requests and switches."""
    if scheme is not None:
        layout, comm, entry_first, packing = SCHEMES[scheme]
    lib = load()
    p, keep = _problem(stage_times, 0.0, layout, comm, entry_first, packing)
    n = ctypes.c_int64(0)
    st = lib.vpp_sched_event_count(ctypes.byref(p), ctypes.byref(n))
    del keep
    if st != 0:
        raise SchedError(st, "vpp_sched_event_count")
    return int(n.value)


def vpp_sched_simulate(stage_times: Sequence[Sequence[float]], comm_time: float = 0.0, *,
                       scheme: Optional[str] = None, layout: int = LAYOUT_VPP, comm: int = COMM_SYNC,
                       entry_first: int = 0, packing: int = 0, events: bool = False) -> Dict:
    """Run the model. ``stage_times[r][k]`` is the time of one virtual stage (a quarter of
    the layers) of chunk k of request r; ``scheme`` (a key of SCHEMES) overrides the four
    switches. Returns a dict with makespan, compute, exposed_comm, idle, bubble_ratio,
    request_end and, if asked, the list of timeline intervals."""
    if scheme is not None:
        layout, comm, entry_first, packing = SCHEMES[scheme]
    lib = load()
    p, keep = _problem(stage_times, comm_time, layout, comm, entry_first, packing)
    s = Summary()
    nreq = max(len(stage_times), 1)
    req_end = np.zeros(nreq, dtype=np.float64)
    ev_buf = None
    cap = 0
    if events:
        cap = vpp_sched_event_count(stage_times, layout=layout, comm=comm,
                                    entry_first=entry_first, packing=packing)
        ev_buf = (Event * max(cap, 1))()
    st = lib.vpp_sched_simulate(ctypes.byref(p), ctypes.byref(s), req_end.ctypes.data,
                                ctypes.addressof(ev_buf) if ev_buf is not None else None, cap)
    del keep
    if st != 0:
        raise SchedError(st, "vpp_sched_simulate")
    out = {"makespan": s.makespan, "compute": list(s.compute), "exposed_comm": list(s.exposed_comm),
           "idle": list(s.idle), "bubble_ratio": s.bubble_ratio, "request_end": req_end.tolist()}
    if events:
        out["events"] = [(e.request, e.chunk, e.stage, e.rank, e.start, e.end) for e in ev_buf[:cap]]
    return out


def compare_schemes(stage_times: Sequence[Sequence[float]], comm_time: float = 0.0) -> Dict[str, Dict]:
    """All four schemes of SCHEMES on the same requests (summaries only)."""
    return {name: vpp_sched_simulate(stage_times, comm_time, scheme=name) for name in SCHEMES}


def stage_times_from_curve(chunk_ms: Sequence[float], layers_per_stage: int = 1,
                           fixed_ms: float = 0.0) -> List[float]:
    """Per-chunk virtual-stage times (ms) from a measured one-layer attention latency curve:
    layers_per_stage x (attention latency of the chunk + a fixed per-chunk per-layer cost,
    e.g. the projections and MoE that the attention kernel does not cover)."""
    return [layers_per_stage * (float(t) + fixed_ms) for t in chunk_ms]
