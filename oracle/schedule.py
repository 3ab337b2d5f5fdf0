"""Reference model of the pipeline schedules of sections 2.4 and 5.1-5.3 (pure Python).

TEST INFRASTRUCTURE ONLY: this is the checker of the native schedule model
(paper_2608_26523_amd/csrc/vpp_sched.cpp), not the product. Only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may use it,
and it shares no code with the native model.

What it computes, in the paper's terms (two pipeline ranks pp0, pp1):

* CPP (sections 2.4, 4): stage 0 of every chunk on pp0, stage 1 on pp1, chunks in
  order; a physical stage holds two virtual stages' worth of layers.
* VPP (section 5.1): virtual stages s0..s3 with s0, s3 on pp0 and s1, s2 on pp1;
  chunk k goes s0 -> s1 -> s2 -> s3. pp0 runs s0 of chunks 0 and 1, then in each
  period k = 1 .. N-1 the exit s3 of chunk k-1 and the entry s0 of chunk k+1
  (exit first), and finally s3 of chunk N-1. pp1 runs s1, s2 of each chunk in
  order. Handoffs are blocking: the forward handoff of chunk k+1 and the back
  handoff of chunk k are one bidirectional exchange at the end of a period.
* VPP-Async (section 5.2): the entry of chunk k+1 goes before the exit of chunk
  k-1, and handoffs are non-blocking (they arrive comm_time after the producer).
* Pipelined packing (section 5.3): when the current request's next operation
  is not ready, a free rank runs the next request's first ready operation.

An operation needs its chunk's previous stage (plus the handoff time when that
ran on the other rank, non-blocking mode) and the previous chunk's same stage
(its KV cache). Time advances from event to event; at each time rank 0, then
rank 1, starts whatever is ready, until nothing more starts.

Parity pins: closed forms derived from Eq. 2 and Eq. 3 (see the tests).
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

INF = math.inf


def _rank_of_stage(layout: str, s: int) -> int:
    if layout == "cpp":
        return s
    return 1 if s in (1, 2) else 0


def simulate(stage_times: Sequence[Sequence[float]], comm_time: float = 0.0, *,
             layout: str = "vpp", blocking: bool = True, entry_first: bool = False,
             packing: bool = False) -> Dict:
    """Return {"makespan", "compute", "exposed_comm", "idle", "bubble_ratio",
    "request_end", "ops"}; ops maps (request, chunk, stage) -> (start, end)."""
    assert layout in ("cpp", "vpp")
    assert not (packing and blocking), "packing is defined with non-blocking handoffs"
    nst = 2 if layout == "cpp" else 4
    dur = {}
    for r, chunks in enumerate(stage_times):
        for k, tau in enumerate(chunks):
            for s in range(nst):
                dur[(r, k, s)] = 2 * tau if layout == "cpp" else tau
                # (2 * tau equals tau + tau exactly in binary floating point)

    # programs: per rank, per request, a list of ("op", key) / ("x", exchange id)
    progs = [[[] for _ in stage_times], [[] for _ in stage_times]]
    exchanges = {}  # id -> {"req": r, "arrived": set(), "start": None}

    def new_x(r):
        i = len(exchanges)
        exchanges[i] = {"req": r, "arrived": set(), "start": None}
        return i

    for r, chunks in enumerate(stage_times):
        n = len(chunks)
        if layout == "cpp":
            for k in range(n):
                progs[0][r].append(("op", (r, k, 0)))
                if blocking:
                    x = new_x(r)
                    progs[0][r].append(("x", x))
                    progs[1][r].append(("x", x))
                progs[1][r].append(("op", (r, k, 1)))
            continue
        xs = [new_x(r) for _ in range(n + 1)] if blocking else None
        # pp1
        if blocking:
            progs[1][r].append(("x", xs[0]))
        for k in range(n):
            progs[1][r].append(("op", (r, k, 1)))
            progs[1][r].append(("op", (r, k, 2)))
            if blocking:
                progs[1][r].append(("x", xs[k + 1]))
        # pp0
        p0 = progs[0][r]
        p0.append(("op", (r, 0, 0)))
        if blocking:
            p0.append(("x", xs[0]))
        if n >= 2:
            p0.append(("op", (r, 1, 0)))
            if blocking:
                p0.append(("x", xs[1]))
        for k in range(1, n):
            pair = [("op", (r, k - 1, 3))]
            if k + 1 < n:
                pair.append(("op", (r, k + 1, 0)))
                if entry_first:
                    pair.reverse()
            p0.extend(pair)
            if blocking:
                p0.append(("x", xs[k + 1]))
        if n == 1 and blocking:
            p0.append(("x", xs[1]))
        p0.append(("op", (r, n - 1, 3)))

    start, end = {}, {}

    def ready_time(key) -> float:
        r, k, s = key
        t = 0.0
        if k > 0:
            prev = (r, k - 1, s)
            if prev not in end:
                return INF
            t = max(t, end[prev])
        if s > 0:
            prev = (r, k, s - 1)
            if prev not in end:
                return INF
            hop = _rank_of_stage(layout, s - 1) != _rank_of_stage(layout, s)
            t = max(t, end[prev] + comm_time if (hop and not blocking) else end[prev])
        return t

    pos = [[0] * len(stage_times), [0] * len(stage_times)]
    free = [0.0, 0.0]
    compute = [0.0, 0.0]
    exposed = [0.0, 0.0]
    left = sum(len(p) for rp in progs for p in rp)

    def open_requests(rank):
        return [r for r in range(len(stage_times)) if pos[rank][r] < len(progs[rank][r])]

    def step(rank, now) -> bool:
        """Start one item on `rank` at `now` if possible."""
        nonlocal left
        if free[rank] > now:
            return False
        reqs = open_requests(rank)
        if not packing:
            reqs = reqs[:1]
        for r in reqs:
            kind, what = progs[rank][r][pos[rank][r]]
            if kind == "x":
                ex = exchanges[what]
                ex["arrived"].add(rank)
                if len(ex["arrived"]) < 2:
                    continue
                ex["start"] = now
                for q in (0, 1):
                    free[q] = now + comm_time
                    exposed[q] += comm_time
                    pos[q][r] += 1
                    left -= 1
                return True
            t = ready_time(what)
            if t > now:
                continue
            rr, k, s = what
            if s > 0 and not blocking and _rank_of_stage(layout, s - 1) != rank:
                waited_for = max([free[rank], end[(rr, k, s - 1)]] +
                                 ([end[(rr, k - 1, s)]] if k > 0 else []))
                if now > waited_for:
                    exposed[rank] += now - waited_for
            start[what] = now
            end[what] = now + dur[what]
            free[rank] = end[what]
            compute[rank] += dur[what]
            pos[rank][r] += 1
            left -= 1
            return True
        return False

    now = 0.0
    while left > 0:
        progress = True
        while progress:
            progress = False
            for rank in (0, 1):
                while step(rank, now):
                    progress = True
        if left == 0:
            break
        later = [f for f in free if f > now]
        for rank in (0, 1):
            for r in open_requests(rank):
                kind, what = progs[rank][r][pos[rank][r]]
                if kind == "op":
                    t = ready_time(what)
                    if now < t < INF:
                        later.append(t)
        if not later:
            raise RuntimeError("the schedule cannot make progress")
        now = min(later)

    makespan = max([0.0] + list(end.values()) +
                   [ex["start"] + comm_time for ex in exchanges.values()])
    idle = [makespan - compute[q] - exposed[q] for q in (0, 1)]
    req_end = [0.0] * len(stage_times)
    for (r, _, _), e in end.items():
        req_end[r] = max(req_end[r], e)
    for ex in exchanges.values():
        req_end[ex["req"]] = max(req_end[ex["req"]], ex["start"] + comm_time)
    return {"makespan": makespan, "compute": compute, "exposed_comm": exposed, "idle": idle,
            "bubble_ratio": (idle[0] + idle[1]) / (2 * makespan) if makespan > 0 else 0.0,
            "request_end": req_end, "ops": {key: (start[key], end[key]) for key in start}}


SCHEMES = {
    "cpp": dict(layout="cpp", blocking=True, entry_first=False, packing=False),
    "vpp": dict(layout="vpp", blocking=True, entry_first=False, packing=False),
    "vpp_async": dict(layout="vpp", blocking=False, entry_first=True, packing=False),
    "vpp_async_packed": dict(layout="vpp", blocking=False, entry_first=True, packing=True),
}


def simulate_scheme(name: str, stage_times, comm_time: float = 0.0) -> Dict:
    return simulate(stage_times, comm_time, **SCHEMES[name])


def linear_taus(n: int, t: float = 1.0) -> List[float]:
    """Eq. 2: the stage latency of chunk k is (k+1) t."""
    return [(k + 1) * t for k in range(n)]


def busy_intervals(res: Dict, rank: int, layout: str = "vpp") -> List[Tuple[float, float]]:
    """Compute intervals of one rank, in time order (helper for bubble checks)."""
    iv = [(s, e) for (r, k, st), (s, e) in res["ops"].items() if _rank_of_stage(layout, st) == rank]
    return sorted(iv)
