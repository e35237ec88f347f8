"""Timeline of the allreduce's kernel launches (paper section 6, Horovod Timeline).

The paper's timeline shows what every node did at each time step in Chrome's
about:tracing viewer and is switched on by one environment variable.  Here the
library brackets each kernel it launches with HIP events while a timeline
records (hvdx_timeline_begin / hvdx_timeline_end); this module turns the records
into Chrome trace JSON with one track per simulated rank, naming for every ring
step the chunk the rank sends to its right neighbour and the chunk it receives
from its left one, plus one track for the GPU kernels themselves.

    with Timeline() as tl:
        allreduce()
    tl.save("trace.json")

or set HVDX_TIMELINE=trace.json before the first FusedAllreduce is built: every
allreduce of the process is then recorded and the trace written at exit.
"""
from __future__ import annotations

import atexit
import json
import os

from . import _lib as L

KIND_NAMES = {
    L.KERNEL_PACK: "copy in",
    L.KERNEL_REDUCE_SCATTER: "reduce-scatter",
    L.KERNEL_ALLGATHER: "allgather",
    L.KERNEL_UNPACK: "copy out",
    L.KERNEL_ROUNDTRIP: "fp16 round trip",
    L.KERNEL_BROADCAST: "broadcast",
    L.KERNEL_RS_AG: "reduce-scatter + allgather",
    L.KERNEL_FOLD: "fold",
    L.KERNEL_PACK_RS: "copy in + reduce-scatter",
    L.KERNEL_AG_UNPACK: "allgather + copy out",
    L.KERNEL_RING_SMALL: "whole ring (one launch)",
    L.KERNEL_CYCLE_SMALL: "copy in + whole ring + copy out (one launch)",
}


def chunks_of_step(kind: int, step: int, rank: int, n: int):
    """(chunk sent to rank+1, chunk received from rank-1) in one ring step: in adding
    step s rank r sends chunk (r - s) mod N, in replacing step s chunk (r + 1 - s) mod N."""
    if kind == L.KERNEL_REDUCE_SCATTER:
        return (rank - step) % n, (rank - 1 - step) % n
    return (rank + 1 - step) % n, (rank - step) % n


def broadcast_step_args(step: int, rank: int, root: int, n: int) -> dict:
    """What `rank` does in broadcast step `step`: rank root+k forwards chunk step-k to
    its right neighbour (k = 0..N-2) and received chunk step-k+1 from its left one."""
    k = (rank - root) % n
    args = {}
    if k <= n - 2 and 0 <= step - k < n:
        args["send chunk"] = step - k
        args["to"] = (rank + 1) % n
    if k >= 1 and 0 <= step - k + 1 < n:
        args["recv chunk"] = step - k + 1
        args["from"] = (rank - 1) % n
    return args


class Timeline:
    """per_phase=False records every launch; True records each run of launches of one
    kernel inside a library call as one record (see hvdx_timeline_begin)."""

    def __init__(self, capacity: int = 1 << 16, per_phase: bool = False):
        self.capacity = capacity
        self.per_phase = per_phase
        self.records: list = []
        self.dropped = 0

    def __enter__(self):
        L.hvdx_timeline_begin(self.capacity, self.per_phase)
        return self

    def __exit__(self, *exc):
        self.records, self.dropped = L.hvdx_timeline_end(self.capacity)
        return False

    def chrome_trace(self) -> dict:
        events = [
            {"ph": "M", "pid": 0, "tid": 0, "name": "process_name", "args": {"name": "hvdx (one MI355X)"}},
            {"ph": "M", "pid": 0, "tid": 0, "name": "thread_name", "args": {"name": "GPU kernels"}},
        ]
        named = set()
        for rec in self.records:
            kind, n, step = rec["kind"], rec["nranks"], rec["step"]
            name = KIND_NAMES.get(kind, str(kind)) + (f" {step}" if step >= 0 else "")
            if rec["launches"] > 1:
                name += f"-{step + rec['launches'] - 1}"
            common = {"ph": "X", "pid": 0, "ts": rec["start_us"], "dur": rec["duration_us"], "cat": "hvdx"}
            events.append(dict(common, tid=0, name=name, args={"elements_per_rank": rec["count"], "ranks": n}))
            for r in range(n):
                if r not in named:
                    named.add(r)
                    events.append({"ph": "M", "pid": 0, "tid": r + 1, "name": "thread_name",
                                   "args": {"name": f"rank {r}"}})
                args = {}
                if kind == L.KERNEL_BROADCAST:
                    args = broadcast_step_args(step, r, rec["root"], n)
                if kind in (L.KERNEL_RING_SMALL, L.KERNEL_CYCLE_SMALL):
                    args = {"steps": f"adding 0-{n - 2}, replacing 0-{n - 2}", "to": (r + 1) % n,
                            "from": (r - 1) % n}
                if kind == L.KERNEL_RS_AG:  # adding step N-2, then replacing step 0
                    args = {"send chunks": [(r + 2) % n, (r + 1) % n], "to": (r + 1) % n,
                            "recv chunks": [(r + 1) % n, r], "from": (r - 1) % n,
                            "incoming chunk": "summed in, then overwrites"}
                ring_kind = {L.KERNEL_PACK_RS: L.KERNEL_REDUCE_SCATTER, L.KERNEL_AG_UNPACK: L.KERNEL_ALLGATHER}.get(
                    kind, kind)
                if ring_kind in (L.KERNEL_REDUCE_SCATTER, L.KERNEL_ALLGATHER) and rec["launches"] == 1:
                    sent, recv = chunks_of_step(ring_kind, step, r, n)
                    args = {"send chunk": sent, "to": (r + 1) % n, "recv chunk": recv, "from": (r - 1) % n,
                            "incoming chunk": "summed in" if ring_kind == L.KERNEL_REDUCE_SCATTER else "overwrites"}
                events.append(dict(common, tid=r + 1, name=name, args=args))
        return {"traceEvents": events, "displayTimeUnit": "ms",
                "otherData": {"dropped_launches": self.dropped}}

    def save(self, path: str) -> None:
        with open(path, "w") as f:
            json.dump(self.chrome_trace(), f)


_env_timeline: Timeline | None = None


def start_from_env() -> None:
    """Record every launch of this process into $HVDX_TIMELINE (written at exit)."""
    global _env_timeline
    path = os.environ.get("HVDX_TIMELINE")
    if not path or _env_timeline is not None:
        return
    tl = Timeline(int(os.environ.get("HVDX_TIMELINE_CAPACITY", 1 << 20)))
    tl.__enter__()
    _env_timeline = tl

    def finish():
        tl.__exit__(None, None, None)
        tl.save(path)

    atexit.register(finish)
