"""Ring-allreduce, simulated step by step over N rank buffers (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper, section 3, the paragraph after the ring-allreduce figure: the N workers form
a ring and, over 2(N-1) rounds, each passes one chunk of its buffer to a neighbour
and takes one from the other.  During the first N-1 rounds the incoming chunk is
summed into the local copy; during the last N-1 rounds it overwrites the local copy.

The ring figure itself is lost, so these readings fill what the text leaves open:

* R1 direction and schedule.  Rank r sends to rank (r+1) mod N.  In adding step
  s (s = 0..N-2) chunk c travels from rank (c+s) mod N to rank (c+s+1) mod N; the
  sum of chunk c therefore starts at rank c, and after the last adding step rank
  (c-1) mod N holds the complete chunk.  In replacing step s chunk c travels from
  rank (c-1+s) mod N to rank (c+s) mod N.  Equivalently: in adding step s rank r
  sends chunk (r-s) mod N; in replacing step s it sends chunk (r+1-s) mod N.
* R2 partition.  ``count`` elements are cut into N contiguous chunks; with
  q, rem = divmod(count, N) chunk c starts at c*q + min(c, rem) and the first rem
  chunks hold q+1 elements, the others q.  Chunks may be empty when count < N.
* R3 summation order is the ring order: element e of chunk c ends as
  (((x_c + x_{c+1}) + x_{c+2}) + ... + x_{c+N-1}), ranks mod N.
* R4 averaging (the step of paper section 3's data-parallel recipe that averages
  the gradients, and section 5's optimizer wrapper): the complete sum is divided by N once, in the buffer's
  precision, by the rank that completes it at the last adding step; the replacing
  steps then carry the average.  N = 1 divides by 1.

All steps of one iteration happen at the same time on a real ring.  Updating the
buffers in place chunk by chunk is the same thing, because within one step no
rank reads a chunk that another rank writes in that step (the chunk a rank
receives is never the chunk it sends).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "SUM",
    "AVERAGE",
    "chunk_bounds",
    "rs_sender",
    "rs_receiver",
    "ag_sender",
    "ag_receiver",
    "add",
    "divide",
    "ring_allreduce",
    "new_traffic",
]

SUM = "sum"
AVERAGE = "average"


def chunk_bounds(count: int, nranks: int):
    """(starts, lengths) of the N chunks of a `count`-element buffer (reading R2)."""
    q, rem = divmod(count, nranks)
    starts = [c * q + min(c, rem) for c in range(nranks)]
    lengths = [q + (1 if c < rem else 0) for c in range(nranks)]
    return starts, lengths


def rs_sender(c: int, s: int, n: int) -> int:
    """Rank that sends chunk c in adding step s (reading R1)."""
    return (c + s) % n


def rs_receiver(c: int, s: int, n: int) -> int:
    """Rank that receives chunk c in adding step s (reading R1)."""
    return (c + s + 1) % n


def ag_sender(c: int, s: int, n: int) -> int:
    """Rank that sends chunk c in replacing step s (reading R1)."""
    return (c - 1 + s) % n


def ag_receiver(c: int, s: int, n: int) -> int:
    """Rank that receives chunk c in replacing step s (reading R1)."""
    return (c + s) % n


def add(local, received):
    """Elementwise sum in the buffer's precision, rounded to nearest even.

    binary32: the IEEE binary32 sum.  binary16: the exact sum rounded once to
    binary16, computed as the binary32 sum of the two widened values rounded to
    binary16 -- binary32 keeps 24 >= 2*11 + 2 significand bits, so the double
    rounding equals a single correct rounding.
    """
    if local.dtype == np.float32:
        return (local + received).astype(np.float32)
    if local.dtype == np.float16:
        with np.errstate(over="ignore"):  # overflow to infinity is the defined result
            return (local.astype(np.float32) + received.astype(np.float32)).astype(np.float16)
    raise TypeError(f"unsupported buffer dtype {local.dtype}")


def divide(x, n: int):
    """x / n correctly rounded in the buffer's precision (reading R4)."""
    if x.dtype == np.float32:
        return (x / np.float32(n)).astype(np.float32)
    if x.dtype == np.float16:
        return (x.astype(np.float32) / np.float32(n)).astype(np.float16)
    raise TypeError(f"unsupported buffer dtype {x.dtype}")


def new_traffic(nranks: int):
    """Per-rank counters of elements sent and received."""
    return {"sent": np.zeros(nranks, dtype=np.int64), "recvd": np.zeros(nranks, dtype=np.int64)}


def ring_allreduce(bufs, op: str, count: int | None = None, elems=None, traffic=None, observe=None):
    """Run the 2(N-1) ring iterations in place on `bufs` and return it.

    bufs    -- array (N, m): row r is rank r's buffer, or the columns of it listed
               in `elems`.
    count   -- length of each rank's whole buffer (defaults to m).
    elems   -- sorted element indices that the m columns hold (defaults to all of
               0..count-1).  Every element's arithmetic involves only that element,
               so a subset of columns gives the same values as the whole run.
    traffic -- optional counters from `new_traffic`; every message adds the full
               chunk length to its sender's "sent" and receiver's "recvd".
    observe -- optional callable(phase, s, bufs), phase "rs" or "ag", called after
               every iteration with the buffers as they stand.
    """
    n, m = bufs.shape
    if count is None:
        count = m
    if elems is None:
        if m != count:
            raise ValueError("bufs must hold count columns when elems is not given")
        elems = np.arange(count)
    elems = np.asarray(elems)
    if op not in (SUM, AVERAGE):
        raise ValueError(f"unknown op {op!r}")
    starts, lengths = chunk_bounds(count, n)
    cols = []
    for c in range(n):
        lo = int(np.searchsorted(elems, starts[c], side="left"))
        hi = int(np.searchsorted(elems, starts[c] + lengths[c], side="left"))
        cols.append(slice(lo, hi))

    def message(snd, rcv, c):
        if traffic is not None:
            traffic["sent"][snd] += lengths[c]
            traffic["recvd"][rcv] += lengths[c]

    # rounds 1 .. N-1: the incoming chunk is summed into the receiver's copy
    for s in range(n - 1):
        for c in range(n):
            snd, rcv = rs_sender(c, s, n), rs_receiver(c, s, n)
            v = add(bufs[rcv, cols[c]], bufs[snd, cols[c]])
            if op == AVERAGE and s == n - 2:
                v = divide(v, n)
            bufs[rcv, cols[c]] = v
            message(snd, rcv, c)
        if observe is not None:
            observe("rs", s, bufs)
    if op == AVERAGE and n == 1:
        bufs[0] = divide(bufs[0], 1)

    # rounds N .. 2N-2: the incoming chunk overwrites the receiver's copy
    for s in range(n - 1):
        for c in range(n):
            snd, rcv = ag_sender(c, s, n), ag_receiver(c, s, n)
            bufs[rcv, cols[c]] = bufs[snd, cols[c]]
            message(snd, rcv, c)
        if observe is not None:
            observe("ag", s, bufs)
    return bufs
