"""Broadcast from one rank to all (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper section 4 (the fourth change: a broadcast operation that makes every
worker start from the same model) and section 5 (the fourth API change:
variables are broadcast from the first process to all others).  The result is
fixed by that definition: every rank ends holding the root's bytes.

How the bytes travel is a reading (B1): a pipelined chain along the ring.  The
buffer is cut into N chunks of whole 16-byte units (the last unit may be short),
the first (units mod N) chunks one unit longer; rank root+k forwards chunk j to
rank root+k+1 in step j+k, for k = 0..N-2, so chunk j leaves the root in step j
and reaches the last rank in step j+N-2: 2N-2 steps in all.

Many tensors in one call (reading B2): the call's tensors are laid end to end in a
virtual byte space, each starting at the next multiple of 16 bytes after the
previous one's end (the gaps belong to no tensor), and the chain above runs over
that space as over one buffer.  Every rank still ends with the root's bytes of
every tensor; only how the bytes are grouped into messages differs from one chain
per tensor.
"""
from __future__ import annotations

import numpy as np

__all__ = ["UNIT", "chunk_bytes", "chain_broadcast", "new_traffic", "tensor_layout", "chain_broadcast_tensors"]

UNIT = 16  # bytes


def chunk_bytes(nbytes: int, nranks: int):
    """[start, end) byte range of each of the N chunks."""
    units = -(-nbytes // UNIT)
    q, rem = divmod(units, nranks)
    out, u = [], 0
    for j in range(nranks):
        n = q + (1 if j < rem else 0)
        out.append((min(u * UNIT, nbytes), min((u + n) * UNIT, nbytes)))
        u += n
    return out


def new_traffic(nranks: int):
    return {"sent": np.zeros(nranks, dtype=np.int64), "recvd": np.zeros(nranks, dtype=np.int64)}


def chain_broadcast(bufs, root: int, traffic=None, observe=None):
    """Run the chain in place on `bufs` (N, nbytes) uint8 and return it.

    observe(step, bufs) is called after every step.
    """
    n, nbytes = bufs.shape
    if not 0 <= root < n:
        raise ValueError("root out of range")
    chunks = chunk_bytes(nbytes, n)
    for step in range(2 * n - 2):
        for k in range(n - 1):  # link from rank root+k to root+k+1
            j = step - k
            if 0 <= j < n:
                src, dst = (root + k) % n, (root + k + 1) % n
                lo, hi = chunks[j]
                bufs[dst, lo:hi] = bufs[src, lo:hi]
                if traffic is not None:
                    traffic["sent"][src] += hi - lo
                    traffic["recvd"][dst] += hi - lo
        if observe is not None:
            observe(step, bufs)
    return bufs


def tensor_layout(nbytes):
    """(start of each tensor in the virtual byte space, length of the space): each
    tensor starts at the first multiple of UNIT at or after the previous one's end."""
    starts, end = [], 0
    for b in nbytes:
        start = -(-end // UNIT) * UNIT
        starts.append(start)
        end = start + int(b)
    return starts, end


def chain_broadcast_tensors(per_rank, root: int, observe=None):
    """The chain over a list of tensors (reading B2), in place.

    per_rank[r][t]: rank r's tensor t as a 1-D uint8 array (its bytes); all ranks hold
    the same sizes.  observe(step, per_rank) is called after every step.
    """
    n = len(per_rank)
    sizes = [a.size for a in per_rank[0]] if n else []
    starts, total = tensor_layout(sizes)
    space = np.zeros((n, total), dtype=np.uint8)
    for r in range(n):
        for a, s in zip(per_rank[r], starts):
            space[r, s : s + a.size] = a

    def back(step, bufs):
        for r in range(n):
            for a, s in zip(per_rank[r], starts):
                a[:] = bufs[r, s : s + a.size]
        if observe is not None:
            observe(step, per_rank)

    chain_broadcast(space, root, observe=back)
    return per_rank
