"""Tensor Fusion (oracle): which tensors share a fusion buffer, and the copies.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper, section 7, the numbered list, in other words: (1) among the tensors ready
for reduction, choose a leading group that shares a data type and whose total size
fits the buffer; (2) create the fusion buffer the first time it is needed (64 MB
unless configured otherwise); (3) copy the chosen tensors into it; (4) allreduce it;
(5) copy the reduced values back to the output tensors; (6) continue until no tensor
is left.

Readings where the paper is silent:

* R5 which ready tensors join a buffer: a contiguous run of the ready list, in order, never
  skipping ahead; a tensor fits if the buffer's used bytes including its padding
  and the tensor stay within the threshold (equality fits).
* R6 the default size of 64 MB is 64 MiB = 67,108,864 bytes, counted in the buffer's data type
  (binary16 bytes when the gradients are compressed to fp16).
* R7 a tensor larger than the whole buffer cannot be copied in; it is reduced on
  its own ("direct"), as a one-tensor buffer with offset 0 and no padding.
* R8 layout: each tensor starts at a byte offset that is a multiple of `align`
  (16 bytes by default).  Gaps are zero padding; they are reduced like data and
  never copied out.  A buffer's length is the end of its last tensor.
* R9 readiness: every tensor is ready, in the given (backpropagation) order.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = ["Bucket", "fuse_plan", "pack", "unpack", "buffer_origin", "cast"]


@dataclass
class Bucket:
    tensors: list = field(default_factory=list)  # indices into the ready list
    offsets: list = field(default_factory=list)  # element offset of each tensor
    count: int = 0  # buffer length in elements
    direct: bool = False  # one oversize tensor reduced without a copy


def fuse_plan(numel, esize: int, threshold: int = 64 << 20, align: int = 16):
    """Group the ready tensors into fusion buffers (section 7, steps 1, 2 and 6)."""
    if align <= 0 or align & (align - 1) or align % esize:
        raise ValueError("align must be a power of two and a multiple of the element size")
    if threshold < 0:
        raise ValueError("threshold must be non-negative")
    plan = []
    cur = None
    for t, n in enumerate(numel):
        nbytes = n * esize
        if nbytes > threshold:  # R7: larger than the whole buffer
            if cur is not None:
                plan.append(cur)
                cur = None
            plan.append(Bucket([t], [0], n, True))
            continue
        if cur is None:
            cur = Bucket()
        start_bytes = -(-cur.count * esize // align) * align  # next aligned offset
        if cur.tensors and start_bytes + nbytes > threshold:  # R5: does not fit
            plan.append(cur)
            cur = Bucket()
            start_bytes = 0
        start = start_bytes // esize
        cur.tensors.append(t)
        cur.offsets.append(start)
        cur.count = start + n
    if cur is not None:
        plan.append(cur)
    return plan


def cast(x, dtype):
    """Copy into the buffer type: identity, or binary32 -> binary16 rounded to nearest
    even with gradual underflow and overflow to infinity; binary16 -> binary32 is exact."""
    with np.errstate(over="ignore"):  # overflow to infinity is the defined result
        return np.asarray(x).astype(dtype)


def pack(tensors, bucket: Bucket, dtype):
    """Section 7 step 3: one rank's tensors copied into a zeroed fusion buffer."""
    buf = np.zeros(bucket.count, dtype=dtype)
    for x, off in zip(tensors, bucket.offsets):
        x = np.asarray(x).reshape(-1)
        buf[off : off + x.size] = cast(x, dtype)
    return buf


def unpack(buf, bucket: Bucket, numel, dtype):
    """Section 7 step 5: one rank's output tensors copied out of its buffer."""
    return [cast(buf[off : off + numel[t]], dtype) for t, off in zip(bucket.tensors, bucket.offsets)]


def buffer_origin(bucket: Bucket, numel, elems):
    """For buffer positions `elems`: (tensor index or -1 for padding, index inside it)."""
    elems = np.asarray(elems, dtype=np.int64)
    tensor = np.full(elems.shape, -1, dtype=np.int64)
    local = np.zeros(elems.shape, dtype=np.int64)
    for t, off in zip(bucket.tensors, bucket.offsets):
        inside = (elems >= off) & (elems < off + numel[t])
        tensor[inside] = t
        local[inside] = elems[inside] - off
    return tensor, local
