"""One averaging allreduce over every rank's gradient tensors (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper section 5 (the optimizer wrapper averages gradients with ring-allreduce) and
section 7 (Tensor Fusion): plan the buffers, copy each rank's tensors in, run the
ring of section 3 on the buffers, copy the results out, repeat per buffer.

Compression to fp16 (an option of this build, not of the paper): the gradients are
rounded to binary16 when copied in (a direct tensor is rounded as a whole), the
ring adds and divides in binary16, and the results are widened exactly to binary32
when copied out.  The fusion threshold then counts binary16 bytes.
"""
from __future__ import annotations

import numpy as np

from . import fusion, ring

__all__ = ["allreduce", "bucket_columns", "ring_columns"]


def allreduce(per_rank, op=ring.AVERAGE, compress=False, threshold=64 << 20, align=16, traffic=None):
    """Return every rank's reduced tensors.

    per_rank -- per_rank[r][t] is rank r's t-th gradient (ready order), binary32
                or binary16 arrays; all ranks hold the same shapes.
    traffic  -- optional dict bucket index -> counters from ``ring.new_traffic``;
                filled for every buffer.
    """
    n = len(per_rank)
    src_dtype = np.asarray(per_rank[0][0]).dtype if per_rank[0] else np.dtype(np.float32)
    buf_dtype = np.dtype(np.float16) if compress else src_dtype
    if compress and src_dtype != np.float32:
        raise ValueError("compression applies to binary32 gradients")
    numel = [np.asarray(x).size for x in per_rank[0]]
    plan = fusion.fuse_plan(numel, buf_dtype.itemsize, threshold, align)
    out = [[None] * len(numel) for _ in range(n)]
    for b, bucket in enumerate(plan):
        bufs = np.stack([fusion.pack([per_rank[r][t] for t in bucket.tensors], bucket, buf_dtype) for r in range(n)])
        counters = None
        if traffic is not None:
            counters = traffic.setdefault(b, ring.new_traffic(n))
        ring.ring_allreduce(bufs, op, count=bucket.count, traffic=counters)
        for r in range(n):
            for t, y in zip(bucket.tensors, fusion.unpack(bufs[r], bucket, numel, src_dtype)):
                out[r][t] = y.reshape(np.asarray(per_rank[r][t]).shape)
    return out


def bucket_columns(bucket, numel, elems, value_of, nranks, buf_dtype):
    """Buffer contents after packing, at positions `elems`, for every rank.

    value_of(rank, tensor, local_indices) returns that tensor's binary32 (or
    binary16) values at those indices.  Padding positions hold zero.
    """
    tensor, local = fusion.buffer_origin(bucket, numel, elems)
    cols = np.zeros((nranks, len(elems)), dtype=buf_dtype)
    for t in np.unique(tensor[tensor >= 0]):
        sel = tensor == t
        for r in range(nranks):
            cols[r, sel] = fusion.cast(value_of(r, int(t), local[sel]), buf_dtype)
    return cols


def ring_columns(bucket, numel, elems, value_of, nranks, op=ring.AVERAGE, compress=False, out_dtype=np.float32):
    """Reduced values at buffer positions `elems` (sorted) of one bucket, per rank.

    The same ring as ``allreduce`` restricted to a subset of elements, for buffers
    too large to simulate whole.  Returns (values (N, m) in out_dtype, tensor
    index per position or -1 for padding, index inside the tensor).
    """
    buf_dtype = np.dtype(np.float16) if compress else np.dtype(out_dtype)
    cols = bucket_columns(bucket, numel, elems, value_of, nranks, buf_dtype)
    ring.ring_allreduce(cols, op, count=bucket.count, elems=elems)
    tensor, local = fusion.buffer_origin(bucket, numel, elems)
    return fusion.cast(cols, out_dtype), tensor, local
