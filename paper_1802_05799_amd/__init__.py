"""hvdx: Horovod's data-parallel hot path (Tensor Fusion + ring-allreduce) on MI355X.

Python binding of libhvdx.so.  torch is imported first so that the library binds
to the HIP runtime torch already loaded (one runtime per process).

    from paper_1802_05799_amd import FusedAllreduce
    ar = FusedAllreduce(per_rank_grads, op="average")   # plan + buffers, once
    ar()                                                  # reduce in place
"""
import operator

import torch  # noqa: F401  (must precede the library load)

from ._lib import (  # noqa: F401
    AVERAGE,
    COMPRESS_FP16,
    COMPRESS_NONE,
    DEFAULT_FUSION_ALIGN,
    DEFAULT_FUSION_THRESHOLD,
    ERR_ALIAS,
    ERR_HIP,
    ERR_INVALID,
    ERR_UNSUPPORTED,
    ERR_WORKSPACE,
    FLOAT16,
    FLOAT32,
    LIB_PATH,
    MAX_RANKS,
    OK,
    PHASE_ALLGATHER,
    PHASE_REDUCE_SCATTER,
    TILED_ADD_FROM_TENSORS,
    TILED_BUFFERS,
    TILED_MAX_BUCKETS,
    TILED_MAX_BUFFERS,
    TILED_REPLACE_IN_TENSORS,
    SMALL_BUCKET_BYTES,
    SUM,
    HvdxError,
    hvdx_broadcast,
    hvdx_broadcast_step,
    hvdx_broadcast_layout,
    hvdx_broadcast_tensors,
    hvdx_broadcast_tensors_step,
    hvdx_fold_allreduce,
    hvdx_fuse_ag_unpack,
    hvdx_fuse_allreduce,
    hvdx_fuse_allreduce_pair,
    hvdx_fuse_allreduce_tiled,
    hvdx_fuse_copy_tiles,
    hvdx_fuse_tile_elems,
    COPY_IN,
    COPY_OUT,
    hvdx_fuse_allreduce_small,
    hvdx_fuse_pack,
    hvdx_fuse_pack_rs,
    hvdx_fuse_plan,
    hvdx_fuse_unpack,
    hvdx_last_error,
    hvdx_ring_allgather,
    hvdx_ring_allreduce,
    hvdx_ring_allreduce_small,
    hvdx_ring_allreduce_noalloc,
    hvdx_ring_noalloc_max_bytes,
    hvdx_ring_chunk,
    hvdx_ring_reduce_scatter,
    hvdx_ring_step,
    hvdx_ring_workspace_bytes,
    hvdx_strerror,
    hvdx_timeline_begin,
    hvdx_timeline_end,
    hvdx_version,
)
from .cycle import FusedAllreduce  # noqa: F401
from .timeline import Timeline  # noqa: F401


_NBYTES = operator.attrgetter("nbytes")


class TensorBroadcast:
    """Rank `root`'s tensors copied into every other rank's (paper sections 4 and 5:
    consistent initial variables), every tensor of the list in one chain:
    hvdx_broadcast_tensors runs the 2N-2 chain steps once for the whole list, over the
    tensors laid end to end at 16-byte aligned starts.  Bytes are copied, not
    interpreted: tensor t must have the same byte count on every rank (any dtype), be
    contiguous, on one GPU, and share memory with no other tensor.  The descriptor
    tables are uploaded once (asynchronously, from pinned memory); the tensors must stay
    allocated and in place."""

    def __init__(self, per_rank):
        import numpy as np

        if not per_rank or len(per_rank) > MAX_RANKS:
            raise ValueError(f"need 1..{MAX_RANKS} ranks")
        self.nranks = n = len(per_rank)
        self.ntensors = nt = len(per_rank[0])
        if any(len(ts) != nt for ts in per_rank):
            raise ValueError("every rank needs the same number of tensors")
        flat = [x for ts in per_rank for x in ts]
        # four passes over the tensors, each one torch call per tensor (map: no bytecode per item)
        if not all(map(torch.Tensor.is_contiguous, flat)):
            raise ValueError("broadcast needs contiguous GPU tensors")
        devices = set(map(torch.Tensor.get_device, flat))  # -1: not on a GPU
        if -1 in devices:
            raise ValueError("broadcast needs contiguous GPU tensors")
        if len(devices) > 1:
            raise ValueError("broadcast needs every tensor on one GPU")
        ptr = np.fromiter(map(torch.Tensor.data_ptr, flat), dtype=np.int64, count=len(flat))
        nbytes = np.fromiter(map(_NBYTES, flat), dtype=np.int64, count=len(flat)).reshape(n, nt)
        if (nbytes != nbytes[:1]).any():
            raise ValueError("tensor t must have the same byte count on every rank")
        live = nbytes.reshape(-1) > 0
        starts = ptr[live]
        order = np.argsort(starts, kind="stable")
        ends = starts[order] + nbytes.reshape(-1)[live][order]
        if (ends[:-1] > starts[order][1:]).any():
            raise ValueError("tensors overlap in memory")
        self.device = flat[0].device if flat else torch.device("cuda", torch.cuda.current_device())
        voff, self.total = hvdx_broadcast_layout(nbytes[0].tolist() if nt else [])
        # one upload: the rank-major pointer table, then the byte counts, then the starts
        host = torch.from_numpy(np.concatenate([ptr, nbytes[0], np.asarray(voff, dtype=np.int64), [0]]))
        self.tables = host.pin_memory().to(self.device, non_blocking=True)
        upload = torch.cuda.current_stream(self.device)
        self._ready = torch.cuda.Event()  # a call on another stream waits for the upload
        self._ready.record(upload)
        self._waited = {upload.cuda_stream}  # calls on the upload stream follow it in order
        k = n * nt
        self._args = (self.tables.data_ptr(), self.tables.data_ptr() + 8 * k, self.tables.data_ptr() + 8 * (k + nt),
                      nt, self.total, n)
        self.tensors = per_rank  # keeps the tensors alive as long as the tables point at them

    def _stream(self, stream):
        if stream is None:
            stream = torch.cuda.current_stream(self.device).cuda_stream
        if stream not in self._waited:  # once per stream: the tables' upload precedes the first launch
            torch.cuda.ExternalStream(stream, device=self.device).wait_event(self._ready)
            self._waited.add(stream)
        return stream

    def __call__(self, root: int = 0, stream: int | None = None) -> None:
        hvdx_broadcast_tensors(*self._args, root, self._stream(stream))

    def step(self, root: int, step: int, stream: int | None = None) -> None:
        """One chain step alone (hvdx_broadcast_tensors_step)."""
        hvdx_broadcast_tensors_step(*self._args, root, step, self._stream(stream))


def broadcast_(per_rank, root: int = 0) -> None:
    """Copy rank `root`'s tensors into every other rank's, all of them in one chain
    (TensorBroadcast)."""
    TensorBroadcast(per_rank)(root)


def allreduce_(per_rank, op: str = "average", compress: bool = False,
               threshold_bytes: int = DEFAULT_FUSION_THRESHOLD, align_bytes: int = DEFAULT_FUSION_ALIGN) -> None:
    """One in-place allreduce of every rank's tensor list (builds a one-off plan)."""
    FusedAllreduce(per_rank, op, compress, threshold_bytes, align_bytes)()
