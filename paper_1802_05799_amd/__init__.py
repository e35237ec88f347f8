"""hvdx: Horovod's data-parallel hot path (Tensor Fusion + ring-allreduce) on MI355X.

Python binding of libhvdx.so.  torch is imported first so that the library binds
to the HIP runtime torch already loaded (one runtime per process).

    from paper_1802_05799_amd import FusedAllreduce
    ar = FusedAllreduce(per_rank_grads, op="average")   # plan + buffers, once
    ar()                                                  # reduce in place
"""
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
    SMALL_BUCKET_BYTES,
    SUM,
    HvdxError,
    hvdx_broadcast,
    hvdx_broadcast_step,
    hvdx_fold_allreduce,
    hvdx_fuse_ag_unpack,
    hvdx_fuse_allreduce,
    hvdx_fuse_allreduce_pair,
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


def broadcast_(per_rank, root: int = 0) -> None:
    """Copy rank `root`'s tensors into every other rank's, tensor by tensor (paper
    sections 4 and 5: consistent initial variables).  Tensors must be contiguous GPU
    tensors of matching shapes and dtypes across ranks."""
    n = len(per_rank)
    for ts in zip(*per_rank):
        ref = ts[0]
        for x in ts:
            if x.shape != ref.shape or x.dtype != ref.dtype or not x.is_contiguous() or x.device.type != "cuda":
                raise ValueError("broadcast needs contiguous GPU tensors matching across ranks")
        stream = torch.cuda.current_stream(ref.device).cuda_stream
        hvdx_broadcast([x.data_ptr() for x in ts], n, ref.numel() * ref.element_size(), root, stream)


def allreduce_(per_rank, op: str = "average", compress: bool = False,
               threshold_bytes: int = DEFAULT_FUSION_THRESHOLD, align_bytes: int = DEFAULT_FUSION_ALIGN) -> None:
    """One in-place allreduce of every rank's tensor list (builds a one-off plan)."""
    FusedAllreduce(per_rank, op, compress, threshold_bytes, align_bytes)()
