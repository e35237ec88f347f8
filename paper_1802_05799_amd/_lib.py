"""ctypes binding of libhvdx.so: one Python function per C entry point, same names.

Only argument marshalling happens here; every step of the path runs in the HIP
kernels behind the C-ABI.  A missing library raises at import: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhvdx.so")  # the library build() makes, next to this file

FLOAT32, FLOAT16 = 0, 1
SUM, AVERAGE = 0, 1
COMPRESS_NONE, COMPRESS_FP16 = 0, 1
PHASE_REDUCE_SCATTER, PHASE_ALLGATHER = 0, 1
COPY_IN, COPY_OUT = 0, 1
OK, ERR_INVALID, ERR_ALIAS, ERR_WORKSPACE, ERR_HIP, ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
MAX_RANKS = 128
DEFAULT_FUSION_THRESHOLD = 64 << 20
DEFAULT_FUSION_ALIGN = 16
SMALL_BUCKET_BYTES = 4 << 20  # HVDX_SMALL_BUCKET_BYTES

_p = ctypes.c_void_p
_i = ctypes.c_int
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t
_pp = ctypes.POINTER(ctypes.c_void_p)
_pi64 = ctypes.POINTER(ctypes.c_int64)
_pi32 = ctypes.POINTER(ctypes.c_int32)

_SIGNATURES = {
    "hvdx_fuse_plan": (_i, [_pi64, _i, _i, _i64, _i64, _pi32, _pi64, _pi64, _pi32, _pi32]),
    "hvdx_fuse_pack": (_i, [_p, _p, _p, _i, _i, _pp, _i64, _i, _i, _p]),
    "hvdx_fuse_unpack": (_i, [_pp, _i64, _i, _p, _p, _p, _i, _i, _i, _p]),
    "hvdx_fuse_pack_rs": (_i, [_p, _p, _p, _i, _i, _pp, _i64, _i, _i, _p]),
    "hvdx_fuse_ag_unpack": (_i, [_pp, _i64, _i, _p, _p, _p, _i, _i, _i, _p]),
    "hvdx_fuse_allreduce": (_i, [_p, _p, _p, _i, _i, _pp, _i64, _i, _i, _i, _p]),
    "hvdx_fuse_allreduce_small": (_i, [_p, _p, _p, _i, _i, _pp, _i64, _i, _i, _i, _p]),
    "hvdx_fuse_allreduce_pair": (_i, [_p, _p, _i, _i, _i, _i, _p]),
    "hvdx_fuse_copy_tiles": (_i64, [_pi64, _p, _i, _i64, _i, _i, _i, _i, _p, _i64]),
    "hvdx_fuse_allreduce_tiled": (_i, [_p, _i, _i, _i, _i, _i, _i, _p]),
    "hvdx_fuse_tile_elems": (_i64, [_i, _i]),
    "hvdx_ring_allreduce": (_i, [_pp, _i, _i64, _i, _i, _i, _p, _sz, _p]),
    "hvdx_ring_allreduce_small": (_i, [_pp, _i, _i64, _i, _i, _p]),
    "hvdx_ring_allreduce_noalloc": (_i, [_pp, _i, _i64, _i, _i, _i, _p]),
    "hvdx_ring_noalloc_max_bytes": (_sz, []),
    "hvdx_ring_step": (_i, [_pp, _i, _i64, _i, _i, _i, _i, _i, _p, _sz, _p]),
    "hvdx_ring_reduce_scatter": (_i, [_pp, _i, _i64, _i, _i, _i, _p, _sz, _p]),
    "hvdx_ring_allgather": (_i, [_pp, _i, _i64, _i, _i, _i, _p, _sz, _p]),
    "hvdx_ring_workspace_bytes": (_sz, [_i, _i64, _i, _i]),
    "hvdx_ring_chunk": (_i, [_i64, _i, _i, _pi64, _pi64]),
    "hvdx_strerror": (ctypes.c_char_p, [_i]),
    "hvdx_last_error": (ctypes.c_char_p, []),
    "hvdx_version": (_i, []),
    "hvdx_broadcast": (_i, [_pp, _i, _i64, _i, _p]),
    "hvdx_broadcast_step": (_i, [_pp, _i, _i64, _i, _i, _p]),
    "hvdx_broadcast_layout": (_i, [_pi64, _i, _pi64, _pi64]),
    "hvdx_broadcast_tensors": (_i, [_p, _p, _p, _i, _i64, _i, _i, _p]),
    "hvdx_broadcast_tensors_step": (_i, [_p, _p, _p, _i, _i64, _i, _i, _i, _p]),
    "hvdx_fold_allreduce": (_i, [_pp, _i, _i64, _i, _i, _i, _p]),
    "hvdx_timeline_begin": (_i, [_i, _i]),
    "hvdx_timeline_end": (_i, [_p, _i, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]),
}

KERNEL_PACK, KERNEL_REDUCE_SCATTER, KERNEL_ALLGATHER, KERNEL_UNPACK, KERNEL_ROUNDTRIP = 0, 1, 2, 3, 4
KERNEL_BROADCAST, KERNEL_RS_AG, KERNEL_FOLD = 5, 6, 7
KERNEL_PACK_RS, KERNEL_AG_UNPACK = 8, 9
KERNEL_RING_SMALL, KERNEL_CYCLE_SMALL = 10, 11
TILED_BUFFERS, TILED_REPLACE_IN_TENSORS, TILED_ADD_FROM_TENSORS = 0, 1, 2
TILED_MAX_BUCKETS, TILED_MAX_BUFFERS = 4, 256  # buckets per call; buckets x ranks in the tensor modes


class Bucket(ctypes.Structure):
    """hvdx_bucket: one fusion buffer's descriptors (device tables, host rank pointers)."""

    _fields_ = [
        ("tensors", ctypes.c_void_p),
        ("numel", ctypes.c_void_p),
        ("offset", ctypes.c_void_p),
        ("ntensors", ctypes.c_int),
        ("bufs", _pp),
        ("buf_count", ctypes.c_int64),
    ]


class CopyTile(ctypes.Structure):
    """hvdx_copy_tile: one tile of a fused copy (a stretch of one tensor or of padding,
    inside one ring chunk)."""

    _fields_ = [
        ("pos", ctypes.c_int64),
        ("li", ctypes.c_int64),
        ("tensor", ctypes.c_int32),
        ("len", ctypes.c_int32),
        ("chunk", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class TiledBucket(ctypes.Structure):
    """hvdx_tiled_bucket: a bucket and the device tile tables of its two fused copies."""

    _fields_ = [
        ("b", Bucket),
        ("in_tiles", ctypes.c_void_p),
        ("n_in", ctypes.c_int64),
        ("out_tiles", ctypes.c_void_p),
        ("n_out", ctypes.c_int64),
    ]


class TraceRecord(ctypes.Structure):
    """hvdx_trace_record"""

    _fields_ = [
        ("kind", ctypes.c_int32),
        ("step", ctypes.c_int32),
        ("launches", ctypes.c_int32),
        ("nranks", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("compress", ctypes.c_int32),
        ("root", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("count", ctypes.c_int64),
        ("start_us", ctypes.c_double),
        ("duration_us", ctypes.c_double),
    ]


class HvdxError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"hvdx status {status}: {detail}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_1802_05799_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def _check(status: int) -> None:
    if status != OK:
        detail = lib.hvdx_last_error().decode() or lib.hvdx_strerror(status).decode()
        raise HvdxError(status, detail)


def _ptr_array(ptrs):
    arr = (ctypes.c_void_p * max(1, len(ptrs)))(*[int(p) for p in ptrs])
    return ctypes.cast(arr, _pp), arr


def hvdx_version() -> int:
    return lib.hvdx_version()


def hvdx_strerror(status: int) -> str:
    return lib.hvdx_strerror(status).decode()


def hvdx_last_error() -> str:
    return lib.hvdx_last_error().decode()


def hvdx_ring_chunk(count: int, nranks: int, c: int):
    start, length = ctypes.c_int64(), ctypes.c_int64()
    _check(lib.hvdx_ring_chunk(count, nranks, c, ctypes.byref(start), ctypes.byref(length)))
    return start.value, length.value


def hvdx_ring_workspace_bytes(nranks: int, count: int, dtype: int, compress: int) -> int:
    return lib.hvdx_ring_workspace_bytes(nranks, count, dtype, compress)


def hvdx_fuse_plan(numel, buf_dtype: int, threshold_bytes: int = DEFAULT_FUSION_THRESHOLD,
                   align_bytes: int = DEFAULT_FUSION_ALIGN):
    """Return (bucket_of, offset, bucket_count, bucket_direct) as Python lists."""
    n = len(numel)
    a_numel = (ctypes.c_int64 * max(1, n))(*numel)
    bucket_of = (ctypes.c_int32 * max(1, n))()
    offset = (ctypes.c_int64 * max(1, n))()
    count = (ctypes.c_int64 * max(1, n))()
    direct = (ctypes.c_int32 * max(1, n))()
    nb = ctypes.c_int32()
    _check(lib.hvdx_fuse_plan(a_numel, n, buf_dtype, threshold_bytes, align_bytes, bucket_of, offset, count,
                              direct, ctypes.byref(nb)))
    k = nb.value
    return list(bucket_of[:n]), list(offset[:n]), list(count[:k]), list(direct[:k])


def hvdx_fuse_pack(srcs_dev: int, numel_dev: int, offset_dev: int, ntensors: int, src_dtype: int, bufs,
                   buf_count: int, buf_dtype: int, nranks: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fuse_pack(srcs_dev, numel_dev, offset_dev, ntensors, src_dtype, pb, buf_count, buf_dtype,
                              nranks, stream))


def hvdx_fuse_unpack(bufs, buf_count: int, buf_dtype: int, dsts_dev: int, numel_dev: int, offset_dev: int,
                     ntensors: int, dst_dtype: int, nranks: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fuse_unpack(pb, buf_count, buf_dtype, dsts_dev, numel_dev, offset_dev, ntensors, dst_dtype,
                                nranks, stream))


def hvdx_fuse_pack_rs(srcs_dev: int, numel_dev: int, offset_dev: int, ntensors: int, src_dtype: int, bufs,
                      buf_count: int, buf_dtype: int, nranks: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fuse_pack_rs(srcs_dev, numel_dev, offset_dev, ntensors, src_dtype, pb, buf_count, buf_dtype,
                                 nranks, stream))


def hvdx_fuse_ag_unpack(bufs, buf_count: int, buf_dtype: int, dsts_dev: int, numel_dev: int, offset_dev: int,
                        ntensors: int, dst_dtype: int, nranks: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fuse_ag_unpack(pb, buf_count, buf_dtype, dsts_dev, numel_dev, offset_dev, ntensors, dst_dtype,
                                   nranks, stream))


def hvdx_fuse_allreduce(tensors_dev: int, numel_dev: int, offset_dev: int, ntensors: int, tensor_dtype: int, bufs,
                        buf_count: int, buf_dtype: int, nranks: int, op: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fuse_allreduce(tensors_dev, numel_dev, offset_dev, ntensors, tensor_dtype, pb, buf_count,
                                   buf_dtype, nranks, op, stream))


def hvdx_fuse_allreduce_pair(b0, b1, tensor_dtype: int, buf_dtype: int, nranks: int, op: int,
                             stream: int = 0) -> None:
    """b0, b1: (tensors_dev, numel_dev, offset_dev, ntensors, bufs, buf_count) each."""
    keep = []

    def desc(b):
        tensors_dev, numel_dev, offset_dev, ntensors, bufs, buf_count = b
        pb, arr = _ptr_array(bufs)
        keep.append(arr)
        return Bucket(tensors_dev, numel_dev, offset_dev, ntensors, pb, buf_count)

    d0, d1 = desc(b0), desc(b1)
    _check(lib.hvdx_fuse_allreduce_pair(ctypes.addressof(d0), ctypes.addressof(d1), tensor_dtype, buf_dtype, nranks,
                                        op, stream))


def hvdx_fuse_copy_tiles(numel, offset, buf_count: int, tensor_dtype: int, buf_dtype: int, nranks: int,
                         direction: int):
    """The tile table of one fused copy of a buffer (host arrays in, a ctypes array of
    CopyTile out)."""
    n = len(numel)
    a_numel = (ctypes.c_int64 * max(1, n))(*numel)
    a_off = (ctypes.c_int64 * max(1, n))(*offset)
    args = (a_numel, a_off, n, buf_count, tensor_dtype, buf_dtype, nranks, direction)
    k = lib.hvdx_fuse_copy_tiles(*args, None, 0)
    if k < 0:
        _check(int(k))
    tiles = (CopyTile * max(1, k))()
    got = lib.hvdx_fuse_copy_tiles(*args, ctypes.cast(tiles, ctypes.c_void_p), k)
    if got < 0:
        _check(int(got))
    return tiles, k


def hvdx_fuse_tile_elems(tensor_dtype: int, buf_dtype: int) -> int:
    return lib.hvdx_fuse_tile_elems(tensor_dtype, buf_dtype)


def hvdx_fuse_allreduce_tiled(descs, tensor_dtype: int, buf_dtype: int, nranks: int, op: int, flags: int,
                              stream: int = 0) -> None:
    """descs: one to TILED_MAX_BUCKETS buckets, each (tensors_dev, numel_dev, offset_dev,
    ntensors, bufs, buf_count, in_tiles_dev, n_in, out_tiles_dev, n_out); flags:
    TILED_BUFFERS, or TILED_REPLACE_IN_TENSORS, optionally | TILED_ADD_FROM_TENSORS."""
    keep = []
    arr = (TiledBucket * max(1, len(descs)))()
    for i, t in enumerate(descs):
        tensors_dev, numel_dev, offset_dev, ntensors, bufs, buf_count, in_dev, n_in, out_dev, n_out = t
        pb, a = _ptr_array(bufs)
        keep.append(a)
        arr[i] = TiledBucket(Bucket(tensors_dev, numel_dev, offset_dev, ntensors, pb, buf_count), in_dev, n_in,
                             out_dev, n_out)
    _check(lib.hvdx_fuse_allreduce_tiled(ctypes.addressof(arr), len(descs), tensor_dtype, buf_dtype, nranks, op,
                                         flags, stream))


def hvdx_fuse_allreduce_small(tensors_dev: int, numel_dev: int, offset_dev: int, ntensors: int, tensor_dtype: int,
                              bufs, buf_count: int, buf_dtype: int, nranks: int, op: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fuse_allreduce_small(tensors_dev, numel_dev, offset_dev, ntensors, tensor_dtype, pb, buf_count,
                                         buf_dtype, nranks, op, stream))


def hvdx_ring_allreduce_small(bufs, nranks: int, count: int, dtype: int, op: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_ring_allreduce_small(pb, nranks, count, dtype, op, stream))


def hvdx_ring_allreduce(bufs, nranks: int, count: int, dtype: int, op: int, compress: int = COMPRESS_NONE,
                        workspace: int = 0, workspace_bytes: int = 0, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_ring_allreduce(pb, nranks, count, dtype, op, compress, workspace, workspace_bytes, stream))


def hvdx_ring_allreduce_noalloc(bufs, nranks: int, count: int, dtype: int, op: int, compress: int = COMPRESS_NONE,
                                stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_ring_allreduce_noalloc(pb, nranks, count, dtype, op, compress, stream))


def hvdx_ring_noalloc_max_bytes() -> int:
    return lib.hvdx_ring_noalloc_max_bytes()


def hvdx_ring_reduce_scatter(bufs, nranks: int, count: int, dtype: int, op: int, compress: int = COMPRESS_NONE,
                             workspace: int = 0, workspace_bytes: int = 0, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_ring_reduce_scatter(pb, nranks, count, dtype, op, compress, workspace, workspace_bytes, stream))


def hvdx_ring_allgather(bufs, nranks: int, count: int, dtype: int, op: int, compress: int = COMPRESS_NONE,
                        workspace: int = 0, workspace_bytes: int = 0, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_ring_allgather(pb, nranks, count, dtype, op, compress, workspace, workspace_bytes, stream))


def hvdx_ring_step(bufs, nranks: int, count: int, dtype: int, op: int, compress: int, phase: int, step: int,
                   workspace: int = 0, workspace_bytes: int = 0, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_ring_step(pb, nranks, count, dtype, op, compress, phase, step, workspace, workspace_bytes,
                              stream))


def hvdx_timeline_begin(capacity: int, per_phase: bool = False) -> None:
    _check(lib.hvdx_timeline_begin(capacity, 1 if per_phase else 0))


def hvdx_timeline_end(capacity: int):
    """Return (records as dicts, number dropped)."""
    arr = (TraceRecord * max(1, capacity))()
    n, dropped = ctypes.c_int(), ctypes.c_int()
    _check(lib.hvdx_timeline_end(ctypes.cast(arr, ctypes.c_void_p), capacity, ctypes.byref(n), ctypes.byref(dropped)))
    recs = [{f: getattr(arr[i], f) for f, _ in TraceRecord._fields_ if f != "reserved"} for i in range(n.value)]
    return recs, dropped.value


def hvdx_broadcast(bufs, nranks: int, nbytes: int, root: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_broadcast(pb, nranks, nbytes, root, stream))


def hvdx_broadcast_step(bufs, nranks: int, nbytes: int, root: int, step: int, stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_broadcast_step(pb, nranks, nbytes, root, step, stream))


def hvdx_fold_allreduce(bufs, nranks: int, count: int, dtype: int, op: int, compress: int = COMPRESS_NONE,
                        stream: int = 0) -> None:
    pb, _keep = _ptr_array(bufs)
    _check(lib.hvdx_fold_allreduce(pb, nranks, count, dtype, op, compress, stream))


def hvdx_broadcast_layout(nbytes):
    """(virtual start of each tensor, length of the space) for hvdx_broadcast_tensors."""
    n = len(nbytes)
    a = (ctypes.c_int64 * max(1, n))(*nbytes)
    off = (ctypes.c_int64 * max(1, n))()
    total = ctypes.c_int64()
    _check(lib.hvdx_broadcast_layout(a, n, off, ctypes.byref(total)))
    return list(off[:n]), total.value


def hvdx_broadcast_tensors(ptrs_dev: int, nbytes_dev: int, voffset_dev: int, ntensors: int, total_bytes: int,
                           nranks: int, root: int, stream: int = 0) -> None:
    _check(lib.hvdx_broadcast_tensors(ptrs_dev, nbytes_dev, voffset_dev, ntensors, total_bytes, nranks, root, stream))


def hvdx_broadcast_tensors_step(ptrs_dev: int, nbytes_dev: int, voffset_dev: int, ntensors: int, total_bytes: int,
                                nranks: int, root: int, step: int, stream: int = 0) -> None:
    _check(lib.hvdx_broadcast_tensors_step(ptrs_dev, nbytes_dev, voffset_dev, ntensors, total_bytes, nranks, root,
                                           step, stream))
