"""ctypes binding of the plain C oracle (oracle/csrc/oracle.c).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The C oracle computes what ``allreduce``, ``fusion`` and ``ring`` compute, in the
same order and precision (section 7's fusion steps around section 3's ring,
averaged as in section 5), over whole workloads and optionally on several host
threads.  The library is built by ``oracle/build.py`` (also run by the package's
top-level build); it is compiled here on first use only when it is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import ring

__all__ = ["lib", "allreduce", "workspace_bytes", "ring_allreduce", "fuse_plan", "f32_to_f16", "f16_to_f32", "max_threads"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None
lib_path = [os.path.join(_HERE, "liboracle.so")]

F32, F16 = 0, 1
_OPS = {ring.SUM: 0, ring.AVERAGE: 1}


def lib():
    global _LIB
    if _LIB is None:
        path = lib_path[0]
        if not os.path.exists(path):
            import importlib.util

            spec = importlib.util.spec_from_file_location("_oracle_build", os.path.join(_HERE, "build.py"))
            mod = importlib.util.module_from_spec(spec)
            spec.loader.exec_module(mod)
            mod.build()
        L = C.CDLL(path)
        P, I64 = C.c_void_p, C.c_int64
        L.oracle_last_error.restype = C.c_char_p
        L.oracle_fuse_plan.argtypes = [P, C.c_int, C.c_int, I64, I64, P, P, P, P, C.POINTER(C.c_int)]
        L.oracle_ring.argtypes = [P, C.c_int, I64, C.c_int, C.c_int, C.c_int]
        L.oracle_allreduce.argtypes = [P, P, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, I64, I64, P, P, I64,
                                       C.c_int]
        L.oracle_workspace_bytes.argtypes = [P, C.c_int, C.c_int, C.c_int, C.c_int, I64, I64]
        L.oracle_workspace_bytes.restype = I64
        L.oracle_f32_to_f16_array.argtypes = [P, P, I64]
        L.oracle_f16_to_f32_array.argtypes = [P, P, I64]
        L.oracle_f32_to_f16_array.restype = None
        L.oracle_f16_to_f32_array.restype = None
        L.oracle_max_threads.restype = C.c_int
        _LIB = L
    return _LIB


def use_library(path):
    """Bind to another build of the C source (the tests load planted-mistake copies);
    returns the previously bound library handle."""
    global _LIB
    prev = _LIB
    _LIB = None
    lib_path[0] = path
    lib()
    return prev


def restore_library(handle):
    global _LIB
    _LIB = handle
    lib_path[0] = os.path.join(_HERE, "liboracle.so")


def _check(rc):
    if rc != 0:
        raise ValueError(lib().oracle_last_error().decode())


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p)


def max_threads() -> int:
    return int(lib().oracle_max_threads())


def f32_to_f16(x):
    """binary32 -> binary16, rounded to nearest even (array in, uint16 bit patterns out)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_f32_to_f16_array(_ptr(x), _ptr(out), x.size)
    return out


def f16_to_f32(h):
    """binary16 bit patterns (uint16) -> binary32, exact."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, dtype=np.float32)
    lib().oracle_f16_to_f32_array(_ptr(h), _ptr(out), h.size)
    return out


def fuse_plan(numel, esize, threshold=64 << 20, align=16):
    """(bucket of each tensor, element offset of each tensor, direct flag per bucket,
    length per bucket) of section 7's plan."""
    t = len(numel)
    nm = np.asarray(numel, dtype=np.int64)
    bucket_of = np.zeros(max(t, 1), dtype=np.int32)
    offset = np.zeros(max(t, 1), dtype=np.int64)
    direct = np.zeros(max(t, 1), dtype=np.int32)
    count = np.zeros(max(t, 1), dtype=np.int64)
    nb = C.c_int(0)
    _check(lib().oracle_fuse_plan(_ptr(nm), t, esize, threshold, align, _ptr(bucket_of), _ptr(offset), _ptr(direct),
                                  _ptr(count), C.byref(nb)))
    b = nb.value
    return bucket_of[:t], offset[:t], direct[:b].astype(bool), count[:b]


def ring_allreduce(bufs, op=ring.AVERAGE, threads=1):
    """Section 3's ring in place on `bufs` (N, count), binary32 or binary16."""
    if bufs.dtype == np.float32:
        dtype = F32
    elif bufs.dtype == np.float16:
        dtype = F16
    else:
        raise TypeError(f"unsupported buffer dtype {bufs.dtype}")
    if not bufs.flags.c_contiguous:
        raise ValueError("bufs must be C-contiguous")
    n, count = bufs.shape
    ptrs = (C.c_void_p * n)(*[bufs[r].ctypes.data for r in range(n)])
    _check(lib().oracle_ring(ptrs, n, count, dtype, _OPS[op], threads))
    return bufs


def workspace_bytes(numel, nranks, dtype=np.float32, compress=False, threshold=64 << 20, align=16):
    """Bytes of the N fusion buffers of the plan's largest buffer."""
    nm = np.asarray(numel, dtype=np.int64) if len(numel) else np.zeros(1, dtype=np.int64)
    src = F16 if np.dtype(dtype) == np.float16 else F32
    v = lib().oracle_workspace_bytes(_ptr(nm), len(numel), nranks, src, int(bool(compress)), threshold, align)
    if v < 0:
        raise ValueError(lib().oracle_last_error().decode())
    return int(v)


def allreduce(per_rank, op=ring.AVERAGE, compress=False, threshold=64 << 20, align=16, threads=1, out=None,
              workspace=None):
    """Every rank's reduced tensors, as ``oracle.allreduce.allreduce`` returns them.

    per_rank  -- per_rank[r][t]: rank r's t-th tensor, binary32 or binary16, contiguous.
    out       -- optional preallocated outputs of the same shapes (reused across calls).
    workspace -- optional uint8 array of at least ``workspace_bytes`` bytes holding the
                 fusion buffers (reused across calls, as the paper allocates the fusion
                 buffer once); without it every buffer is allocated per call.
    """
    n = len(per_rank)
    t = len(per_rank[0]) if n else 0
    xs = [[np.ascontiguousarray(a) for a in ts] for ts in per_rank]
    src = xs[0][0].dtype if t else np.dtype(np.float32)
    if src == np.float32:
        dtype = F32
    elif src == np.float16:
        dtype = F16
    else:
        raise TypeError(f"unsupported tensor dtype {src}")
    if out is None:
        out = [[np.empty_like(a) for a in ts] for ts in xs]
    numel = np.asarray([a.size for a in xs[0]], dtype=np.int64) if t else np.zeros(1, dtype=np.int64)
    xp = (C.c_void_p * max(n * t, 1))(*[a.ctypes.data for ts in xs for a in ts])
    yp = (C.c_void_p * max(n * t, 1))(*[a.ctypes.data for ts in out for a in ts])
    ws, ws_bytes = (None, 0) if workspace is None else (_ptr(workspace), workspace.nbytes)
    _check(lib().oracle_allreduce(xp, _ptr(numel), t, n, dtype, _OPS[op], int(bool(compress)), threshold, align, yp,
                                  ws, ws_bytes, threads))
    return out
