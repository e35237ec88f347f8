"""Fill GPU tensors with the synthetic values of `workloads.rng` (ctypes binding of
libwlfill.so).  torch must be imported before this module loads the library."""
from __future__ import annotations

import ctypes
import os

import torch

from . import configs

_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwlfill.so")
if not os.path.exists(_LIB):
    raise ImportError(f"{_LIB} is not built; run `python -m workloads.build`")
_lib = ctypes.CDLL(_LIB)
_lib.wl_fill_f32.restype = ctypes.c_int
_lib.wl_fill_f32.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int64, ctypes.c_int,
                             ctypes.c_float, ctypes.c_void_p]
_DIST = {"uniform": 0, "normal": 1}


def fill_(x: torch.Tensor, dist: str, key: int, first_index: int, sigma: float = 0.01) -> torch.Tensor:
    """Write values for element indices first_index .. first_index + x.numel() - 1."""
    if x.dtype != torch.float32 or not x.is_contiguous() or x.device.type != "cuda":
        raise ValueError("fill_ needs a contiguous float32 GPU tensor")
    stream = torch.cuda.current_stream(x.device).cuda_stream
    rc = _lib.wl_fill_f32(x.data_ptr(), x.numel(), key, first_index, _DIST[dist], sigma, stream)
    if rc != 0:
        raise RuntimeError(f"wl_fill_f32 failed ({rc})")
    return x


def make_rank_tensors(w: configs.Workload, device="cuda", align_elems: int = 64):
    """Every rank's gradient tensors for workload `w`, filled with its values.

    Each rank's tensors are views into one zeroed allocation, each starting at a
    multiple of `align_elems` elements (256 bytes by default, like separate
    allocations would), so setting up thousands of tensors costs one allocation per
    rank.  Returns (per-rank tensor lists, per-rank flat storage, view starts).
    """
    numel = w.numel()
    starts, acc = [], 0
    for n in numel:
        starts.append(acc)
        acc += -(-n // align_elems) * align_elems
    out, storage = [], []
    for r in range(w.nranks):
        flat = torch.zeros(max(acc, 1), dtype=torch.float32, device=device)
        storage.append(flat)
        ts = []
        for (name, shape), s, n, pre in zip(w.tensors(), starts, numel, w.prefix()):
            t = flat[s : s + n].view(shape)
            fill_(t.view(-1), w.dist, w.key(r), pre, w.sigma)
            ts.append(t)
        out.append(ts)
    return out, storage, starts


def fill_rank_flat_(flat: torch.Tensor, w: configs.Workload, rank: int, starts) -> torch.Tensor:
    """Rewrite one rank's values into a flat storage laid out as by make_rank_tensors."""
    for s, n, pre in zip(starts, w.numel(), w.prefix()):
        fill_(flat[s : s + n], w.dist, w.key(rank), pre, w.sigma)
    return flat
