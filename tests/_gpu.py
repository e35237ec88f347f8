"""Helpers for the GPU parity tests (host side: moving numpy arrays to and from the GPU
and calling the C-ABI through the binding)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import paper_1802_05799_amd as hv

NP_TO_HV = {np.dtype(np.float32): hv.FLOAT32, np.dtype(np.float16): hv.FLOAT16}
NP_TO_TORCH = {np.dtype(np.float32): torch.float32, np.dtype(np.float16): torch.float16}
OPS = {"sum": hv.SUM, "average": hv.AVERAGE}


def say(msg: str) -> None:
    """Name the case before GPU work starts, so a fault report says which case it was."""
    print(msg, flush=True)
    sys.stdout.flush()


def to_gpu_rows(x: np.ndarray, offset_elems: int = 0):
    """One GPU tensor per row; with offset_elems > 0 each is a view that starts that many
    elements into its allocation (so it is not 16-byte aligned)."""
    out, keep = [], []
    for row in x:
        base = torch.zeros(row.size + offset_elems + 64, dtype=NP_TO_TORCH[x.dtype], device="cuda")
        v = base[offset_elems : offset_elems + row.size]
        v.copy_(torch.from_numpy(np.ascontiguousarray(row)))
        out.append(v)
        keep.append(base)
    return out, keep


def from_gpu_rows(rows) -> np.ndarray:
    torch.cuda.synchronize()
    return np.stack([r.cpu().numpy() for r in rows]) if rows else np.zeros((0, 0))


def gpu_ring(x: np.ndarray, op: str, compress: bool = False, offset_elems: int = 0) -> np.ndarray:
    """hvdx_ring_allreduce on a copy of x (N, count); returns the N result rows."""
    n, count = x.shape
    rows, keep = to_gpu_rows(x, offset_elems)
    dt = NP_TO_HV[x.dtype]
    cmp = hv.COMPRESS_FP16 if compress else hv.COMPRESS_NONE
    wsb = hv.hvdx_ring_workspace_bytes(n, count, dt, cmp)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device="cuda")
    hv.hvdx_ring_allreduce([r.data_ptr() for r in rows], n, count, dt, OPS[op], cmp, ws.data_ptr() if wsb else 0,
                           wsb, torch.cuda.current_stream().cuda_stream)
    out = from_gpu_rows(rows)
    del keep
    return out


def bits(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    return a.view({1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[a.dtype.itemsize])


def assert_bits_equal(got: np.ndarray, want: np.ndarray, what: str = "") -> None:
    assert got.dtype == want.dtype and got.shape == want.shape, (what, got.dtype, want.dtype, got.shape, want.shape)
    gb, wb = bits(got), bits(want)
    if not np.array_equal(gb, wb):
        bad = np.argwhere(gb != wb)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} mismatches, first at {i}: got {got[i]!r} want {want[i]!r}")
