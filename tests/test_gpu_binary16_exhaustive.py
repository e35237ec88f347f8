"""Every binary16 sum and every binary32 -> binary16 rounding, on the GPU, against the oracle.

Sums: a two-rank SUM ring computes each element as one addition of the two ranks'
values (rank 1 adds rank 0's chunk-0 value to its own, rank 0 adds rank 1's chunk-1
value; the replacing step copies the sums across).  Rank 0 holds every binary16
pattern a and rank 1 every pattern b, so 2^32 elements, in eight slices by the top
three bits of a, cover every pair once.

Rounding: the copy-in of one binary32 tensor into a binary16 buffer (the compressed
path's first step) sees every one of the 2^32 binary32 patterns, in eight slices.

Results must equal the oracle bit for bit: that pins the GPU's binary16 addition and
its binary32 -> binary16 conversion (round to nearest even, subnormals kept, overflow
to infinity) on every input, not only on the workloads' values.  NaN results are
compared as "both NaN": payloads are not part of the claim.  The oracle runs in a
pool of spawned processes (numpy's binary16 conversions are slow)."""
import multiprocessing
import os

import numpy as np
import pytest
import torch

import _binary16_oracle as O
import paper_1802_05799_amd as hv
from _gpu import bits, gpu_ring, say

pytestmark = pytest.mark.gpu

SLICES = 8
PER_SLICE = (1 << 32) // SLICES
BLOCK = 1 << 25  # oracle elements per worker task


@pytest.fixture(scope="module")
def pool():
    workers = max(1, min(16, os.cpu_count() or 1))
    with multiprocessing.get_context("spawn").Pool(workers) as p:
        yield p


def is_nan16(u: np.ndarray) -> np.ndarray:
    return ((u & 0x7C00) == 0x7C00) & ((u & 0x03FF) != 0)


def assert_same16(got: np.ndarray, want: np.ndarray, what: str) -> None:
    gb, wb = bits(got), bits(want)
    same = (gb == wb) | (is_nan16(wb) & is_nan16(gb))
    if not same.all():
        i = int(np.argmin(same))
        raise AssertionError(f"{what}: {int((~same).sum())} mismatches, first at element {i}: "
                             f"got {gb[i]:#06x} want {wb[i]:#06x}")


@pytest.mark.parametrize("part", range(SLICES))
def test_every_binary16_sum(part, pool):
    say(f"binary16 sums: slice {part} of {SLICES}, {PER_SLICE} pairs")
    base = part * (PER_SLICE >> 16)
    tasks = [(base, lo, lo + BLOCK, PER_SLICE) for lo in range(0, PER_SLICE, BLOCK)]
    pending = pool.map_async(O.ring_sum_block, tasks)  # the oracle, while the GPU works
    got = gpu_ring(O.pairs(base, 0, PER_SLICE), "sum")
    want = np.concatenate(pending.get(timeout=100), axis=1)
    for r in range(2):
        assert_same16(got[r], want[r], f"rank {r} slice {part}")


@pytest.mark.parametrize("part", range(SLICES))
def test_every_binary32_to_binary16(part, pool):
    lo = part * PER_SLICE
    say(f"binary32 -> binary16 copy-in: patterns {lo:#010x} .. {lo + PER_SLICE - 1:#010x}")
    pending = pool.map_async(O.pack16_block, [(b, b + BLOCK) for b in range(lo, lo + PER_SLICE, BLOCK)])
    src = torch.from_numpy(O.patterns32(lo, lo + PER_SLICE)).cuda()
    buf = torch.empty(PER_SLICE, dtype=torch.float16, device="cuda")
    ptrs = torch.tensor([src.data_ptr()], dtype=torch.int64, device="cuda")
    numel = torch.tensor([PER_SLICE], dtype=torch.int64, device="cuda")
    offset = torch.zeros(1, dtype=torch.int64, device="cuda")
    hv.hvdx_fuse_pack(ptrs.data_ptr(), numel.data_ptr(), offset.data_ptr(), 1, hv.FLOAT32, [buf.data_ptr()],
                      PER_SLICE, hv.FLOAT16, 1, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got = buf.cpu().numpy()
    del src, buf
    want = np.concatenate(pending.get(timeout=110))
    assert_same16(got, want, f"slice {part}")
