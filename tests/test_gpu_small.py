"""The one-launch paths for small buffers against the oracle, bit for bit:
hvdx_ring_allreduce_small (every ring step for every element, in place, in one launch)
and hvdx_fuse_allreduce_small (copy-in, the whole ring and copy-out in one launch), plus
FusedAllreduce choosing them for small buckets."""
import numpy as np
import pytest
import torch

import paper_1802_05799_amd as hv
from _gpu import NP_TO_HV, OPS, assert_bits_equal, from_gpu_rows, say, to_gpu_rows
from oracle import allreduce, fusion, ring
from test_gpu_fusion import descriptors, make_tensors
from test_gpu_ring import CASES, inputs, oracle_ring

pytestmark = pytest.mark.gpu


def gpu_ring_small(x: np.ndarray, op: str, offset_elems: int = 0) -> np.ndarray:
    n, count = x.shape
    rows, keep = to_gpu_rows(x, offset_elems)
    hv.hvdx_ring_allreduce_small([r.data_ptr() for r in rows], n, count, NP_TO_HV[x.dtype], OPS[op],
                                 torch.cuda.current_stream().cuda_stream)
    return from_gpu_rows(rows)


@pytest.mark.parametrize("dtype", [np.float32, np.float16], ids=["f32", "f16"])
def test_ring_small_matches_oracle(dtype):
    rng = np.random.default_rng(200)
    for n, count in CASES:
        for op in ("sum", "average"):
            say(f"small ring dtype={np.dtype(dtype).name} n={n} count={count} op={op}")
            x = inputs(rng, n, count, dtype)
            assert_bits_equal(gpu_ring_small(x, op), oracle_ring(x, op), f"n={n} count={count} op={op}")


def test_ring_small_unaligned_and_special_values():
    rng = np.random.default_rng(201)
    for off in (1, 3):
        for n, count in ((3, 1001), (8, 40000), (5, 7)):
            for dtype in (np.float32, np.float16):
                say(f"small ring unaligned off={off} n={n} count={count} {np.dtype(dtype).name}")
                x = inputs(rng, n, count, dtype)
                assert_bits_equal(gpu_ring_small(x, "average", off), oracle_ring(x, "average"))
    x32 = (rng.standard_normal((4, 4096)) * 1e-5).astype(np.float32)
    x32[:, :8] = np.array([0.0, -0.0, 1.0, 2.0 ** -24, 65504.0, 65520.0, np.inf, -np.inf], np.float32)
    x32[1, 8:16] = 2.0 ** 24
    x32[:, 16:24] = 1.0
    x16 = fusion.cast(x32, np.float16)
    for nr in (4, 3, 2):
        for op in ("sum", "average"):
            say(f"small ring special values n={nr} op={op}")
            assert_bits_equal(gpu_ring_small(x32[:nr].copy(), op), oracle_ring(x32[:nr].copy(), op), "f32")
            assert_bits_equal(gpu_ring_small(x16[:nr].copy(), op), oracle_ring(x16[:nr].copy(), op), "f16")


SMALL_CASES = [
    # (numel list, nranks, buffer dtype, align bytes, op)
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, np.float32, 16, "average"),  # the tiny workload
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 1, np.float32, 16, "average"),  # one rank
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 2, np.float16, 16, "sum"),  # binary16 buffer
    ([0, 1, 0, 3, 5, 0, 0, 2, 17], 3, np.float32, 16, "sum"),  # empty and tiny tensors
    ([1] * 3000 + [5000], 5, np.float32, 16, "average"),  # many tensors per tile
    ([33, 31, 1, 2, 3, 4, 5, 6, 7, 8, 9, 100000], 7, np.float32, 4, "average"),  # vectors cross chunk ends
    ([257] * 40 + [70000, 3, 9000], 6, np.float16, 16, "average"),
    ([1, 0, 2], 8, np.float32, 16, "sum"),  # fewer buffer elements than ranks
    ([3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9], 13, np.float16, 2, "average"),
    ([5000, 300, 70000], 32, np.float32, 16, "average"),
    ([5000, 300, 70001], 128, np.float16, 2, "average"),  # the most ranks a call takes
]


@pytest.mark.parametrize("misalign", [False, True], ids=["aligned", "misaligned"])
@pytest.mark.parametrize("case", range(len(SMALL_CASES)))
def test_fuse_allreduce_small_matches_oracle(case, misalign):
    numel, n, buf_np, align, op = SMALL_CASES[case]
    rng = np.random.default_rng(210 + case)
    host, dev, keep = make_tensors(rng, n, numel, np.float32, misalign)
    (b,) = fusion.fuse_plan(numel, np.dtype(buf_np).itemsize, 1 << 40, align)
    say(f"small cycle case={case} n={n} buffer={np.dtype(buf_np).name} misalign={misalign} count={b.count}")
    ptrs, nm, off = descriptors(dev, b, numel)
    bufs = [torch.full((max(b.count, 1),), 7.0, dtype=torch.float32 if buf_np == np.float32 else torch.float16,
                       device="cuda") for _ in range(n)]
    hv.hvdx_fuse_allreduce_small(ptrs.data_ptr(), nm.data_ptr(), off.data_ptr(), len(numel), hv.FLOAT32,
                                 [x.data_ptr() for x in bufs], b.count, NP_TO_HV[np.dtype(buf_np)], n, OPS[op],
                                 torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    work = np.stack([fusion.pack(host[r], b, buf_np) for r in range(n)])
    ring.ring_allreduce(work, op)
    for r in range(n):
        want = fusion.unpack(work[r], b, numel, np.float32)
        for t in range(len(numel)):
            assert_bits_equal(dev[r][t].cpu().numpy(), want[t], f"rank {r} tensor {t}")


@pytest.mark.parametrize("small_bytes", [0, hv.SMALL_BUCKET_BYTES, 1 << 40], ids=["per-step", "default", "all"])
def test_fused_allreduce_picks_either_path_with_the_same_bits(small_bytes):
    """Mixed plan (fused buckets, direct tensors, compression) through FusedAllreduce
    with no, the default, and every bucket on the one-launch path."""
    numel = [3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9, 7]
    for compress in (False, True):
        rng = np.random.default_rng(220)
        host, dev, keep = make_tensors(rng, 6, numel, np.float32)
        say(f"FusedAllreduce small_bucket_bytes={small_bytes} compress={compress}")
        ar = hv.FusedAllreduce(dev, op="average", compress=compress, threshold_bytes=40000,
                               small_bucket_bytes=small_bytes)
        kinds = {k for k, _, _ in ar.kernel_sequence()}
        assert ("cycle_small" in kinds) == (small_bytes > 0)
        ar()
        torch.cuda.synchronize()
        want = allreduce.allreduce(host, "average", compress=compress, threshold=40000)
        for r in range(6):
            for t in range(len(numel)):
                assert_bits_equal(dev[r][t].cpu().numpy(), want[r][t], f"rank {r} tensor {t}")
