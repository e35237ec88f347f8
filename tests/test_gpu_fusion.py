"""GPU copy-in / copy-out kernels and the whole Tensor Fusion cycle against the oracle."""
import numpy as np
import pytest
import torch

import paper_1802_05799_amd as hv
from _gpu import NP_TO_HV, NP_TO_TORCH, assert_bits_equal, say
from oracle import allreduce, fusion, ring

pytestmark = pytest.mark.gpu


def make_tensors(rng, n, numel, dtype, misalign=False):
    """Per-rank numpy tensors and their GPU copies (optionally at odd element offsets)."""
    host = [[(rng.standard_normal(k) * 0.01).astype(dtype) for k in numel] for _ in range(n)]
    dev, keep = [], []
    for r in range(n):
        row = []
        for t, x in enumerate(host[r]):
            off = (t * 3 + r) % 5 if misalign else 0
            base = torch.zeros(x.size + off + 8, dtype=NP_TO_TORCH[x.dtype], device="cuda")
            v = base[off : off + x.size]
            v.copy_(torch.from_numpy(x))
            row.append(v)
            keep.append(base)
        dev.append(row)
    return host, dev, keep


def descriptors(dev, bucket, numel):
    n = len(dev)
    ptrs = torch.tensor([dev[r][t].data_ptr() for r in range(n) for t in bucket.tensors], dtype=torch.int64,
                        device="cuda")
    nm = torch.tensor([numel[t] for t in bucket.tensors], dtype=torch.int64, device="cuda")
    off = torch.tensor(bucket.offsets, dtype=torch.int64, device="cuda")
    return ptrs, nm, off


PACK_CASES = [
    # (numel list, nranks, buffer esize, align bytes)
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, 4, 16),
    ([0, 1, 0, 3, 5, 0, 0, 2, 17], 3, 4, 16),
    ([1] * 3000 + [5000], 2, 4, 16),  # 1024 tensors in one tile
    ([1] * 3000 + [5000], 2, 4, 4),  # more tensors in one tile than LDS holds
    ([0] * 2000 + [5, 0, 0, 7] + [0] * 500 + [100], 3, 4, 16),  # runs of empty tensors
    ([33, 31, 1, 2, 3, 4, 5, 6, 7, 8, 9, 100000], 5, 4, 4),  # no padding between tensors
    ([33, 31, 1, 2, 3, 4, 5, 6, 7, 8, 9, 100000], 5, 4, 64),
    ([257] * 40 + [70000, 3, 9000], 7, 2, 16),  # binary16 buffer
    ([257] * 40 + [70000, 3, 9000], 7, 2, 2),
    ([5000, 3, 70000], 128, 4, 16),  # the most ranks a call takes
]


@pytest.mark.parametrize("misalign", [False, True], ids=["aligned", "misaligned"])
@pytest.mark.parametrize("case", range(len(PACK_CASES)))
def test_pack_unpack_match_oracle(case, misalign):
    numel, n, esize, align = PACK_CASES[case]
    rng = np.random.default_rng(200 + case)
    buf_np = np.float32 if esize == 4 else np.float16
    host, dev, keep = make_tensors(rng, n, numel, np.float32, misalign)
    plan = fusion.fuse_plan(numel, esize, threshold=1 << 30, align=align)
    (b,) = plan
    say(f"pack case={case} misalign={misalign} count={b.count} tensors={len(numel)} n={n}")
    ptrs, nm, off = descriptors(dev, b, numel)
    bufs = [torch.full((b.count + 64,), 7.0, dtype=NP_TO_TORCH[np.dtype(buf_np)], device="cuda") for _ in range(n)]
    st = torch.cuda.current_stream().cuda_stream
    hv.hvdx_fuse_pack(ptrs.data_ptr(), nm.data_ptr(), off.data_ptr(), len(b.tensors), hv.FLOAT32,
                      [x.data_ptr() for x in bufs], b.count, NP_TO_HV[np.dtype(buf_np)], n, st)
    torch.cuda.synchronize()
    for r in range(n):
        want = fusion.pack(host[r], b, buf_np)
        got = bufs[r].cpu().numpy()
        assert_bits_equal(got[: b.count], want, f"pack rank {r}")
        assert np.all(got[b.count :] == 7.0), "pack wrote past the buffer"
    # scribble the tensors, then copy the buffers back out
    for r in range(n):
        for x in dev[r]:
            x.fill_(-3.0)
    hv.hvdx_fuse_unpack([x.data_ptr() for x in bufs], b.count, NP_TO_HV[np.dtype(buf_np)], ptrs.data_ptr(),
                        nm.data_ptr(), off.data_ptr(), len(b.tensors), hv.FLOAT32, n, st)
    torch.cuda.synchronize()
    for r in range(n):
        want = fusion.unpack(fusion.pack(host[r], b, buf_np), b, numel, np.float32)
        for t in b.tensors:
            assert_bits_equal(dev[r][t].cpu().numpy(), want[t], f"unpack rank {r} tensor {t}")


def test_unpack_does_not_write_outside_tensors():
    rng = np.random.default_rng(210)
    numel = [5, 3, 9, 1]
    n = 2
    plan = fusion.fuse_plan(numel, 4, threshold=1 << 20)
    (b,) = plan
    guard = [torch.full((64,), 11.0, device="cuda") for _ in range(n * len(numel))]
    dev = [[guard[r * len(numel) + t][8 : 8 + numel[t]] for t in range(len(numel))] for r in range(n)]
    ptrs, nm, off = descriptors(dev, b, numel)
    bufs = [torch.from_numpy((rng.standard_normal(b.count)).astype(np.float32)).cuda() for _ in range(n)]
    hv.hvdx_fuse_unpack([x.data_ptr() for x in bufs], b.count, hv.FLOAT32, ptrs.data_ptr(), nm.data_ptr(),
                        off.data_ptr(), len(numel), hv.FLOAT32, n, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    for r in range(n):
        for t in range(len(numel)):
            g = guard[r * len(numel) + t].cpu().numpy()
            assert np.all(g[:8] == 11.0) and np.all(g[8 + numel[t] :] == 11.0)
            assert_bits_equal(g[8 : 8 + numel[t]], bufs[r].cpu().numpy()[b.offsets[t] : b.offsets[t] + numel[t]])


CYCLE_CASES = [
    # (numel, nranks, threshold bytes, compress, op)
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, 64 << 20, False, "average"),
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, 4096, False, "sum"),  # several buckets + direct tensors
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 3, 4096, True, "average"),
    ([3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9], 6, 40000, True, "average"),
    ([3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9], 5, 40000, False, "average"),
    ([1], 1, 64, True, "average"),
    ([5000, 300, 70000, 9], 128, 40000, False, "average"),  # the most ranks a call takes
    ([5000, 300, 70000, 9], 128, 40000, True, "average"),
    ([0, 5, 0, 0, 7, 1, 0], 8, 64 << 20, False, "average"),  # empty tensors; fewer elements than ranks
    ([0, 5, 0, 0, 7, 1, 0], 8, 64 << 20, True, "sum"),
    ([1, 0, 1], 3, 64, False, "sum"),  # one element per bucket
]


@pytest.mark.parametrize("mode", ["ring", "ring-misaligned", "ring-copy-in", "ring-buffers", "ring-lookup",
                                  "ring-one-launch", "ring-separate", "fold"])
@pytest.mark.parametrize("case", range(len(CYCLE_CASES)))
def test_fused_allreduce_matches_oracle(case, mode):
    """"ring": the fused boundary, tile-driven, with the adding steps reading the ranks' own
    values from their tensors and the replacing steps delivering into them (compressed:
    the compressed ring's form of it); "ring-misaligned": the same with tensors at odd element offsets
    (the element paths); "ring-copy-in": the copy-in fused with adding step 0, the rest
    of the adding steps in the buffers, the replacing steps into the tensors;
    "ring-buffers": the ring in the fusion buffers between the fused copies;
    "ring-lookup": the copies that find their tensors in the kernel (hvdx_fuse_allreduce,
    hvdx_fuse_allreduce_pair)."""
    numel, n, threshold, compress, op = CYCLE_CASES[case]
    rng = np.random.default_rng(300 + case)
    host, dev, keep = make_tensors(rng, n, numel, np.float32, misalign=mode == "ring-misaligned")
    say(f"cycle case={case} n={n} threshold={threshold} compress={compress} mode={mode}")
    ar = hv.FusedAllreduce(dev, op=op, compress=compress, threshold_bytes=threshold,
                           schedule="fold" if mode == "fold" else "ring",
                           fuse_boundary=mode in ("ring", "ring-misaligned", "ring-copy-in", "ring-buffers",
                                                  "ring-lookup", "ring-one-launch"),
                           small_bucket_bytes=hv.SMALL_BUCKET_BYTES if mode == "ring-one-launch" else 0,
                           tiled=mode != "ring-lookup", replace_in_tensors=mode != "ring-buffers",
                           add_from_tensors=mode not in ("ring-copy-in", "ring-buffers"))
    ar()
    torch.cuda.synchronize()
    want = allreduce.allreduce(host, op, compress=compress, threshold=threshold)
    for r in range(n):
        for t in range(len(numel)):
            assert_bits_equal(dev[r][t].cpu().numpy(), want[r][t], f"rank {r} tensor {t}")


FUSED_CASES = [
    # (numel list, nranks, buffer dtype, align bytes)
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 3, np.float32, 16),
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, np.float32, 16),
    ([1] * 3000 + [5000], 5, np.float32, 16),  # many tensors per tile
    ([33, 31, 1, 2, 3, 4, 5, 6, 7, 8, 9, 100000], 7, np.float32, 4),  # no padding: vectors cross chunk ends
    ([257] * 40 + [70000, 3, 9000], 6, np.float16, 16),  # binary16 buffer
    ([1, 0, 2], 8, np.float32, 16),  # fewer buffer elements than ranks: empty chunks
    ([3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9], 13, np.float16, 2),
    ([5000, 300, 70000], 128, np.float32, 16),  # the most ranks a call takes
    ([5000, 300, 70001], 128, np.float16, 2),
]


@pytest.mark.parametrize("misalign", [False, True], ids=["aligned", "misaligned"])
@pytest.mark.parametrize("case", range(len(FUSED_CASES)))
def test_copy_kernels_fused_with_ring_steps(case, misalign):
    """hvdx_fuse_pack_rs leaves the buffers as the copy-in and adding step 0 do;
    hvdx_fuse_ag_unpack, started from the state before replacing step N-2, gives every
    tensor what that step and the copy-out give it, and writes no buffer."""
    numel, n, buf_np, align = FUSED_CASES[case]
    rng = np.random.default_rng(400 + case)
    host, dev, keep = make_tensors(rng, n, numel, np.float32, misalign)
    (b,) = fusion.fuse_plan(numel, np.dtype(buf_np).itemsize, threshold=1 << 30, align=align)
    say(f"fused copy case={case} misalign={misalign} count={b.count} n={n}")
    hv_buf = NP_TO_HV[np.dtype(buf_np)]
    ptrs, nm, off = descriptors(dev, b, numel)
    bufs = [torch.full((b.count + 64,), 7.0, dtype=NP_TO_TORCH[np.dtype(buf_np)], device="cuda") for _ in range(n)]
    st = torch.cuda.current_stream().cuda_stream
    hv.hvdx_fuse_pack_rs(ptrs.data_ptr(), nm.data_ptr(), off.data_ptr(), len(b.tensors), hv.FLOAT32,
                         [x.data_ptr() for x in bufs], b.count, hv_buf, n, st)
    torch.cuda.synchronize()

    states = {}
    work = np.stack([fusion.pack(host[r], b, buf_np) for r in range(n)])
    ring.ring_allreduce(work, "average", observe=lambda ph, s_, x: states.__setitem__((ph, s_), x.copy()))
    got = np.stack([x.cpu().numpy() for x in bufs])
    assert_bits_equal(got[:, : b.count], states[("rs", 0)], "copy-in + adding step 0")
    assert np.all(got[:, b.count :] == 7.0), "wrote past the buffer"

    before = states[("ag", n - 3)]
    for r in range(n):
        bufs[r][: b.count].copy_(torch.from_numpy(before[r]))
        for x in dev[r]:
            x.fill_(-3.0)
    torch.cuda.synchronize()
    hv.hvdx_fuse_ag_unpack([x.data_ptr() for x in bufs], b.count, hv_buf, ptrs.data_ptr(), nm.data_ptr(),
                           off.data_ptr(), len(b.tensors), hv.FLOAT32, n, st)
    torch.cuda.synchronize()
    final = states[("ag", n - 2)]
    for r in range(n):
        want = fusion.unpack(final[r], b, numel, np.float32)
        for t in b.tensors:
            assert_bits_equal(dev[r][t].cpu().numpy(), want[t], f"rank {r} tensor {t}")
        assert_bits_equal(bufs[r][: b.count].cpu().numpy(), before[r], f"buffer of rank {r}")



BINARY16_CASES = [
    # (numel, nranks, threshold bytes, op): binary16 tensors and buffers, no compression
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, 64 << 20, "average"),
    ([3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9], 6, 40000, "average"),  # buckets and direct tensors
    ([5000, 300, 70001, 9, 2048 * 3 + 5], 13, 16384, "sum"),
    ([5000, 300, 70000, 9], 128, 20000, "average"),
]


@pytest.mark.parametrize("mode", ["tensors", "tensors-misaligned", "copy-in", "buffers", "lookup"])
@pytest.mark.parametrize("case", range(len(BINARY16_CASES)))
def test_binary16_tensors_every_mode(case, mode):
    """binary16 gradients (binary16 buffers, no compression) through each way of running
    the fused buckets: the ring on the tensors (aligned, and at odd element offsets: the
    element paths), the copy-in kept, the ring in the buffers, the searching copies."""
    numel, n, threshold, op = BINARY16_CASES[case]
    rng = np.random.default_rng(700 + case)
    host, dev, keep = make_tensors(rng, n, numel, np.float16, misalign=mode == "tensors-misaligned")
    say(f"binary16 tensors case={case} n={n} mode={mode}")
    ar = hv.FusedAllreduce(dev, op=op, threshold_bytes=threshold, small_bucket_bytes=0, tiled=mode != "lookup",
                           replace_in_tensors=mode not in ("buffers", "lookup"),
                           add_from_tensors=mode in ("tensors", "tensors-misaligned"))
    want = allreduce.allreduce(host, op, threshold=threshold)
    for rep in range(2):  # the second call reduces the first's result again
        ar()
        torch.cuda.synchronize()
        for r in range(n):
            for t in range(len(numel)):
                assert_bits_equal(dev[r][t].cpu().numpy(), want[r][t], f"call {rep} rank {r} tensor {t}")
        want = allreduce.allreduce(want, op, threshold=threshold)
