"""Two fusion buffers' cycles with each ring step of both in one launch
(hvdx_fuse_allreduce_pair, used by FusedAllreduce for fused buckets paired in plan
order, also across a direct tensor between them):
bit for bit the oracle's result, and the same as running the buckets one by one."""
import numpy as np
import pytest
import torch

import paper_1802_05799_amd as hv
from _gpu import assert_bits_equal, say
from oracle import allreduce, fusion

pytestmark = pytest.mark.gpu

CASES = [
    # (numel, nranks, threshold bytes, compress, op, the pairs FusedAllreduce forms)
    # buckets [0,1] [2,3] [4,5] fused, [6] direct, [7] fused: the second pair spans the direct tensor
    ([6000, 3000, 7001, 2500, 9000, 40, 12000, 333], 5, 40000, False, "average", [(0, 1), (2, 4)]),
    # binary16 buffers: three fused buckets, the last alone
    ([6000, 3000, 7001, 2500, 9000, 40, 12000, 333], 8, 40000, True, "sum", [(0, 1)]),
    ([3, 5], 8, 32, False, "average", [(0, 1)]),  # both rings shorter than the rank count
    # three ranks (no plain ring step): fused, fused, direct, fused (alone)
    ([1000, 1, 1500, 70000, 513, 700], 3, 8192, False, "sum", [(0, 1)]),
    ([2048] * 5 + [100], 13, 16384, False, "average", [(0, 1)]),  # a pair, the last bucket alone
    ([100003, 31, 64000, 7], 4, 256 << 10, True, "average", [(0, 1)]),  # rings of very different lengths
    # the most ranks a call takes (full rank-pointer tables in the kernel argument):
    # fused [0,1,2] and [3] paired, [4] direct, [5] alone; binary32 and binary16 buffers
    ([3000, 5000, 257, 9000, 70000, 4100], 128, 40000, False, "average", [(0, 1)]),
    ([3000, 5000, 257, 9000, 70000, 4100], 128, 20000, True, "average", [(0, 1)]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_pairs_match_oracle_and_single_cycles(case):
    numel, n, threshold, compress, op, pairs = CASES[case]
    say(f"pair case {case}: N={n} numel={numel[:4]}... threshold={threshold} compress={compress} {op}")
    rng = np.random.default_rng(4200 + case)
    host = [[(rng.standard_normal(k) * 0.01).astype(np.float32) for k in numel] for _ in range(n)]
    want1 = allreduce.allreduce(host, op, compress=compress, threshold=threshold)
    want2 = allreduce.allreduce(want1, op, compress=compress, threshold=threshold)
    for pair, tiled, into, add in ((True, True, True, True), (False, True, True, True), (True, True, True, False),
                                   (False, True, True, False), (True, True, False, False), (False, True, False, False),
                                   (True, False, False, False), (False, False, False, False)):
        dev = [[torch.from_numpy(x).cuda() for x in row] for row in host]
        ar = hv.FusedAllreduce(dev, op=op, compress=compress, threshold_bytes=threshold, small_bucket_bytes=0,
                               pair_buckets=pair, tiled=tiled, replace_in_tensors=into, add_from_tensors=add)
        want_flags = hv.TILED_REPLACE_IN_TENSORS | (hv.TILED_ADD_FROM_TENSORS * add) if into else 0
        assert ar.tiled_flags == want_flags
        # groups of up to four with the ring on the tensors (two at 128 ranks), else pairs
        size = min(hv.TILED_MAX_BUCKETS, hv.TILED_MAX_BUFFERS // n) if want_flags & hv.TILED_ADD_FROM_TENSORS else 2
        per_step = sorted({i for p in pairs for i in p} | {i for i, b in enumerate(fusion.fuse_plan(
            numel, 2 if compress else 4, threshold)) if not b.direct and b.count > 0})
        want_groups = [tuple(per_step[g : g + size]) for g in range(0, len(per_step), size)] if pair else []
        want_groups = [g for g in want_groups if len(g) > 1]
        assert ar.groups == want_groups
        if size == 2 and pair:
            assert want_groups == pairs
        for rep, want in enumerate((want1, want2)):  # the second call reduces the first's result again
            ar()
            torch.cuda.synchronize()
            for r in range(n):
                for t in range(len(numel)):
                    assert_bits_equal(dev[r][t].cpu().numpy(), want[r][t],
                                      f"pair={pair} tiled={tiled} flags={want_flags} call {rep} rank {r} t {t}")


def test_pair_entry_point_directly():
    """The C entry point on two hand-built buckets of one rank set, against the
    oracle, with a bucket of count 0 as the degenerate partner."""
    n = 6
    say("pair entry point: two buckets and an empty partner")
    rng = np.random.default_rng(77)
    numel = [[4001, 17], [2999]]
    per_rank = [[(rng.standard_normal(k) * 0.01).astype(np.float32) for ks in numel for k in ks] for _ in range(n)]
    dev = [[torch.from_numpy(x).cuda() for x in row] for row in per_rank]
    descs, keep = [], []
    t0 = 0
    for ks in numel:
        offs, count = [], 0
        for k in ks:
            start = (count + 3) // 4 * 4
            offs.append(start)
            count = start + k
        idx = list(range(t0, t0 + len(ks)))
        t0 += len(ks)
        bufs = [torch.full((count,), float("nan"), device="cuda") for _ in range(n)]
        ptrs = torch.tensor([dev[r][t].data_ptr() for r in range(n) for t in idx], dtype=torch.int64, device="cuda")
        nm = torch.tensor(ks, dtype=torch.int64, device="cuda")
        off = torch.tensor(offs, dtype=torch.int64, device="cuda")
        keep += [bufs, ptrs, nm, off]
        descs.append((ptrs.data_ptr(), nm.data_ptr(), off.data_ptr(), len(ks), [b.data_ptr() for b in bufs], count))
    stream = torch.cuda.current_stream().cuda_stream
    hv.hvdx_fuse_allreduce_pair(descs[0], descs[1], hv.FLOAT32, hv.FLOAT32, n, hv.AVERAGE, stream)
    torch.cuda.synchronize()
    # each bucket alone, as the oracle's plan would form it (threshold large enough for one bucket each)
    want = [[None] * 3 for _ in range(n)]
    for ids in ([0, 1], [2]):
        sub = [[per_rank[r][t] for t in ids] for r in range(n)]
        got = allreduce.allreduce(sub, "average", threshold=1 << 30)
        for r in range(n):
            for j, t in enumerate(ids):
                want[r][t] = got[r][j]
    for r in range(n):
        for t in range(3):
            assert_bits_equal(dev[r][t].cpu().numpy(), want[r][t], f"rank {r} t {t}")
    # a partner with nothing to reduce: the other bucket runs alone
    empty = (descs[1][0], descs[1][1], descs[1][2], 1, descs[1][4], 0)
    before = [[x.cpu().numpy().copy() for x in row] for row in dev]
    hv.hvdx_fuse_allreduce_pair(descs[0], empty, hv.FLOAT32, hv.FLOAT32, n, hv.SUM, stream)
    torch.cuda.synchronize()
    sub = [[before[r][t] for t in (0, 1)] for r in range(n)]
    got = allreduce.allreduce(sub, "sum", threshold=1 << 30)
    for r in range(n):
        for t in (0, 1):
            assert_bits_equal(dev[r][t].cpu().numpy(), got[r][t], f"empty partner: rank {r} t {t}")
        assert_bits_equal(dev[r][2].cpu().numpy(), before[r][2], f"empty partner untouched: rank {r}")


def test_small_bucket_rides_along_with_a_lone_one():
    """Buckets 0 (tensors 0, 1), 1 (tensor 2) and 4 (tensor 5) on the per-step path, 2
    (tensor 3: 400 bytes per rank) small, 3 (tensor 4) direct: the group of three takes
    bucket 2 along instead of bucket 2 running its own launch."""
    numel = [9000, 7000, 16384, 100, 20000, 15000]
    n = 6
    rng = np.random.default_rng(4300)
    host = [[(rng.standard_normal(k) * 0.01).astype(np.float32) for k in numel] for _ in range(n)]
    for op in ("average", "sum"):
        say(f"small bucket riding along: {op}")
        want = allreduce.allreduce(host, op, threshold=65536)
        dev = [[torch.from_numpy(x).cuda() for x in row] for row in host]
        ar = hv.FusedAllreduce(dev, op=op, threshold_bytes=65536, small_bucket_bytes=4096)
        assert ar.groups == [(0, 1, 2, 4)]
        assert not any(k == "cycle_small" for k, _, _ in ar.kernel_sequence())
        ar()
        torch.cuda.synchronize()
        for r in range(n):
            for t in range(len(numel)):
                assert_bits_equal(dev[r][t].cpu().numpy(), want[r][t], f"{op} rank {r} t {t}")
