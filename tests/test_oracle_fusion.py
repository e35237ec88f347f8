"""Pins of the oracle's Tensor Fusion (paper section 7) and the composed allreduce."""
import numpy as np
import pytest

import _pins
from oracle import allreduce, fusion, ring
from workloads import configs

MiB64 = 64 << 20


def check_plan_invariants(numel, esize, plan, threshold=MiB64, align=16):
    """The greedy contiguous plan is the unique plan with these properties."""
    seen = []
    for b in plan:
        seen += b.tensors
        if b.direct:
            (t,) = b.tensors
            assert numel[t] * esize > threshold and b.offsets == [0] and b.count == numel[t]
            continue
        end = 0
        for t, off in zip(b.tensors, b.offsets):
            assert numel[t] * esize <= threshold
            assert off * esize % align == 0  # aligned
            assert off >= end  # non-overlapping, in order
            assert off * esize - end * esize < align  # the nearest aligned offset
            end = off + numel[t]
        assert b.count == end
        assert b.count * esize <= threshold  # fits
    assert seen == list(range(len(numel)))  # ready order, nothing skipped or repeated
    # maximal: a bucket closes only when the next tensor is direct or does not fit
    for b, nxt in zip(plan, plan[1:]):
        if b.direct or nxt.direct:
            continue
        t = nxt.tensors[0]
        start = -(-b.count * esize // align) * align
        assert start + numel[t] * esize > threshold


@pytest.mark.parametrize("name", list(configs.WORKLOADS))
def test_plan_invariants_on_workloads(name):
    w = configs.get(name)
    es = 2 if w.compress else 4
    plan = fusion.fuse_plan(w.numel(), es)
    check_plan_invariants(w.numel(), es, plan)
    assert sum(sum(w.numel()[t] for t in b.tensors) for b in plan) == sum(w.numel())


def test_plan_invariants_random_lists():
    rng = np.random.default_rng(21)
    for trial in range(300):
        numel = list(rng.integers(0, 40, size=rng.integers(0, 30)))
        if trial % 3 == 0:
            numel += [int(rng.integers(0, 200))]
        esize = int(rng.choice([2, 4]))
        align = int(rng.choice([esize, 8, 16, 64]))
        threshold = int(rng.integers(0, 160))
        plan = fusion.fuse_plan(numel, esize, threshold, align)
        check_plan_invariants(numel, esize, plan, threshold, align)


def test_plan_tie_fits_and_oversize_is_direct():
    # exactly the threshold fits (VGG-16's fc7 gradient is 4096*4096*4 B = 64 MiB)
    plan = fusion.fuse_plan([4096 * 4096], 4)
    assert len(plan) == 1 and not plan[0].direct
    plan = fusion.fuse_plan([4096 * 4096 + 1], 4)
    assert plan[0].direct
    # after a 1-element tensor the next one must start at byte 16
    plan = fusion.fuse_plan([1, (MiB64 - 16) // 4], 4)
    assert len(plan) == 1 and plan[0].offsets == [0, 4]
    plan = fusion.fuse_plan([1, (MiB64 - 12) // 4], 4)
    assert len(plan) == 2
    with pytest.raises(ValueError):
        fusion.fuse_plan([1], 4, align=12)
    with pytest.raises(ValueError):
        fusion.fuse_plan([1], 4, align=2)


def test_expected_bucket_layouts():
    """Reading R5-R8 applied to the five workloads (tests/golden/plans.txt, written by
    tests/golden/make_plans.py from the oracle, checked here and against the GPU library)."""
    rows = {}
    with open(_pins.GOLDEN + "/plans.txt") as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                rows.setdefault(line[0], []).append(tuple(int(v) for v in line[1:]))
    for name, w in configs.WORKLOADS.items():
        plan = fusion.fuse_plan(w.numel(), 2 if w.compress else 4)
        assert [(b.count, len(b.tensors), int(b.direct)) for b in plan] == rows[name]
    # the counts quoted for these layouts when the workloads were specified
    assert rows["tiny"] == [(20391, 8, 0)]
    assert [r[0] for r in rows["vgg16fp16"]] == [20882408, 102760448, 14714688]


def test_pack_places_every_tensor_and_zero_pads():
    numel = [3, 5, 1, 8, 2]
    plan = fusion.fuse_plan(numel, 4, threshold=1 << 20)
    (b,) = plan
    xs = [np.arange(n, dtype=np.float32) + 100 * (t + 1) for t, n in enumerate(numel)]
    buf = fusion.pack(xs, b, np.float32)
    mask = np.zeros(b.count, bool)
    for t, off in zip(b.tensors, b.offsets):
        assert np.array_equal(buf[off : off + numel[t]], xs[t])
        mask[off : off + numel[t]] = True
    assert np.all(buf[~mask] == 0)
    assert b.offsets == [0, 4, 12, 16, 24] and b.count == 26
    back = fusion.unpack(buf, b, numel, np.float32)
    assert all(np.array_equal(u, x) for u, x in zip(back, xs))
    tensor, local = fusion.buffer_origin(b, numel, np.arange(b.count))
    for e in range(b.count):
        if tensor[e] >= 0:
            assert buf[e] == xs[tensor[e]][local[e]]
        else:
            assert not mask[e]


def test_single_rank_allreduce_is_identity_and_cast_roundtrip():
    rng = np.random.default_rng(22)
    xs = [[(rng.standard_normal(n) * 0.01).astype(np.float32) for n in (5, 17, 1, 300)]]
    for op in ("sum", "average"):
        out = allreduce.allreduce(xs, op, threshold=256)
        assert all(_pins.bits_equal(a, b) for a, b in zip(out[0], xs[0]))
        outc = allreduce.allreduce(xs, op, compress=True, threshold=256)
        assert all(_pins.bits_equal(a, b.astype(np.float16).astype(np.float32)) for a, b in zip(outc[0], xs[0]))


def _tensor_allreduce_reference(per_rank, op, compress):
    """Each tensor reduced on its own by the mailbox simulation (no fusion)."""
    n = len(per_rank)
    out = [[None] * len(per_rank[0]) for _ in range(n)]
    for t in range(len(per_rank[0])):
        x = [np.asarray(per_rank[r][t]).reshape(-1) for r in range(n)]
        if compress:
            x = [v.astype(np.float16) for v in x]
        res = _pins.mailbox_allreduce(x, op)
        for r in range(n):
            out[r][t] = res[r].astype(np.float32)
    return out


def test_fusion_only_changes_chunking_exact_integers():
    """With integer-valued gradients every order and chunking gives the exact sum, so
    the fused result must equal per-tensor mailbox allreduces, whatever the buckets."""
    rng = np.random.default_rng(23)
    for compress in (False, True):
        for n in (1, 2, 3, 4, 8):
            numel = [7, 64, 100, 33, 1000, 1]
            per_rank = [[rng.integers(-30, 31, size=k).astype(np.float32) for k in numel] for _ in range(n)]
            for threshold in (64, 400, 4096, MiB64):
                out = allreduce.allreduce(per_rank, "sum", compress=compress, threshold=threshold)
                ref = _tensor_allreduce_reference(per_rank, "sum", compress)
                for r in range(n):
                    for t in range(len(numel)):
                        assert _pins.bits_equal(out[r][t], ref[r][t]), (compress, n, threshold, r, t)


def test_tiny_workload_checks_1_to_4():
    """The tiny workload in full: identical ranks, fp64 bound, traffic, and the same
    buffer through the mailbox brute force."""
    from workloads import rng as wrng

    w = configs.get("tiny")
    n = w.nranks
    numel = w.numel()
    prefix = w.prefix()
    per_rank = [[wrng.uniform(w.key(r), np.arange(p, p + k)) for p, k in zip(prefix, numel)] for r in range(n)]
    traffic = {}
    out = allreduce.allreduce(per_rank, "average", traffic=traffic)
    flat = [np.concatenate(o) for o in out]
    assert all(_pins.bits_equal(f, flat[0]) for f in flat)
    x = np.stack([np.concatenate(p) for p in per_rank]).astype(np.float64)
    ref = x.sum(axis=0) / n
    absum = np.abs(x).sum(axis=0) / n
    assert np.all(np.abs(flat[0] - ref) <= 1e-6 * n * absum)
    (b,) = fusion.fuse_plan(numel, 4)
    assert b.count == 20391
    tr = traffic[0]
    _, sizes = ring.chunk_bounds(b.count, n)
    assert int(tr["sent"].sum()) == 2 * (n - 1) * b.count
    for r in range(n):
        assert tr["sent"][r] == 2 * b.count - sizes[(r + 1) % n] - sizes[(r + 2) % n]
    bufs = [fusion.pack(per_rank[r], b, np.float32) for r in range(n)]
    mb = _pins.mailbox_allreduce(bufs, "average")
    for r in range(n):
        assert all(_pins.bits_equal(a, b2) for a, b2 in zip(fusion.unpack(mb[r], b, numel, np.float32), out[r]))


def test_ring_columns_matches_whole_allreduce():
    rng = np.random.default_rng(24)
    n = 5
    numel = [13, 200, 1, 77, 40]
    per_rank = [[(rng.standard_normal(k) * 0.01).astype(np.float32) for k in numel] for _ in range(n)]
    for compress in (False, True):
        plan = fusion.fuse_plan(numel, 2 if compress else 4, threshold=512)
        out = allreduce.allreduce(per_rank, "average", compress=compress, threshold=512)
        for b in plan:
            elems = np.sort(rng.choice(b.count, size=max(1, b.count // 2), replace=False))
            vals, tensor, local = allreduce.ring_columns(
                b, numel, elems, lambda r, t, i: per_rank[r][t][i], n, "average", compress
            )
            for j in range(len(elems)):
                if tensor[j] >= 0:
                    for r in range(n):
                        assert vals[r, j].view(np.uint32) == out[r][tensor[j]][local[j]].view(np.uint32)
