"""The C-ABI without a GPU: exported symbols, host-only entry points against the
oracle, and argument checks (which return before any HIP call)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_1802_05799_amd as hv
from oracle import fusion, ring
from workloads import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7F0000000000  # a plausible device address; never dereferenced by these calls


def declared_symbols():
    with open(os.path.join(ROOT, "include", "hvdx.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hvdx_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    syms = declared_symbols()
    assert len(syms) >= 10
    lib = ctypes.CDLL(hv.LIB_PATH)
    for s in syms:
        assert hasattr(lib, s), s


def test_version_and_strerror():
    assert hv.hvdx_version() == 1
    for code in (hv.OK, hv.ERR_INVALID, hv.ERR_ALIAS, hv.ERR_WORKSPACE, hv.ERR_HIP, hv.ERR_UNSUPPORTED):
        assert hv.hvdx_strerror(code) and hv.hvdx_strerror(code) != "unknown status"
    assert hv.hvdx_strerror(12345) == "unknown status"


def plan_as_buckets(numel, buf_dtype, threshold, align):
    bucket_of, offset, counts, direct = hv.hvdx_fuse_plan(numel, buf_dtype, threshold, align)
    out = [([], [], c, bool(d)) for c, d in zip(counts, direct)]
    for t, (b, o) in enumerate(zip(bucket_of, offset)):
        out[b][0].append(t)
        out[b][1].append(o)
    return out


def oracle_buckets(numel, esize, threshold, align):
    return [(b.tensors, b.offsets, b.count, b.direct) for b in fusion.fuse_plan(numel, esize, threshold, align)]


@pytest.mark.parametrize("name", list(configs.WORKLOADS))
def test_plan_matches_oracle_on_workloads(name):
    w = configs.get(name)
    dt, es = (hv.FLOAT16, 2) if w.compress else (hv.FLOAT32, 4)
    assert plan_as_buckets(w.numel(), dt, 64 << 20, 16) == oracle_buckets(w.numel(), es, 64 << 20, 16)


def test_plan_matches_oracle_on_random_lists():
    rng = np.random.default_rng(31)
    for _ in range(500):
        numel = [int(v) for v in rng.integers(0, 60, size=rng.integers(0, 40))]
        dt, es = [(hv.FLOAT32, 4), (hv.FLOAT16, 2)][int(rng.integers(0, 2))]
        align = int(rng.choice([es, 8, 16, 32, 256]))
        threshold = int(rng.integers(0, 300))
        assert plan_as_buckets(numel, dt, threshold, align) == oracle_buckets(numel, es, threshold, align)


def test_ring_chunk_matches_oracle():
    for n in (1, 2, 3, 7, 64, 128):
        for count in (0, 1, n - 1, n, 20391, 102760448, 2**40 + 3):
            starts, lengths = ring.chunk_bounds(count, n)
            for c in range(n):
                assert hv.hvdx_ring_chunk(count, n, c) == (starts[c], lengths[c])


def test_workspace_bytes():
    assert hv.hvdx_ring_workspace_bytes(64, 102760448, hv.FLOAT32, hv.COMPRESS_FP16) == 64 * 102760448 * 2
    assert hv.hvdx_ring_workspace_bytes(4, 130, hv.FLOAT32, hv.COMPRESS_FP16) == 4 * 256 * 2
    assert hv.hvdx_ring_workspace_bytes(4, 130, hv.FLOAT32, hv.COMPRESS_NONE) == 0
    assert hv.hvdx_ring_workspace_bytes(1, 130, hv.FLOAT32, hv.COMPRESS_FP16) == 0
    assert hv.hvdx_ring_workspace_bytes(4, 0, hv.FLOAT32, hv.COMPRESS_FP16) == 0


def status_of(fn, *args):
    """Status of a call that must be refused by the argument checks (or be a no-op):
    these calls use fake device addresses and must never reach a kernel launch."""
    try:
        fn(*args)
    except hv.HvdxError as e:
        return e.status
    return hv.OK


def bufs(n, count, esize=4, stride=None):
    stride = stride if stride is not None else ((count * esize + 255) // 256) * 256 + 256
    return [FAKE + r * stride for r in range(n)]


def test_ring_argument_errors():
    ar = hv.hvdx_ring_allreduce
    assert status_of(ar, bufs(2, 8), 0, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # nranks 0
    assert status_of(ar, bufs(129, 8), 129, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # too many ranks
    assert status_of(ar, bufs(2, 8), 2, -1, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # negative count
    assert status_of(ar, bufs(2, 8), 2, 1 << 62, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # byte extents overflow
    assert status_of(ar, bufs(2, 8), 2, 8, 7, hv.SUM) == hv.ERR_INVALID  # dtype
    assert status_of(ar, bufs(2, 8), 2, 8, hv.FLOAT32, 9) == hv.ERR_INVALID  # op
    assert status_of(ar, bufs(2, 8), 2, 8, hv.FLOAT32, hv.SUM, 5) == hv.ERR_INVALID  # compression
    assert status_of(ar, bufs(2, 8), 2, 8, hv.FLOAT16, hv.SUM, hv.COMPRESS_FP16) == hv.ERR_INVALID
    assert status_of(ar, [FAKE, 0], 2, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # null buffer
    assert status_of(ar, [FAKE, FAKE + 2], 2, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # misaligned
    assert status_of(ar, [FAKE, FAKE + 16], 2, 8, hv.FLOAT32, hv.SUM) == hv.ERR_ALIAS  # overlap
    assert status_of(ar, [FAKE + 64, FAKE, FAKE + 32], 3, 9, hv.FLOAT32, hv.SUM) == hv.ERR_ALIAS
    # compression needs a large enough, aligned, disjoint workspace
    b = bufs(4, 1000)
    need = hv.hvdx_ring_workspace_bytes(4, 1000, hv.FLOAT32, hv.COMPRESS_FP16)
    ws = FAKE + (1 << 30)
    assert status_of(ar, b, 4, 1000, hv.FLOAT32, hv.AVERAGE, hv.COMPRESS_FP16, 0, 0) == hv.ERR_WORKSPACE
    assert status_of(ar, b, 4, 1000, hv.FLOAT32, hv.AVERAGE, hv.COMPRESS_FP16, ws, need - 1) == hv.ERR_WORKSPACE
    assert status_of(ar, b, 4, 1000, hv.FLOAT32, hv.AVERAGE, hv.COMPRESS_FP16, ws + 16, need) == hv.ERR_WORKSPACE
    assert status_of(ar, b, 4, 1000, hv.FLOAT32, hv.AVERAGE, hv.COMPRESS_FP16, b[1], need) == hv.ERR_ALIAS
    # count 0 is a no-op and touches nothing
    assert status_of(ar, bufs(4, 0), 4, 0, hv.FLOAT32, hv.AVERAGE) == hv.OK
    st = hv.hvdx_ring_step
    assert status_of(st, bufs(3, 8), 3, 8, hv.FLOAT32, hv.SUM, 0, 2, 0) == hv.ERR_INVALID  # phase
    assert status_of(st, bufs(3, 8), 3, 8, hv.FLOAT32, hv.SUM, 0, 0, 2) == hv.ERR_INVALID  # step > N-2
    assert status_of(st, bufs(3, 8), 3, 8, hv.FLOAT32, hv.SUM, 0, 0, -1) == hv.ERR_INVALID
    assert status_of(st, bufs(1, 8), 1, 8, hv.FLOAT32, hv.SUM, 0, 0, 0) == hv.ERR_INVALID  # no steps at N=1
    assert "overlap" in hv.hvdx_last_error() or hv.hvdx_last_error()


def test_fusion_argument_errors():
    pk, up = hv.hvdx_fuse_pack, hv.hvdx_fuse_unpack
    b = bufs(2, 64)
    assert status_of(pk, 0, FAKE, FAKE, 3, hv.FLOAT32, b, 64, hv.FLOAT32, 2) == hv.ERR_INVALID
    assert status_of(pk, FAKE, FAKE, FAKE, -1, hv.FLOAT32, b, 64, hv.FLOAT32, 2) == hv.ERR_INVALID
    assert status_of(pk, FAKE, FAKE, FAKE, 3, hv.FLOAT16, b, 64, hv.FLOAT32, 2) == hv.ERR_UNSUPPORTED
    assert status_of(pk, FAKE, FAKE, FAKE, 3, 5, b, 64, hv.FLOAT32, 2) == hv.ERR_INVALID
    assert status_of(pk, FAKE, FAKE, FAKE, 3, hv.FLOAT32, [FAKE, FAKE + 64], 64, hv.FLOAT32, 2) == hv.ERR_ALIAS
    assert status_of(pk, FAKE, FAKE, FAKE, 3, hv.FLOAT32, [FAKE + 4, FAKE + 4096], 64, hv.FLOAT32, 2) == hv.ERR_INVALID
    assert status_of(up, b, 64, hv.FLOAT32, 0, FAKE, FAKE, 3, hv.FLOAT32, 2) == hv.ERR_INVALID
    assert status_of(up, b, -5, hv.FLOAT32, FAKE, FAKE, FAKE, 3, hv.FLOAT32, 2) == hv.ERR_INVALID
    assert status_of(up, b, 64, hv.FLOAT32, FAKE, FAKE, FAKE, 3, hv.FLOAT32, 0) == hv.ERR_INVALID
    # an empty buffer is a no-op
    assert status_of(pk, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b, 0, hv.FLOAT32, 2) == hv.OK


def test_fused_boundary_argument_errors():
    pr, au, fa = hv.hvdx_fuse_pack_rs, hv.hvdx_fuse_ag_unpack, hv.hvdx_fuse_allreduce
    b2, b3 = bufs(2, 64), bufs(3, 64)
    # the fused copy kernels need a first adding step that is not the last one
    assert status_of(pr, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b2, 64, hv.FLOAT32, 2) == hv.ERR_UNSUPPORTED
    assert status_of(au, b2, 64, hv.FLOAT32, FAKE, FAKE, FAKE, 3, hv.FLOAT32, 2) == hv.ERR_UNSUPPORTED
    assert status_of(pr, 0, FAKE, FAKE, 3, hv.FLOAT32, b3, 64, hv.FLOAT32, 3) == hv.ERR_INVALID
    assert status_of(au, b3, 64, hv.FLOAT32, 0, FAKE, FAKE, 3, hv.FLOAT32, 3) == hv.ERR_INVALID
    assert status_of(fa, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b3, 64, hv.FLOAT32, 3, 7) == hv.ERR_INVALID  # op
    assert status_of(fa, 0, FAKE, FAKE, 3, hv.FLOAT32, b3, 64, hv.FLOAT32, 3, hv.SUM) == hv.ERR_INVALID
    assert status_of(fa, FAKE, FAKE, FAKE, 3, hv.FLOAT16, b3, 64, hv.FLOAT32, 3, hv.SUM) == hv.ERR_UNSUPPORTED
    assert status_of(fa, FAKE, FAKE, FAKE, 3, hv.FLOAT32, [FAKE, FAKE + 64, FAKE + 4096], 64, hv.FLOAT32, 3,
                     hv.SUM) == hv.ERR_ALIAS
    # empty buffers are a no-op
    assert status_of(pr, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b3, 0, hv.FLOAT32, 3) == hv.OK
    assert status_of(au, b3, 0, hv.FLOAT32, FAKE, FAKE, FAKE, 3, hv.FLOAT32, 3) == hv.OK
    assert status_of(fa, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b3, 0, hv.FLOAT32, 3, hv.AVERAGE) == hv.OK


def test_plan_argument_errors():
    with pytest.raises(hv.HvdxError):
        hv.hvdx_fuse_plan([1, -2], hv.FLOAT32)
    with pytest.raises(hv.HvdxError):
        hv.hvdx_fuse_plan([1], hv.FLOAT32, 64, 12)
    with pytest.raises(hv.HvdxError):
        hv.hvdx_fuse_plan([1], hv.FLOAT32, 64, 2)
    with pytest.raises(hv.HvdxError):
        hv.hvdx_fuse_plan([1], 3)
    with pytest.raises(hv.HvdxError):
        hv.hvdx_fuse_plan([1], hv.FLOAT32, -1)
    assert hv.hvdx_fuse_plan([], hv.FLOAT32) == ([], [], [], [])


def test_broadcast_argument_errors():
    bc = hv.hvdx_broadcast
    assert status_of(bc, bufs(3, 64), 3, 64, 3) == hv.ERR_INVALID  # root out of range
    assert status_of(bc, bufs(3, 64), 3, 64, -1) == hv.ERR_INVALID
    assert status_of(bc, bufs(3, 64), 3, -1, 0) == hv.ERR_INVALID
    assert status_of(bc, [FAKE, FAKE + 32, FAKE + 4096], 3, 64, 0) == hv.ERR_ALIAS
    assert status_of(bc, bufs(3, 64), 0, 64, 0) == hv.ERR_INVALID
    assert status_of(bc, bufs(3, 0), 3, 0, 1) == hv.OK  # nothing to copy
    st = hv.hvdx_broadcast_step
    assert status_of(st, bufs(3, 64), 3, 64, 0, 4) == hv.ERR_INVALID  # steps are 0..2N-3
    assert status_of(st, bufs(1, 64), 1, 64, 0, 0) == hv.ERR_INVALID  # no steps with one rank


def test_fold_argument_errors():
    fo = hv.hvdx_fold_allreduce
    assert status_of(fo, bufs(2, 8), 0, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID
    assert status_of(fo, bufs(2, 8), 2, 8, hv.FLOAT16, hv.SUM, hv.COMPRESS_FP16) == hv.ERR_INVALID
    assert status_of(fo, bufs(2, 8), 2, 8, hv.FLOAT32, hv.SUM, 7) == hv.ERR_INVALID
    assert status_of(fo, [FAKE, FAKE + 16], 2, 8, hv.FLOAT32, hv.SUM) == hv.ERR_ALIAS
    assert status_of(fo, bufs(2, 0), 2, 0, hv.FLOAT32, hv.AVERAGE) == hv.OK


def test_small_path_argument_errors():
    rs, fs = hv.hvdx_ring_allreduce_small, hv.hvdx_fuse_allreduce_small
    assert status_of(rs, bufs(2, 8), 0, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # nranks 0
    assert status_of(rs, bufs(2, 8), 2, -1, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID
    assert status_of(rs, bufs(2, 8), 2, 8, 7, hv.SUM) == hv.ERR_INVALID  # dtype
    assert status_of(rs, bufs(2, 8), 2, 8, hv.FLOAT32, 9) == hv.ERR_INVALID  # op
    assert status_of(rs, [FAKE, FAKE + 16], 2, 8, hv.FLOAT32, hv.SUM) == hv.ERR_ALIAS
    assert status_of(rs, [FAKE, FAKE + 2], 2, 8, hv.FLOAT32, hv.SUM) == hv.ERR_INVALID  # misaligned
    assert status_of(rs, bufs(4, 0), 4, 0, hv.FLOAT32, hv.AVERAGE) == hv.OK  # nothing to do
    assert status_of(rs, bufs(1, 8), 1, 8, hv.FLOAT32, hv.AVERAGE) == hv.OK  # one rank: no messages
    b3 = bufs(3, 64)
    assert status_of(fs, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b3, 64, hv.FLOAT32, 3, 7) == hv.ERR_INVALID  # op
    assert status_of(fs, 0, FAKE, FAKE, 3, hv.FLOAT32, b3, 64, hv.FLOAT32, 3, hv.SUM) == hv.ERR_INVALID
    assert status_of(fs, FAKE, FAKE, FAKE, 3, hv.FLOAT16, b3, 64, hv.FLOAT32, 3, hv.SUM) == hv.ERR_UNSUPPORTED
    assert status_of(fs, FAKE, FAKE, FAKE, 3, hv.FLOAT32, [FAKE, FAKE + 64, FAKE + 4096], 64, hv.FLOAT32, 3,
                     hv.SUM) == hv.ERR_ALIAS
    assert status_of(fs, FAKE, FAKE, FAKE, 3, hv.FLOAT32, [FAKE + 4, FAKE + 4096, FAKE + 8192], 64, hv.FLOAT32,
                     3, hv.SUM) == hv.ERR_INVALID  # fusion buffers must be 16-byte aligned
    assert status_of(fs, FAKE, FAKE, FAKE, 3, hv.FLOAT32, b3, 0, hv.FLOAT32, 3, hv.AVERAGE) == hv.OK


def test_pair_argument_errors():
    """hvdx_fuse_allreduce_pair refuses bad descriptors before any launch."""
    fp = hv.hvdx_fuse_allreduce_pair
    b3 = bufs(3, 64)
    c3 = [x + (1 << 24) for x in b3]  # the second bucket's fusion buffers, disjoint from the first's
    d0, d1 = (FAKE, FAKE, FAKE, 3, b3, 64), (FAKE, FAKE, FAKE, 2, c3, 40)
    assert status_of(fp, d0, d1, hv.FLOAT32, hv.FLOAT32, 3, 7) == hv.ERR_INVALID  # op
    assert status_of(fp, (FAKE, FAKE, FAKE, 3, b3[:2], 64), (FAKE, FAKE, FAKE, 2, c3[:2], 40), hv.FLOAT32,
                     hv.FLOAT32, 2, hv.SUM) == hv.ERR_UNSUPPORTED  # two ranks: no adding step before the last
    assert status_of(fp, (0, FAKE, FAKE, 3, b3, 64), d1, hv.FLOAT32, hv.FLOAT32, 3, hv.SUM) == hv.ERR_INVALID
    assert status_of(fp, d0, (FAKE, FAKE, FAKE, 2, c3, 40), hv.FLOAT16, hv.FLOAT32, 3,
                     hv.SUM) == hv.ERR_UNSUPPORTED  # binary16 tensors, binary32 buffers
    overlap = (FAKE, FAKE, FAKE, 2, [b3[1] + 64, c3[1], c3[2]], 40)  # inside rank 1's first buffer
    assert status_of(fp, d0, overlap, hv.FLOAT32, hv.FLOAT32, 3, hv.SUM) == hv.ERR_ALIAS
    assert status_of(fp, d0, (FAKE, FAKE, FAKE, 2, [c3[0], c3[1] + 8, c3[2]], 40), hv.FLOAT32, hv.FLOAT32, 3,
                     hv.SUM) == hv.ERR_INVALID  # fusion buffers must be 16-byte aligned
    lib = hv._lib.lib
    assert lib.hvdx_fuse_allreduce_pair(None, None, hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, None) == hv.ERR_INVALID


def test_tiled_argument_errors():
    """hvdx_fuse_allreduce_tiled refuses unknown flags, binary16 tensors with binary32
    buffers, and adding from the tensors alone, before any launch."""
    ft = hv.hvdx_fuse_allreduce_tiled
    b3 = bufs(3, 64)
    d0 = (FAKE, FAKE, FAKE, 3, b3, 64, FAKE, 4, FAKE, 4)
    both = hv.TILED_REPLACE_IN_TENSORS | hv.TILED_ADD_FROM_TENSORS
    assert status_of(ft, [d0], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, 4) == hv.ERR_INVALID
    assert status_of(ft, [d0], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, -1) == hv.ERR_INVALID
    for flags in (hv.TILED_REPLACE_IN_TENSORS, both):
        assert status_of(ft, [d0], hv.FLOAT16, hv.FLOAT32, 3, hv.SUM, flags) == hv.ERR_UNSUPPORTED
        assert status_of(ft, [d0], hv.FLOAT32, hv.FLOAT32, 2, hv.SUM, flags) == hv.ERR_UNSUPPORTED
        assert status_of(ft, [(FAKE, FAKE, FAKE, 3, b3, 64, FAKE, 4, 0, 4)], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM,
                         flags) == hv.ERR_INVALID  # the copy-out tiles missing
        assert status_of(ft, [(FAKE, FAKE, FAKE, 3, b3, 0, FAKE, 0, FAKE, 0)], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM,
                         flags) == hv.OK  # an empty bucket: nothing launched
    assert status_of(ft, [d0], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM,
                     hv.TILED_ADD_FROM_TENSORS) == hv.ERR_UNSUPPORTED  # needs the replacing steps in the tensors
    # bucket counts: 1 to 4; three or more only with both tensor flags; buckets x ranks <= 256
    stride = 1 << 24
    many = [(FAKE, FAKE, FAKE, 3, [x + i * stride for x in b3], 64, FAKE, 4, FAKE, 4) for i in range(5)]
    assert status_of(ft, [], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, both) == hv.ERR_INVALID
    assert status_of(ft, many, hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, both) == hv.ERR_INVALID
    assert status_of(ft, many[:3], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM,
                     hv.TILED_REPLACE_IN_TENSORS) == hv.ERR_UNSUPPORTED
    assert status_of(ft, many[:3], hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, hv.TILED_BUFFERS) == hv.ERR_UNSUPPORTED
    b100 = bufs(100, 64)
    big = [(FAKE, FAKE, FAKE, 3, [x + i * (1 << 34) for x in b100], 64, FAKE, 4, FAKE, 4) for i in range(3)]
    assert status_of(ft, big, hv.FLOAT32, hv.FLOAT32, 100, hv.SUM, both) == hv.ERR_UNSUPPORTED  # 300 buffers
    overlap = [many[0], (FAKE, FAKE, FAKE, 3, [b3[0] + 64, many[1][4][1], many[1][4][2]], 64, FAKE, 4, FAKE, 4)]
    assert status_of(ft, overlap, hv.FLOAT32, hv.FLOAT32, 3, hv.SUM, both) == hv.ERR_ALIAS


def test_fused_allreduce_rejects_overlapping_tensors():
    """Paired launches read and write two buckets' tensors at once, so the cycle refuses
    tensors that share memory (checked on the host, before any device work)."""
    import torch

    from paper_1802_05799_amd import cycle

    base = torch.zeros(1000)
    a, b, c = base[0:100], base[100:300], base[300:400]
    cycle._check_disjoint([[a, b], [c, base[400:600]]])  # disjoint: no error
    cycle._check_disjoint([[a, base[0:0]], [c, base[0:0]]])  # empty views take no memory
    with pytest.raises(ValueError, match="overlap"):
        cycle._check_disjoint([[a, b], [a, c]])  # one tensor on two ranks
    with pytest.raises(ValueError, match="overlap"):
        cycle._check_disjoint([[a, base[50:60]]])  # a view inside another
    with pytest.raises(ValueError, match="overlap"):
        cycle._check_disjoint([[base[0:101], b], [c, base[500:600]]])  # one element shared


def test_noalloc_ring_argument_checks():
    """The allocation-free ring checks its arguments and the static workspace's size
    before any HIP call (so these run without a GPU)."""
    lib = ctypes.CDLL(hv.LIB_PATH)
    lib.hvdx_ring_allreduce_noalloc.restype = ctypes.c_int
    lib.hvdx_ring_allreduce_noalloc.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int,
                                                ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    cap = hv.hvdx_ring_noalloc_max_bytes()
    assert cap == 64 << 20

    def status(n, count, dtype=hv.FLOAT32, op=hv.AVERAGE, compress=hv.COMPRESS_FP16, ptrs=None):
        ptrs = ptrs or [FAKE + r * (1 << 32) for r in range(n)]
        arr = (ctypes.c_void_p * len(ptrs))(*ptrs)
        return lib.hvdx_ring_allreduce_noalloc(arr, n, count, dtype, op, compress, None)

    assert status(8, 4_194_304 + 1) == hv.ERR_WORKSPACE  # 8 x 4,194,432 binary16 elements > 64 MiB
    assert "static" in hv.hvdx_last_error()
    assert status(128, 262_145) == hv.ERR_WORKSPACE
    assert status(2, 10, dtype=hv.FLOAT16) == hv.ERR_INVALID  # compression needs binary32
    assert status(2, 10, compress=7) == hv.ERR_INVALID
    assert status(2, 10, op=9) == hv.ERR_INVALID
    assert status(0, 10) == hv.ERR_INVALID
    assert status(2, 10, ptrs=[FAKE, FAKE + 8]) == hv.ERR_ALIAS
    assert status(3, 0) == hv.OK  # nothing to do, no HIP call


def test_broadcast_layout_matches_oracle():
    from oracle import broadcast

    g = np.random.default_rng(12)
    for _ in range(200):
        sizes = [int(s) for s in g.integers(0, 100, size=g.integers(0, 12))]
        assert tuple(hv.hvdx_broadcast_layout(sizes)) == broadcast.tensor_layout(sizes)
    with pytest.raises(hv.HvdxError):
        hv.hvdx_broadcast_layout([5, -1])


def test_broadcast_tensors_argument_checks():
    lib = ctypes.CDLL(hv.LIB_PATH)
    f = lib.hvdx_broadcast_tensors
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    fs = lib.hvdx_broadcast_tensors_step
    fs.restype = ctypes.c_int
    fs.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           ctypes.c_void_p]
    assert f(FAKE, FAKE, FAKE, 3, 100, 0, 0, None) == hv.ERR_INVALID  # no ranks
    assert f(FAKE, FAKE, FAKE, 3, 100, 129, 0, None) == hv.ERR_INVALID
    assert f(FAKE, FAKE, FAKE, 3, 100, 4, 4, None) == hv.ERR_INVALID  # root out of range
    assert f(FAKE, FAKE, FAKE, -1, 100, 4, 0, None) == hv.ERR_INVALID
    assert f(None, FAKE, FAKE, 3, 100, 4, 0, None) == hv.ERR_INVALID
    assert f(FAKE, FAKE, None, 3, 100, 4, 0, None) == hv.ERR_INVALID
    assert f(FAKE, FAKE, FAKE, 3, -5, 4, 0, None) == hv.ERR_INVALID
    assert f(FAKE, FAKE, FAKE, 3, 0, 4, 0, None) == hv.OK  # empty space: nothing launched
    assert f(None, None, None, 0, 0, 4, 0, None) == hv.OK
    assert fs(FAKE, FAKE, FAKE, 3, 100, 4, 0, 6, None) == hv.ERR_INVALID  # steps 0..5 for 4 ranks
    assert fs(FAKE, FAKE, FAKE, 3, 100, 4, 0, -1, None) == hv.ERR_INVALID
    assert fs(FAKE, FAKE, FAKE, 3, 0, 4, 0, 5, None) == hv.OK


def test_tensor_broadcast_rejects_bad_lists_before_any_device_work():
    """TensorBroadcast's checks on the tensor list, all on the host before its upload."""
    import torch

    base = torch.zeros(64)
    with pytest.raises(ValueError, match="ranks"):
        hv.TensorBroadcast([])
    with pytest.raises(ValueError, match="same number"):
        hv.TensorBroadcast([[base[:4]], [base[4:8], base[8:12]]])
    with pytest.raises(ValueError, match="GPU"):  # host tensors
        hv.TensorBroadcast([[base[:4]], [base[4:8]]])
    with pytest.raises(ValueError, match="contiguous"):
        hv.TensorBroadcast([[base[::2]], [base[1::2]]])


def _tiles(numel, offset, count, te, be, n, direction):
    arr, k = hv.hvdx_fuse_copy_tiles(numel, offset, count, te, be, n, direction)
    return [(x.pos, x.li, x.tensor, x.len, x.chunk) for x in arr[:k]]


def test_copy_tiles_cover_and_stay_inside_one_tensor_and_chunk():
    """The tile tables of the fused copies: every buffer position (copy-in) or tensor
    element (copy-out) in exactly one tile, each tile inside one tensor (or padding run)
    and one ring chunk, at most 256 vectors long, on its grid (the buffer's for the
    copy-in, the tensor's for the copy-out) except right after a chunk boundary off the
    vector grid, where a short tile reaches the next vector boundary."""
    g = np.random.default_rng(21)
    for case in range(60):
        te, be = [(0, 0), (0, 1), (1, 1)][case % 3]
        vec = 4 if 0 in (te, be) else 8
        tile = hv._lib.hvdx_fuse_tile_elems(te, be)
        assert tile % (256 * vec) == 0 and 256 * vec <= tile <= 1024 * vec
        n = int(g.integers(1, 20))
        numel = [int(x) for x in g.integers(0, 3 * tile, size=g.integers(1, 9))]
        align = [16, 2 if be == 1 else 4][case % 2] // (2 if be == 1 else 4)
        offset, count = [], 0
        for m in numel:
            s = -(-count // align) * align + int(g.integers(0, 3)) * align  # gaps: padding runs
            offset.append(s)
            count = s + m
        count += int(g.integers(0, 40))
        starts, lengths = ring.chunk_bounds(count, n)
        chunk_of = np.repeat(np.arange(n), lengths)
        for direction in (hv.COPY_IN, hv.COPY_OUT):
            tiles = _tiles(numel, offset, count, te, be, n, direction)
            hits = np.zeros(count, np.int64)
            for pos, li, t, length, c in tiles:
                assert 1 <= length <= tile
                hits[pos : pos + length] += 1
                assert (chunk_of[pos : pos + length] == c).all()
                if t >= 0:
                    assert offset[t] <= pos and pos + length <= offset[t] + numel[t] and li == pos - offset[t]
                    base = 0 if direction == hv.COPY_IN else offset[t]
                else:
                    assert direction == hv.COPY_IN and li == 0
                    assert not any(o < pos + length and pos < o + m for o, m in zip(offset, numel) if m)
                    base = 0
                rel = pos - base
                assert (rel + length - 1) // tile == rel // tile  # never across the tile grid
                if rel % vec:  # starts off the vector grid: right after a chunk or tensor boundary
                    assert pos in starts or pos in offset or direction == hv.COPY_IN
                    assert (rel + length) % vec == 0 or pos + length == count or \
                        pos + length in [s + ln for s, ln in zip(starts, lengths)] or \
                        pos + length in [o + m for o, m in zip(offset, numel)] or pos + length in offset
            inside = np.zeros(count, bool)
            for o, m in zip(offset, numel):
                inside[o : o + m] = True
            if direction == hv.COPY_IN:
                assert (hits == 1).all(), case
            else:
                assert (hits[inside] == 1).all() and (hits[~inside] == 0).all(), case


def test_copy_tiles_argument_checks():
    lib = ctypes.CDLL(hv.LIB_PATH)
    f = lib.hvdx_fuse_copy_tiles
    f.restype = ctypes.c_int64
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                  ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64]

    def call(numel, offset, count, te=0, be=0, n=4, d=0, cap=0, tiles=None):
        a = (ctypes.c_int64 * max(1, len(numel)))(*numel)
        o = (ctypes.c_int64 * max(1, len(offset)))(*offset)
        return f(a, o, len(numel), count, te, be, n, d, tiles, cap)

    assert call([10, 20], [0, 12], 32) > 0
    assert call([10, 20], [0, 8], 32) == hv.ERR_INVALID  # overlapping tensors
    assert call([10, 20], [0, 12], 31) == hv.ERR_INVALID  # past the buffer
    assert call([10], [0], 32, d=2) == hv.ERR_INVALID
    assert call([10], [0], 32, te=1, be=0) == hv.ERR_UNSUPPORTED
    assert call([10], [0], 32, n=0) == hv.ERR_INVALID
    buf = (hv._lib.CopyTile * 1)()
    assert call([3000], [0], 3000, cap=1, tiles=ctypes.cast(buf, ctypes.c_void_p)) == hv.ERR_WORKSPACE
    assert call([], [], 0) == 0
