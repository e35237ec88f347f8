"""GPU ring kernels against the oracle, element by element and bit for bit."""
import numpy as np
import pytest
import torch

import _pins
import paper_1802_05799_amd as hv
from _gpu import OPS, assert_bits_equal, from_gpu_rows, gpu_ring, say, to_gpu_rows
from oracle import fusion, ring

pytestmark = pytest.mark.gpu


def inputs(rng, n, count, dtype, scale=0.01):
    x = rng.standard_normal((n, count)) * scale * rng.choice([0.01, 1.0, 100.0], size=(n, count))
    return x.astype(dtype)


def oracle_ring(x, op, compress=False):
    if compress:
        b = fusion.cast(x, np.float16)
        ring.ring_allreduce(b, op)
        return fusion.cast(b, np.float32)
    return ring.ring_allreduce(x.copy(), op)


CASES = []
for _n in (1, 2, 3, 4, 5, 7, 8, 13, 16, 32, 64, 128):
    for _count in sorted({0, 1, _n - 1, _n, 4 * _n + 3, 1000, 8 * 256 * 4 * 4 + 13, 100003}):
        if _count >= 0:
            CASES.append((_n, _count))


@pytest.mark.parametrize("dtype", [np.float32, np.float16], ids=["f32", "f16"])
def test_ring_matches_oracle(dtype):
    rng = np.random.default_rng(100)
    for n, count in CASES:
        for op in ("sum", "average"):
            say(f"ring dtype={np.dtype(dtype).name} n={n} count={count} op={op}")
            x = inputs(rng, n, count, dtype)
            assert_bits_equal(gpu_ring(x, op), oracle_ring(x, op), f"n={n} count={count} op={op}")


def test_compressed_ring_matches_oracle():
    rng = np.random.default_rng(101)
    for n, count in CASES:
        for op in ("sum", "average"):
            say(f"compressed ring n={n} count={count} op={op}")
            x = inputs(rng, n, count, np.float32)
            assert_bits_equal(gpu_ring(x, op, compress=True), oracle_ring(x, op, True), f"n={n} count={count}")


def test_unaligned_buffers_take_the_scalar_path():
    rng = np.random.default_rng(102)
    for off in (1, 2, 3):
        for n, count in ((3, 1001), (8, 40000)):
            for dtype in (np.float32, np.float16):
                say(f"unaligned off={off} n={n} count={count} {np.dtype(dtype).name}")
                x = inputs(rng, n, count, dtype)
                assert_bits_equal(gpu_ring(x, "average", offset_elems=off), oracle_ring(x, "average"))
            x = inputs(rng, n, count, np.float32)
            assert_bits_equal(gpu_ring(x, "average", True, offset_elems=off), oracle_ring(x, "average", True))


def test_special_values():
    """Ties, subnormals (binary16 gradual underflow), signed zeros, infinities."""
    n, count = 4, 4096
    rng = np.random.default_rng(103)
    x32 = (rng.standard_normal((n, count)) * 1e-5).astype(np.float32)  # many binary16 subnormals
    x32[:, :8] = np.array([0.0, -0.0, 1.0, 2.0 ** -24, 65504.0, 65520.0, np.inf, -np.inf], np.float32)
    x32[1, 8:16] = 2.0 ** 24
    x32[:, 16:24] = 1.0
    def fold(x, op, compress=False):
        rows, keep = to_gpu_rows(x)
        dt = hv.FLOAT32 if x.dtype == np.float32 else hv.FLOAT16
        hv.hvdx_fold_allreduce([r.data_ptr() for r in rows], x.shape[0], x.shape[1], dt, OPS[op],
                               hv.COMPRESS_FP16 if compress else hv.COMPRESS_NONE)
        return from_gpu_rows(rows)

    def halves(x, op, compress=False):
        n, count = x.shape
        rows, keep = to_gpu_rows(x)
        dt = hv.FLOAT32 if x.dtype == np.float32 else hv.FLOAT16
        cmp = hv.COMPRESS_FP16 if compress else hv.COMPRESS_NONE
        wsb = hv.hvdx_ring_workspace_bytes(n, count, dt, cmp)
        ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device="cuda")
        ptrs = [r.data_ptr() for r in rows]
        hv.hvdx_ring_reduce_scatter(ptrs, n, count, dt, OPS[op], cmp, ws.data_ptr() if wsb else 0, wsb)
        hv.hvdx_ring_allgather(ptrs, n, count, dt, OPS[op], cmp, ws.data_ptr() if wsb else 0, wsb)
        return from_gpu_rows(rows)

    x16 = fusion.cast(x32, np.float16)
    for nr in (4, 3, 2):
        for op in ("sum", "average"):
            say(f"special values n={nr} op={op}")
            a32, a16 = x32[:nr].copy(), x16[:nr].copy()
            for path in (gpu_ring, fold, halves):
                assert_bits_equal(path(a32, op), oracle_ring(a32, op), f"f32 {path.__name__}")
                assert_bits_equal(path(a16, op), oracle_ring(a16, op), f"f16 {path.__name__}")
                assert_bits_equal(path(a32, op, True), oracle_ring(a32, op, True), f"compressed {path.__name__}")


def test_each_step_matches_oracle_states():
    """hvdx_ring_step, one step at a time: every intermediate state equals the oracle's."""
    rng = np.random.default_rng(104)
    for n, count, dtype in ((3, 7, np.float32), (5, 1234, np.float32), (6, 4099, np.float16), (16, 70001, np.float32)):
        for op in ("sum", "average"):
            say(f"steps n={n} count={count} op={op}")
            x = inputs(rng, n, count, dtype)
            states = []
            ring.ring_allreduce(x.copy(), op, observe=lambda ph, s, b: states.append((ph, s, b.copy())))
            rows, keep = to_gpu_rows(x)
            ptrs = [r.data_ptr() for r in rows]
            dt = hv.FLOAT32 if dtype == np.float32 else hv.FLOAT16
            for ph, s, want in states:
                phase = hv.PHASE_REDUCE_SCATTER if ph == "rs" else hv.PHASE_ALLGATHER
                hv.hvdx_ring_step(ptrs, n, count, dt, OPS[op], hv.COMPRESS_NONE, phase, s)
                assert_bits_equal(from_gpu_rows(rows), want, f"{ph}{s}")


def test_hand_worked_example_on_gpu():
    states, _ = _pins.read_ring_golden()
    rows, keep = to_gpu_rows(states["initial"])
    ptrs = [r.data_ptr() for r in rows]
    for key, phase, s in (("rs0", 0, 0), ("rs1", 0, 1), ("ag0", 1, 0), ("ag1", 1, 1)):
        hv.hvdx_ring_step(ptrs, 3, 7, hv.FLOAT32, hv.SUM, hv.COMPRESS_NONE, phase, s)
        assert_bits_equal(from_gpu_rows(rows), states[key], key)
    assert_bits_equal(gpu_ring(states["initial"], "average"), states["avg_final"], "average")


def test_compressed_steps_wire_and_outputs():
    """Compressed steps: after the adding half the owner's wire copy holds the binary16
    result of the oracle's fp16 ring; at the end every binary32 buffer holds it widened."""
    rng = np.random.default_rng(105)
    n, count = 5, 3001
    x = inputs(rng, n, count, np.float32)
    rows, keep = to_gpu_rows(x)
    ptrs = [r.data_ptr() for r in rows]
    wsb = hv.hvdx_ring_workspace_bytes(n, count, hv.FLOAT32, hv.COMPRESS_FP16)
    ws = torch.zeros(wsb, dtype=torch.uint8, device="cuda")
    states = []
    ring.ring_allreduce(fusion.cast(x, np.float16), "average", observe=lambda ph, s, b: states.append(b.copy()))
    for s in range(n - 1):
        hv.hvdx_ring_step(ptrs, n, count, hv.FLOAT32, hv.AVERAGE, hv.COMPRESS_FP16, hv.PHASE_REDUCE_SCATTER, s,
                          ws.data_ptr(), wsb)
    torch.cuda.synchronize()
    stride = (count + 127) // 128 * 128
    wire = ws.view(torch.float16)[: n * stride].view(n, stride)[:, :count].cpu().numpy()
    after_rs = states[n - 2]
    starts, lengths = ring.chunk_bounds(count, n)
    for c in range(n):
        owner = (c - 1) % n
        sl = slice(starts[c], starts[c] + lengths[c])
        assert_bits_equal(wire[owner, sl], after_rs[owner, sl], f"owner of chunk {c}")
    for s in range(n - 1):
        hv.hvdx_ring_step(ptrs, n, count, hv.FLOAT32, hv.AVERAGE, hv.COMPRESS_FP16, hv.PHASE_ALLGATHER, s,
                          ws.data_ptr(), wsb)
    assert_bits_equal(from_gpu_rows(rows), fusion.cast(states[-1], np.float32), "final")


def test_streams_and_repeat_calls():
    """Work on a side stream, twice in a row on the same buffers."""
    rng = np.random.default_rng(106)
    n, count = 8, 1 << 20
    x = inputs(rng, n, count, np.float32)
    rows, keep = to_gpu_rows(x)
    ptrs = [r.data_ptr() for r in rows]
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        hv.hvdx_ring_allreduce(ptrs, n, count, hv.FLOAT32, hv.SUM, 0, 0, 0, s.cuda_stream)
        hv.hvdx_ring_allreduce(ptrs, n, count, hv.FLOAT32, hv.SUM, 0, 0, 0, s.cuda_stream)
    s.synchronize()
    want = ring.ring_allreduce(ring.ring_allreduce(x.copy(), "sum"), "sum")
    assert_bits_equal(from_gpu_rows(rows), want, "twice")


def test_reduce_scatter_and_allgather_halves():
    """hvdx_ring_reduce_scatter leaves rank (c-1) holding chunk c of the result (the
    oracle's state after the adding half); hvdx_ring_allgather then completes the
    allreduce; alone, the all-gather spreads rank r's chunk (r+1) to every rank."""
    rng = np.random.default_rng(107)
    for n, count, dtype, compress in ((3, 7, np.float32, False), (5, 10007, np.float32, False),
                                      (8, 33001, np.float16, False), (6, 4099, np.float32, True)):
        say(f"halves n={n} count={count} {np.dtype(dtype).name} compress={compress}")
        x = inputs(rng, n, count, dtype)
        states = []
        base = fusion.cast(x, np.float16) if compress else x.copy()
        ring.ring_allreduce(base, "average", observe=lambda ph, s, b: states.append(b.copy()))
        rows, keep = to_gpu_rows(x)
        ptrs = [r.data_ptr() for r in rows]
        dt = hv.FLOAT32 if dtype == np.float32 else hv.FLOAT16
        cmp = hv.COMPRESS_FP16 if compress else hv.COMPRESS_NONE
        wsb = hv.hvdx_ring_workspace_bytes(n, count, dt, cmp)
        ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device="cuda")
        hv.hvdx_ring_reduce_scatter(ptrs, n, count, dt, hv.AVERAGE, cmp, ws.data_ptr() if wsb else 0, wsb)
        starts, lengths = ring.chunk_bounds(count, n)
        if not compress:
            got = from_gpu_rows(rows)
            for c in range(n):
                sl = slice(starts[c], starts[c] + lengths[c])
                assert_bits_equal(got[(c - 1) % n, sl], states[n - 2][(c - 1) % n, sl], f"owner of chunk {c}")
        hv.hvdx_ring_allgather(ptrs, n, count, dt, hv.AVERAGE, cmp, ws.data_ptr() if wsb else 0, wsb)
        want = fusion.cast(states[-1], np.float32) if compress else states[-1]
        assert_bits_equal(from_gpu_rows(rows), want, "after both halves")
    # the all-gather half alone
    n, count = 5, 1003
    x = inputs(rng, n, count, np.float32)
    rows, keep = to_gpu_rows(x)
    hv.hvdx_ring_allgather([r.data_ptr() for r in rows], n, count, hv.FLOAT32, hv.SUM)
    starts, lengths = ring.chunk_bounds(count, n)
    want = np.empty(count, np.float32)
    for c in range(n):
        want[starts[c] : starts[c] + lengths[c]] = x[(c - 1) % n, starts[c] : starts[c] + lengths[c]]
    assert_bits_equal(from_gpu_rows(rows), np.broadcast_to(want, (n, count)).copy(), "allgather alone")


def test_fold_matches_the_ring_bit_for_bit():
    """hvdx_fold_allreduce computes the ring's fold directly: same bits as the oracle's ring."""
    rng = np.random.default_rng(108)
    for n, count in CASES[::3] + [(8, 1 << 20), (64, 100003), (3, 7)]:
        for dtype, compress in ((np.float32, False), (np.float16, False), (np.float32, True)):
            for op in ("sum", "average"):
                say(f"fold n={n} count={count} {np.dtype(dtype).name} compress={compress} {op}")
                x = inputs(rng, n, count, dtype)
                rows, keep = to_gpu_rows(x)
                dt = hv.FLOAT32 if dtype == np.float32 else hv.FLOAT16
                hv.hvdx_fold_allreduce([r.data_ptr() for r in rows], n, count, dt, OPS[op],
                                       hv.COMPRESS_FP16 if compress else hv.COMPRESS_NONE)
                assert_bits_equal(from_gpu_rows(rows), oracle_ring(x, op, compress), f"n={n} count={count}")
    # unaligned buffers take the per-element path
    x = inputs(rng, 5, 1001, np.float32)
    rows, keep = to_gpu_rows(x, offset_elems=1)
    hv.hvdx_fold_allreduce([r.data_ptr() for r in rows], 5, 1001, hv.FLOAT32, hv.AVERAGE)
    assert_bits_equal(from_gpu_rows(rows), oracle_ring(x, "average"), "unaligned")
