"""Pins of the plain C oracle (oracle/csrc/oracle.c) that the host times at full size.

The C oracle is pinned like the numpy one -- against the hand-worked ring and
rounding tables, the rank-centric brute force, closed forms and the integer
round-to-nearest-even reference -- and then shown bit-identical to the numpy
oracle on whole allreduces (plans, casts, the ring, padding, direct tensors),
with one thread and with several.
"""
import numpy as np
import pytest

import _pins
from oracle import allreduce as oall
from oracle import fusion, native, ring
from test_oracle_arith import _structured_f32_patterns, f32_to_f16_ref
from test_oracle_fusion import check_plan_invariants
from workloads import configs, rng


class CRing:
    """The C ring behind the interface the ring pins call."""

    def __init__(self, threads):
        self.threads = threads

    def ring_allreduce(self, bufs, op, count=None, elems=None, traffic=None, observe=None):
        assert count is None and elems is None and traffic is None and observe is None
        b = np.ascontiguousarray(bufs)
        return native.ring_allreduce(b, op, threads=self.threads)


C_RING_PINS = [_pins.pin_bruteforce, _pins.pin_exact_integers, _pins.pin_one_hot, _pins.pin_rank_bits,
               _pins.pin_order]


@pytest.mark.parametrize("threads", [1, 3])
@pytest.mark.parametrize("pin", C_RING_PINS, ids=lambda p: p.__name__)
def test_c_ring_pin(pin, threads):
    assert pin(CRing(threads))


def test_c_ring_hand_worked_example():
    states, _ = _pins.read_ring_golden()
    got = native.ring_allreduce(states["initial"].copy(), ring.SUM)
    assert _pins.bits_equal(got, states["ag1"])
    got = native.ring_allreduce(states["initial"].copy(), ring.AVERAGE)
    assert _pins.bits_equal(got, states["avg_final"])


def test_c_arithmetic_hand_worked_table():
    """The rounding table through the C oracle: casts directly; binary16 sums as a
    two-rank ring; divisions as an AVERAGE over n ranks of (x, +0, ..., +0)."""
    rows = _pins.read_rounding_golden()
    for row in rows:
        kind = row[0]
        if kind == "cast":
            got = native.f32_to_f16(_pins.f32_bits(row[1]))
            assert _pins.bits_equal(got.view(np.float16), _pins.f16_bits(row[2])), row
        elif kind == "add16":
            x = np.stack([_pins.f16_bits(row[1]), _pins.f16_bits(row[2])])
            got = native.ring_allreduce(x, ring.SUM)
            assert all(_pins.bits_equal(got[r], _pins.f16_bits(row[3])) for r in range(2)), row
        elif kind in ("div32", "div16"):
            val = _pins.f32_bits(row[1]) if kind == "div32" else _pins.f16_bits(row[1])
            want = _pins.f32_bits(row[3]) if kind == "div32" else _pins.f16_bits(row[3])
            n = int(row[2])
            if np.signbit(val[0]) and val[0] == 0:
                continue  # -0 + +0 is +0: this form cannot carry a negative zero
            x = np.zeros((n, 1), dtype=val.dtype)
            x[0] = val
            got = native.ring_allreduce(x, ring.AVERAGE)
            assert all(_pins.bits_equal(got[r], want) for r in range(n)), row
        else:
            raise AssertionError(row)


def test_c_cast_to_fp16_structured_patterns():
    """2^26 binary32 patterns (every binade and binary16 quantum, exact ties and one
    past them) against numpy's conversion, and a random quarter of a million of them
    against the integer round-to-nearest-even reference; NaNs stay NaNs."""
    bits = _structured_f32_patterns()
    got = native.f32_to_f16(bits.view(np.float32))
    nan = np.isnan(bits.view(np.float32))
    with np.errstate(over="ignore"):
        want = bits.view(np.float32)[~nan].astype(np.float16).view(np.uint16)
    assert np.array_equal(got[~nan], want)
    assert np.all(np.isnan(got[nan].view(np.float16)))
    pick = np.random.default_rng(5).choice(np.flatnonzero(~nan), size=1 << 18, replace=False)
    assert np.array_equal(got[pick], f32_to_f16_ref(bits[pick]))


def test_c_widen_every_fp16_exactly():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = native.f16_to_f32(h)
    finite = np.isfinite(h.view(np.float16))
    # exact: equal to the value as binary64 computes it from the fields
    s = np.where(h >> 15, -1.0, 1.0)
    e = ((h >> 10) & 0x1F).astype(np.int64)
    m = (h & 0x3FF).astype(np.float64)
    val = s * np.where(e == 0, m * 2.0 ** -24, (1.0 + m / 1024.0) * 2.0 ** (e - 15))
    assert np.array_equal(got[finite].astype(np.float64), val[finite])
    assert np.array_equal(got.view(np.uint32)[~finite] & 0x7F800000, np.full((~finite).sum(), 0x7F800000, np.uint32))
    assert np.array_equal(np.isnan(got[~finite]), np.isnan(h.view(np.float16)[~finite]))


def _plan_rows(plan):
    return [(b.count, list(b.tensors), list(b.offsets), bool(b.direct)) for b in plan]


def _c_plan_rows(numel, esize, threshold, align):
    bucket_of, offset, direct, count = native.fuse_plan(numel, esize, threshold, align)
    rows = []
    for b in range(len(count)):
        ts = [t for t in range(len(numel)) if bucket_of[t] == b]
        rows.append((int(count[b]), ts, [int(offset[t]) for t in ts], bool(direct[b])))
    return rows


@pytest.mark.parametrize("name", list(configs.WORKLOADS))
def test_c_plan_matches_golden_layouts(name):
    w = configs.get(name)
    es = 2 if w.compress else 4
    rows = _c_plan_rows(w.numel(), es, 64 << 20, 16)
    assert rows == _plan_rows(fusion.fuse_plan(w.numel(), es))
    golden = []
    with open(_pins.GOLDEN + "/plans.txt") as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line and line[0] == name:
                golden.append(tuple(int(v) for v in line[1:]))
    assert [(c, len(ts), int(d)) for c, ts, _, d in rows] == golden


def test_c_plan_random_lists_and_invariants():
    g = np.random.default_rng(31)
    for trial in range(300):
        numel = [int(v) for v in g.integers(0, 40, size=g.integers(0, 30))]
        if trial % 3 == 0:
            numel.append(int(g.integers(0, 200)))
        esize = int(g.choice([2, 4]))
        align = int(g.choice([esize, 8, 16, 64]))
        threshold = int(g.integers(0, 160))
        rows = _c_plan_rows(numel, esize, threshold, align)
        plan = [fusion.Bucket(ts, offs, c, d) for c, ts, offs, d in rows]
        check_plan_invariants(numel, esize, plan, threshold, align)
        assert rows == _plan_rows(fusion.fuse_plan(numel, esize, threshold, align))


def test_c_plan_rejects_bad_arguments():
    with pytest.raises(ValueError):
        native.fuse_plan([1], 4, align=12)
    with pytest.raises(ValueError):
        native.fuse_plan([1], 4, align=2)
    with pytest.raises(ValueError):
        native.fuse_plan([1], 4, threshold=-1)


def _bits(a):
    a = np.asarray(a)
    return a.view(np.uint32 if a.dtype == np.float32 else np.uint16)


def _same(c_out, np_out):
    for cr, nr in zip(c_out, np_out):
        for a, b in zip(cr, nr):
            assert a.dtype == b.dtype and a.shape == b.shape
            assert np.array_equal(_bits(a), _bits(b))


def _random_case(g, n, dtype):
    t = int(g.integers(1, 12))
    numel = [int(v) for v in g.integers(0, 300, size=t)]
    scale = g.choice([1e-3, 1.0, 1e3], size=t)
    return [[(g.standard_normal(numel[i]) * scale[i]).astype(dtype) for i in range(t)] for _ in range(n)]


@pytest.mark.parametrize("threads", [1, 4])
def test_c_allreduce_equals_numpy_oracle_random(threads):
    """Ragged tensor lists, 1-9 ranks, thresholds that make several buffers and direct
    tensors, binary32 and binary16 tensors, compression, SUM and AVERAGE."""
    g = np.random.default_rng(41)
    for trial in range(120):
        n = int(g.integers(1, 10))
        dtype = np.float16 if trial % 5 == 4 else np.float32
        per_rank = _random_case(g, n, dtype)
        compress = dtype == np.float32 and trial % 3 == 0
        op = ring.AVERAGE if trial % 2 else ring.SUM
        es = 2 if (compress or dtype == np.float16) else 4
        threshold = int(g.choice([0, 64, 400, 1200, 64 << 20]))
        align = int(g.choice([es, 16, 64]))
        want = oall.allreduce(per_rank, op, compress=compress, threshold=threshold, align=align)
        got = native.allreduce(per_rank, op, compress=compress, threshold=threshold, align=align, threads=threads)
        _same(got, want)


@pytest.mark.parametrize("name", ["tiny"])
def test_c_allreduce_equals_numpy_oracle_workload(name):
    w = configs.get(name)
    numel, prefix = w.numel(), w.prefix()
    per_rank = [[rng.values(w.dist, w.key(r), np.arange(prefix[t], prefix[t] + numel[t]), w.sigma)
                 for t in range(len(numel))] for r in range(w.nranks)]
    want = oall.allreduce(per_rank, w.op, compress=w.compress)
    _same(native.allreduce(per_rank, w.op, compress=w.compress, threads=1), want)
    _same(native.allreduce(per_rank, w.op, compress=w.compress, threads=4), want)
    # and compressed, on the same tensors
    want = oall.allreduce(per_rank, w.op, compress=True)
    _same(native.allreduce(per_rank, w.op, compress=True, threads=2), want)


def test_c_allreduce_large_chunks_across_threads():
    """A buffer large enough that every chunk is split over all threads: the thread
    count never changes a bit."""
    g = np.random.default_rng(43)
    n = 5
    per_rank = [[(g.standard_normal(m) * 0.01).astype(np.float32) for m in (300_001, 7, 120_000)] for _ in range(n)]
    one = native.allreduce(per_rank, ring.AVERAGE, threads=1)
    many = native.allreduce(per_rank, ring.AVERAGE, threads=8)
    _same(many, one)
    _same(one, oall.allreduce(per_rank, ring.AVERAGE))


def test_c_allreduce_workspace_reused_and_checked():
    """Fusion buffers in a caller's workspace, reused across calls whose plans differ
    (stale contents must not leak into the padding), give the allocating form's bits."""
    g = np.random.default_rng(47)
    n = 4
    numel = [5, 17, 1, 33, 2, 9]
    ws = np.full(native.workspace_bytes(numel, n, threshold=96, align=64), 0xFF, dtype=np.uint8)
    for trial in range(3):
        per_rank = [[g.standard_normal(m).astype(np.float32) for m in numel] for _ in range(n)]
        want = native.allreduce(per_rank, ring.SUM, threshold=96, align=64)
        _same(native.allreduce(per_rank, ring.SUM, threshold=96, align=64, workspace=ws), want)
        _same(want, oall.allreduce(per_rank, ring.SUM, threshold=96, align=64))
    with pytest.raises(ValueError):
        native.allreduce(per_rank, ring.SUM, threshold=96, align=64, workspace=ws[:-1])


def test_c_allreduce_rejects_compressing_fp16():
    x = [[np.ones(4, np.float16)] for _ in range(2)]
    with pytest.raises(ValueError):
        native.allreduce(x, ring.SUM, compress=True)


# ---- planted mistakes: every pin above must be able to fail -------------------------
# Each mutant is the C source with one plausible slip, compiled on the CPU into a
# temporary library; at least one of the checks below must reject it.
MUTANTS = {
    "adding step receiver one rank too far": ("rcv = (c + s + 1) % n", "rcv = (c + s + 2) % n"),
    "replacing step sender of the next chunk": ("snd = (c - 1 + s + n) % n", "snd = (c + s + n) % n"),
    "no division by N": ("if (avg && last) v = v / (float)n;", "(void)last;"),
    "division at the first adding step": ("const int last = s == n - 2;", "const int last = s == 0;"),
    "one adding step too few": ("for (int s = 0; s < n - 1; ++s) {\n    const int last", "for (int s = 1; s < n - 1; ++s) {\n    const int last"),
    "partition without the longer first chunks": ("*start = c * q + (c < rem ? c : rem);", "*start = c * q;"),
    "ties rounded up": ("if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) ++h;", "if (rest >= 0x1000u) ++h;"),
    "subnormals truncated": ("if (rest > half || (rest == half && (h & 1u))) ++h;", "(void)rest; (void)half;"),
    "widening drops a fraction bit": ("return sign | ((e - 15 + 127) << 23) | (m << 13);", "return sign | ((e - 15 + 127) << 23) | ((m & 0x3feu) << 13);"),
    "a tie at the threshold does not fit": ("start_bytes + bytes > threshold", "start_bytes + bytes >= threshold"),
    "offsets not aligned": ("(count[nb] * esize + align - 1) / align * align", "count[nb] * esize"),
}


def _mutant_caught():
    """True when some check rejects the currently bound library."""
    try:
        if not all(p(CRing(1)) for p in C_RING_PINS):
            return True
        test_c_ring_hand_worked_example()
        test_c_arithmetic_hand_worked_table()
        test_c_widen_every_fp16_exactly()
        for name in configs.WORKLOADS:
            test_c_plan_matches_golden_layouts(name)
        test_c_plan_random_lists_and_invariants()
        test_c_allreduce_equals_numpy_oracle_random(1)
    except AssertionError:
        return True
    return False


@pytest.mark.parametrize("mutant", list(MUTANTS))
def test_planted_mistake_is_caught(mutant, tmp_path):
    import os
    import subprocess

    from oracle import build as obuild

    src = open(obuild.SRC).read()
    old, new = MUTANTS[mutant]
    assert src.count(old) == 1, "the mutation site moved"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    so = str(tmp_path / "libmutant.so")
    flags = [f for f in obuild.FLAGS if f != "-Werror"]
    subprocess.run(["gcc", *flags, "-w", "-o", so, str(path)], check=True)
    prev = native.use_library(so)
    try:
        assert _mutant_caught(), f"no check rejects: {mutant}"
    finally:
        native.restore_library(prev)
    assert os.path.exists(obuild.LIB)
