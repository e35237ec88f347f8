"""Pins of the oracle's ring (paper section 3) against independent formulations."""
import numpy as np
import pytest

import _pins
from oracle import ring


def test_partition_matches_its_defining_properties():
    # contiguous cover, sizes within one, the longer chunks first: unique
    for n in range(1, 12):
        for count in list(range(0, 4 * n + 3)) + [1000003, 20391]:
            starts, lengths = ring.chunk_bounds(count, n)
            if count < 200:
                assert (starts, lengths) == _pins.partition_ref(count, n)
            assert starts[0] == 0 and sum(lengths) == count
            assert all(starts[c] + lengths[c] == starts[c + 1] for c in range(n - 1))
            assert max(lengths) - min(lengths) <= 1
            assert lengths == sorted(lengths, reverse=True)


@pytest.mark.parametrize("pin", _pins.RING_PINS, ids=lambda p: p.__name__)
def test_ring_pin(pin):
    assert pin(ring)


def test_hand_worked_intermediate_states():
    """Every intermediate state of the hand-worked N=3 example."""
    states, _ = _pins.read_ring_golden()
    seen = {}
    ring.ring_allreduce(states["initial"].copy(), "sum", observe=lambda ph, s, b: seen.__setitem__(f"{ph}{s}", b.copy()))
    for k in ("rs0", "rs1", "ag0", "ag1"):
        assert _pins.bits_equal(seen[k], states[k]), k
    seen.clear()
    ring.ring_allreduce(states["initial"].copy(), "average", observe=lambda ph, s, b: seen.__setitem__(f"{ph}{s}", b.copy()))
    assert _pins.bits_equal(seen["rs1"], states["avg_rs1"])
    assert _pins.bits_equal(seen["ag1"], states["avg_final"])


def test_owner_after_reduce_scatter():
    """After the adding half, rank (c-1) mod N holds the complete sum of chunk c."""
    rng = np.random.default_rng(5)
    for n in (2, 3, 5, 8):
        count = 7 * n + 3
        x = rng.integers(-50, 51, size=(n, count)).astype(np.float32)
        total = x.sum(axis=0)
        snap = {}
        ring.ring_allreduce(x.copy(), "sum", observe=lambda ph, s, b: snap.setdefault((ph, s), b.copy()))
        after = snap[("rs", n - 2)]
        starts, lengths = ring.chunk_bounds(count, n)
        for c in range(n):
            sl = slice(starts[c], starts[c] + lengths[c])
            assert np.array_equal(after[(c - 1) % n, sl], total[sl])


def test_check1_every_rank_identical_and_check2_fp64_bound():
    """Checks (1) and (2): identical ranks; |got - fp64 sum| within the recursive-summation
    bound gamma_{N-1} * sum|x| plus one rounding for the divide (derived in
    _pins.check2_coefficients), and within rel 1e-6*N."""
    rng = np.random.default_rng(6)
    for n in (1, 2, 3, 4, 7, 8, 16, 33):
        count = 3 * n + 101
        x = (rng.standard_normal((n, count)) * 0.01).astype(np.float32)
        for op in ("sum", "average"):
            got = ring.ring_allreduce(x.copy(), op)
            assert all(_pins.bits_equal(got[r], got[0]) for r in range(n))
            d = n if op == "average" else 1
            ref = x.astype(np.float64).sum(axis=0) / d
            absum = np.abs(x.astype(np.float64)).sum(axis=0) / d
            c, eta = _pins.check2_coefficients(n, op, "f32", cast_in=False)
            err = np.abs(got[0].astype(np.float64) - ref)
            assert np.all(err <= c * absum + eta), (n, op)
            assert np.all(err <= 1e-6 * n * absum)


def test_fp16_buffers_fp64_bound():
    """Check (2) for binary16 buffers fed with binary32 values rounded on the way in: the
    bound of _pins.check2_coefficients (the cast's rounding, N-1 binary16 additions, the
    divide, half a subnormal spacing per rounding in the subnormal range)."""
    rng = np.random.default_rng(7)
    for n in (1, 2, 4, 5, 16, 64):
        count = 2 * n + 257
        x32 = (rng.standard_normal((n, count)) * 0.01).astype(np.float32)
        x32[:, :4] *= 2.0 ** -12  # some inputs and sums in binary16's subnormal range
        x16 = x32.astype(np.float16)
        for op in ("sum", "average"):
            got = ring.ring_allreduce(x16.copy(), op)
            d = n if op == "average" else 1
            ref = x32.astype(np.float64).sum(axis=0) / d
            absum = np.abs(x32.astype(np.float64)).sum(axis=0) / d
            c, eta = _pins.check2_coefficients(n, op, "f16", cast_in=True)
            err = np.abs(got[0].astype(np.float64) - ref)
            assert np.all(err <= c * absum + eta), (n, op)


def test_empty_and_single_rank():
    x = np.zeros((4, 0), np.float32)
    assert ring.ring_allreduce(x, "average").shape == (4, 0)
    one = np.array([[1.5, -2.25, 3.0]], np.float32)
    assert _pins.bits_equal(ring.ring_allreduce(one.copy(), "sum"), one)
    assert _pins.bits_equal(ring.ring_allreduce(one.copy(), "average"), one)
    tr = ring.new_traffic(1)
    ring.ring_allreduce(one.copy(), "sum", traffic=tr)
    assert tr["sent"][0] == 0 and tr["recvd"][0] == 0


def test_count_below_nranks_has_empty_chunks():
    n = 6
    x = np.arange(n * 4, dtype=np.float32).reshape(n, 4)
    got = ring.ring_allreduce(x.copy(), "sum")
    assert np.array_equal(got, np.broadcast_to(x.sum(axis=0), x.shape))


def test_rejects_unknown_op():
    with pytest.raises(ValueError):
        ring.ring_allreduce(np.zeros((2, 3), np.float32), "max")
