"""Pins of the oracle's broadcast: the defining result, a hand-worked chain, and traffic."""
import numpy as np
import pytest

import _pins
from oracle import broadcast


def distinct(n, nbytes):
    x = np.zeros((n, nbytes), np.uint8)
    for r in range(n):
        x[r] = (np.arange(nbytes) * 7 + 31 * r + 1) % 251  # rows differ everywhere
    return x


def test_every_rank_ends_with_the_root_bytes():
    for n in range(1, 10):
        for nbytes in (0, 1, 15, 16, 17, 16 * n - 1, 16 * n, 1000, 4099):
            for root in {0, n - 1, n // 2}:
                x = distinct(n, nbytes)
                got = broadcast.chain_broadcast(x.copy(), root)
                assert np.array_equal(got, np.broadcast_to(x[root], x.shape))


def test_hand_worked_chain():
    rows = {}
    with open(_pins.GOLDEN + "/broadcast_n3.txt") as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                rows[line[0]] = line[1:]
    x = distinct(3, 40)
    chunks = broadcast.chunk_bytes(40, 3)
    assert chunks == [(0, 16), (16, 32), (32, 40)]
    seen = {}
    tr = broadcast.new_traffic(3)
    broadcast.chain_broadcast(x.copy(), 1, traffic=tr, observe=lambda s, b: seen.__setitem__(s, b.copy()))
    for s in range(4):
        for r, owners in enumerate(rows[f"step{s}"]):
            for j, src in enumerate(owners.split(",")):
                lo, hi = chunks[j]
                assert np.array_equal(seen[s][r, lo:hi], x[int(src), lo:hi]), (s, r, j)
    assert list(tr["sent"]) == [int(v) for v in rows["sent"]]
    assert list(tr["recvd"]) == [int(v) for v in rows["recvd"]]


def test_chunks_cover_in_units():
    for n in range(1, 9):
        for nbytes in range(0, 200):
            ch = broadcast.chunk_bytes(nbytes, n)
            assert ch[0][0] == 0 and ch[-1][1] == nbytes
            assert all(a[1] == b[0] for a, b in zip(ch, ch[1:]))
            assert all(lo % 16 == 0 for lo, hi in ch if hi > lo)  # non-empty chunks start on a unit
            units = [(-(-hi // 16) - lo // 16) if hi > lo else 0 for lo, hi in ch]  # 16-byte units covered
            assert sum(units) == -(-nbytes // 16)
            assert max(units) - min(units) <= 1 and units == sorted(units, reverse=True)


def test_traffic_each_non_root_receives_everything_once():
    for n in (2, 3, 5, 8):
        nbytes = 1000
        tr = broadcast.new_traffic(n)
        broadcast.chain_broadcast(distinct(n, nbytes), 2 % n, traffic=tr)
        root = 2 % n
        assert all(tr["recvd"][r] == (0 if r == root else nbytes) for r in range(n))
        last = (root - 1) % n
        assert all(tr["sent"][r] == (0 if r == last else nbytes) for r in range(n))


def test_bad_root():
    with pytest.raises(ValueError):
        broadcast.chain_broadcast(np.zeros((3, 8), np.uint8), 3)


# ---- many tensors in one call (reading B2) ----------------------------------------------
def test_tensor_layout_hand_worked():
    assert broadcast.tensor_layout([]) == ([], 0)
    assert broadcast.tensor_layout([5, 16, 0, 33, 1]) == ([0, 16, 32, 32, 80], 81)
    assert broadcast.tensor_layout([16, 16]) == ([0, 16], 32)
    assert broadcast.tensor_layout([0, 0, 7]) == ([0, 0, 0], 7)


def tensors(n, sizes, seed):
    g = np.random.default_rng(seed)
    return [[g.integers(0, 256, size=s, dtype=np.uint8) for s in sizes] for _ in range(n)]


def test_tensors_every_rank_ends_with_the_root_bytes():
    g = np.random.default_rng(11)
    for n in range(1, 10):
        for _ in range(4):
            sizes = [int(s) for s in g.integers(0, 70, size=g.integers(0, 9))]
            root = int(g.integers(0, n))
            x = tensors(n, sizes, int(g.integers(1 << 30)))
            want = [[a.copy() for a in x[root]] for _ in range(n)]
            got = broadcast.chain_broadcast_tensors([[a.copy() for a in row] for row in x], root)
            assert all(np.array_equal(a, b) for ra, rb in zip(got, want) for a, b in zip(ra, rb)), (n, sizes)


def test_tensors_hand_worked_chain():
    rows = {}
    with open(_pins.GOLDEN + "/broadcast_tensors_n3.txt") as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                rows[line[0]] = line[1:]
    starts, total = broadcast.tensor_layout([10, 20])
    assert starts + [total] == [int(v) for v in rows["layout"]]
    x = [[(np.arange(s, dtype=np.int64) * 7 + 31 * r + 1).astype(np.uint8) for s in (10, 20)] for r in range(3)]
    segments = [(0, slice(0, 10)), (1, slice(0, 16)), (1, slice(16, 20))]
    seen = {}
    broadcast.chain_broadcast_tensors([[a.copy() for a in row] for row in x], 1,
                                      observe=lambda s, pr: seen.__setitem__(s, [[a.copy() for a in row] for row in pr]))
    assert sorted(seen) == [0, 1, 2, 3]
    for s in range(4):
        for r, owners in enumerate(rows[f"step{s}"]):
            for (t, sl), src in zip(segments, owners.split(",")):
                assert np.array_equal(seen[s][r][t][sl], x[int(src)][t][sl]), (s, r, t)


def test_one_tensor_is_the_single_buffer_chain():
    """With one tensor the layout is the buffer itself: every step equals chain_broadcast's."""
    for n, nbytes, root in ((2, 33, 1), (5, 1000, 3), (7, 16 * 7, 0)):
        x = distinct(n, nbytes)
        a, b = {}, {}
        broadcast.chain_broadcast(x.copy(), root, observe=lambda s, bufs: a.__setitem__(s, bufs.copy()))
        broadcast.chain_broadcast_tensors([[row.copy()] for row in x], root,
                                          observe=lambda s, pr: b.__setitem__(s, np.stack([r[0] for r in pr])))
        assert sorted(a) == sorted(b) and all(np.array_equal(a[s], b[s]) for s in a)
