"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that the pins
catch every one: a pin that no mutant can fail would pin nothing."""
import importlib.util
import os
import sys
import types

import numpy as np
import pytest

import _pins
from workloads import configs

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def load_mutant(module, old, new):
    path = os.path.join(ORACLE, module + ".py")
    with open(path) as f:
        src = f.read()
    assert src.count(old) >= 1, f"mutation site not found: {old!r}"
    src = src.replace(old, new, 1)
    name = f"oracle_mutant_{module}"
    mod = types.ModuleType(name)
    sys.modules[name] = mod  # dataclasses look their module up here
    try:
        exec(compile(src, path, "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod


def ring_pins_fail(mod):
    for pin in _pins.RING_PINS:
        try:
            if not pin(mod):
                return pin.__name__
        except Exception as exc:  # a crash is a caught mistake too
            return f"{pin.__name__}: {type(exc).__name__}"
    return None


RING_MUTANTS = [
    ("rs sender shifted", "return (c + s) % n", "return (c + s + 1) % n"),
    ("rs direction reversed", "return (c + s + 1) % n", "return (c - s - 1) % n"),
    ("ag sender off by one", "return (c - 1 + s) % n", "return (c + s) % n"),
    ("ag receiver off by one", "    return (c + s) % n\n\n\ndef add", "    return (c + s + 1) % n\n\n\ndef add"),
    ("one adding step dropped", "for s in range(n - 1):\n        for c in range(n):\n            snd, rcv = rs_", "for s in range(n - 2):\n        for c in range(n):\n            snd, rcv = rs_"),
    ("one replacing step dropped", "for s in range(n - 1):\n        for c in range(n):\n            snd, rcv = ag_", "for s in range(n - 2):\n        for c in range(n):\n            snd, rcv = ag_"),
    ("divide dropped", "v = divide(v, n)", "pass"),
    ("divide at first step", "s == n - 2:", "s == 0:"),
    ("divide by N-1", "return (x / np.float32(n)).astype(np.float32)", "return (x / np.float32(max(n - 1, 1))).astype(np.float32)"),
    ("fp16 divide in binary16 steps", "return (x.astype(np.float32) / np.float32(n)).astype(np.float16)", "return (x * np.float16(1.0 / n)).astype(np.float16)"),
    ("sender added to itself", "v = add(bufs[rcv, cols[c]], bufs[snd, cols[c]])", "v = add(bufs[snd, cols[c]], bufs[snd, cols[c]])"),
    ("receiver not accumulated", "v = add(bufs[rcv, cols[c]], bufs[snd, cols[c]])", "v = bufs[snd, cols[c]] + 0"),
    ("replace transposed", "bufs[rcv, cols[c]] = bufs[snd, cols[c]]", "bufs[snd, cols[c]] = bufs[rcv, cols[c]]"),
    ("partition: long chunks last", "lengths = [q + (1 if c < rem else 0)", "lengths = [q + (1 if c >= nranks - rem else 0)"),
    ("partition: starts ignore remainder", "starts = [c * q + min(c, rem)", "starts = [c * q"),
    ("traffic counts only sender", 'traffic["recvd"][rcv] += lengths[c]', "pass"),
    ("traffic counted per column", 'traffic["sent"][snd] += lengths[c]', 'traffic["sent"][snd] += 1'),
    ("column slice off by one", 'hi = int(np.searchsorted(elems, starts[c] + lengths[c], side="left"))', 'hi = int(np.searchsorted(elems, starts[c] + lengths[c], side="right"))'),
]


@pytest.mark.parametrize("label,old,new", RING_MUTANTS, ids=[m[0] for m in RING_MUTANTS])
def test_ring_mutant_is_caught(label, old, new):
    mod = load_mutant("ring", old, new)
    assert ring_pins_fail(mod) is not None, f"no pin caught mutant: {label}"


def test_unmutated_ring_passes_every_pin():
    from oracle import ring

    assert ring_pins_fail(ring) is None


# ---- fusion ----------------------------------------------------------------------------
def fusion_pins_fail(fmod):
    import test_oracle_fusion as tf

    try:
        for name, w in configs.WORKLOADS.items():
            es = 2 if w.compress else 4
            tf.check_plan_invariants(w.numel(), es, fmod.fuse_plan(w.numel(), es))
        if fmod.fuse_plan([4096 * 4096], 4)[0].direct or not fmod.fuse_plan([4096 * 4096 + 1], 4)[0].direct:
            return "tie"
        rng = np.random.default_rng(0)
        for _ in range(100):
            numel = list(rng.integers(0, 40, size=rng.integers(0, 20)))
            tf.check_plan_invariants(numel, 4, fmod.fuse_plan(numel, 4, 96, 16), 96, 16)
        numel = [3, 5, 1, 8, 2]
        (b,) = fmod.fuse_plan(numel, 4, threshold=1 << 20)
        xs = [np.arange(n, dtype=np.float32) + 100 * (t + 1) for t, n in enumerate(numel)]
        buf = fmod.pack(xs, b, np.float32)
        if b.offsets != [0, 4, 12, 16, 24] or b.count != 26:
            return "layout"
        back = fmod.unpack(buf, b, numel, np.float32)
        if not all(np.array_equal(u, x) for u, x in zip(back, xs)):
            return "roundtrip"
        pad = np.ones(b.count, bool)
        for t, off in zip(b.tensors, b.offsets):
            pad[off : off + numel[t]] = False
        if np.any(buf[pad] != 0):
            return "padding"
        tensor, local = fmod.buffer_origin(b, numel, np.arange(b.count))
        for e in range(b.count):
            if (tensor[e] >= 0) == pad[e] or (tensor[e] >= 0 and buf[e] != xs[tensor[e]][local[e]]):
                return "origin"
    except AssertionError:
        return "invariant"
    except Exception as exc:
        return type(exc).__name__
    return None


FUSION_MUTANTS = [
    ("no alignment", "start_bytes = -(-cur.count * esize // align) * align", "start_bytes = cur.count * esize"),
    ("tie does not fit", "if cur.tensors and start_bytes + nbytes > threshold:", "if cur.tensors and start_bytes + nbytes >= threshold:"),
    ("oversize test inclusive", "if nbytes > threshold:", "if nbytes >= threshold:"),
    ("bucket never closed", "if cur.tensors and start_bytes + nbytes > threshold:", "if False:"),
    ("pack shifted by one", "buf[off : off + x.size] = cast(x, dtype)", "buf[off + 1 : off + 1 + x.size] = cast(x, dtype)[: max(0, min(x.size, bucket.count - off - 1))]"),
    ("padding not zeroed", "buf = np.zeros(bucket.count, dtype=dtype)", "buf = np.ones(bucket.count, dtype=dtype)"),
    ("unpack reads wrong tensor offset", "return [cast(buf[off : off + numel[t]], dtype)", "return [cast(buf[off + 1 : off + 1 + numel[t]], dtype)"),
    ("origin off by one", "local[inside] = elems[inside] - off", "local[inside] = elems[inside] - off - 1"),
]


@pytest.mark.parametrize("label,old,new", FUSION_MUTANTS, ids=[m[0] for m in FUSION_MUTANTS])
def test_fusion_mutant_is_caught(label, old, new):
    mod = load_mutant("fusion", old, new)
    assert fusion_pins_fail(mod) is not None, f"no pin caught mutant: {label}"


def test_unmutated_fusion_passes():
    spec = importlib.util.find_spec("oracle.fusion")
    assert spec is not None
    from oracle import fusion

    assert fusion_pins_fail(fusion) is None


# ---- broadcast -------------------------------------------------------------------------
def broadcast_pins_fail(bmod):
    import test_oracle_broadcast as tb

    try:
        for n in (1, 2, 3, 5, 8):
            for nbytes in (0, 1, 17, 16 * n, 1000):
                for root in {0, n - 1, n // 2}:
                    x = tb.distinct(n, nbytes)
                    if not np.array_equal(bmod.chain_broadcast(x.copy(), root), np.broadcast_to(x[root], x.shape)):
                        return "result"
        if bmod.chunk_bytes(40, 3) != [(0, 16), (16, 32), (32, 40)]:
            return "chunks"
        # 80 bytes = 5 units = 3 * 1 + 2: the first two chunks take two units each
        if bmod.chunk_bytes(80, 3) != [(0, 32), (32, 64), (64, 80)]:
            return "chunk remainder"
        for n in (2, 3, 5):
            tr = bmod.new_traffic(n)
            bmod.chain_broadcast(tb.distinct(n, 1000), 1 % n, traffic=tr)
            if any(tr["recvd"][r] != (0 if r == 1 % n else 1000) for r in range(n)):
                return "traffic"
        # hand-worked intermediate states (root 1, three ranks)
        x = tb.distinct(3, 40)
        seen = {}
        bmod.chain_broadcast(x.copy(), 1, observe=lambda s, b: seen.__setitem__(s, b.copy()))
        want_step0 = x.copy()
        want_step0[2, 0:16] = x[1, 0:16]  # step 0: only chunk 0 leaves the root
        if not np.array_equal(seen[0], want_step0):
            return "schedule"
        # many tensors per call (reading B2): layout and the hand-worked two-tensor chain
        if bmod.tensor_layout([5, 16, 0, 33, 1]) != ([0, 16, 32, 32, 80], 81):
            return "layout"
        xs = [[(np.arange(s, dtype=np.int64) * 7 + 31 * r + 1).astype(np.uint8) for s in (10, 20)] for r in range(3)]
        seen = {}
        bmod.chain_broadcast_tensors([[a.copy() for a in row] for row in xs], 1,
                                     observe=lambda s, pr: seen.__setitem__(s, [[a.copy() for a in row] for row in pr]))
        # after step 0 only chunk 0 (tensor 0) has reached rank 2
        if not (np.array_equal(seen[0][2][0], xs[1][0]) and np.array_equal(seen[0][2][1], xs[2][1])
                and np.array_equal(seen[0][0][0], xs[0][0])):
            return "tensor schedule"
        for n in (2, 4):
            ys = [[(np.arange(s) + 13 * r).astype(np.uint8) for s in (3, 40, 0, 17)] for r in range(n)]
            got = bmod.chain_broadcast_tensors([[a.copy() for a in row] for row in ys], n - 1)
            if not all(np.array_equal(a, b) for row in got for a, b in zip(row, ys[n - 1])):
                return "tensor result"
    except Exception as exc:
        return type(exc).__name__
    return None


BROADCAST_MUTANTS = [
    ("chunks not in whole units", "units = -(-nbytes // UNIT)", "units = nbytes"),
    ("long chunks last", "n = q + (1 if j < rem else 0)", "n = q + (1 if j >= nranks - rem else 0)"),
    ("last link dropped", "for k in range(n - 1):  # link", "for k in range(n - 2):  # link"),
    ("one step short", "for step in range(2 * n - 2):", "for step in range(2 * n - 3):"),
    ("chunk schedule not staggered", "j = step - k", "j = step"),
    ("root ignored", "src, dst = (root + k) % n, (root + k + 1) % n", "src, dst = k % n, (k + 1) % n"),
    ("copy reversed", "bufs[dst, lo:hi] = bufs[src, lo:hi]", "bufs[src, lo:hi] = bufs[dst, lo:hi]"),
    ("traffic counts sender as receiver", 'traffic["recvd"][dst] += hi - lo', 'traffic["recvd"][src] += hi - lo'),
    ("tensors packed without alignment", "start = -(-end // UNIT) * UNIT", "start = end"),
    ("tensor gaps rounded down", "start = -(-end // UNIT) * UNIT", "start = end // UNIT * UNIT"),
    ("tensor copied back from rank 0", "a[:] = bufs[r, s : s + a.size]", "a[:] = bufs[0, s : s + a.size]"),
]


@pytest.mark.parametrize("label,old,new", BROADCAST_MUTANTS, ids=[m[0] for m in BROADCAST_MUTANTS])
def test_broadcast_mutant_is_caught(label, old, new):
    mod = load_mutant("broadcast", old, new)
    assert broadcast_pins_fail(mod) is not None, f"no pin caught mutant: {label}"


def test_unmutated_broadcast_passes():
    from oracle import broadcast

    assert broadcast_pins_fail(broadcast) is None
