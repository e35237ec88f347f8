"""Independent formulations that pin the oracle's ring (test helpers, CPU only).

None of these reuses the oracle's code: the arithmetic goes through binary64 and
one final rounding (equal to the correctly rounded binary32/binary16 operation
because binary64 keeps at least 2p+2 bits for both), the schedule is written
rank-centrically instead of chunk-centrically, and the partition comes from its
defining properties.
"""
from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ---- arithmetic through binary64 -----------------------------------------------------
def add_ref(a, b):
    """Correctly rounded sum: exact binary64 sum (or one binary64 rounding) then one
    rounding to the buffer type."""
    with np.errstate(over="ignore"):
        return (np.asarray(a, np.float64) + np.asarray(b, np.float64)).astype(a.dtype)


def div_ref(x, n):
    return (np.asarray(x, np.float64) / float(n)).astype(x.dtype)


# ---- the partition from its properties ---------------------------------------------
def partition_ref(count, n):
    """Deal elements one at a time to the chunk with the fewest so far (lowest index on
    ties), then lay the chunks out contiguously in index order."""
    sizes = [0] * n
    for _ in range(count):
        c = min(range(n), key=lambda k: (sizes[k], k))
        sizes[c] += 1
    starts, acc = [], 0
    for s in sizes:
        starts.append(acc)
        acc += s
    return starts, sizes


# ---- rank-centric message passing (brute force) -------------------------------------
def mailbox_allreduce(x, op):
    """Every rank keeps its own buffer; in each step every rank first writes one message
    to its right neighbour, then all messages are delivered at once.

    Adding step s: rank r sends chunk (r - s) mod N; the receiver adds it.
    Replacing step s: rank r sends chunk (r + 1 - s) mod N; the receiver overwrites.
    """
    n = len(x)
    bufs = [np.array(b, copy=True) for b in x]
    count = bufs[0].size
    starts, sizes = partition_ref(count, n)
    span = lambda c: slice(starts[c], starts[c] + sizes[c])  # noqa: E731
    for s in range(n - 1):
        msgs = [((r + 1) % n, (r - s) % n, bufs[r][span((r - s) % n)].copy()) for r in range(n)]
        for dst, c, payload in msgs:
            v = add_ref(bufs[dst][span(c)], payload)
            if op == "average" and s == n - 2:
                v = div_ref(v, n)
            bufs[dst][span(c)] = v
    if op == "average" and n == 1:
        bufs[0] = div_ref(bufs[0], 1)
    for s in range(n - 1):
        msgs = [((r + 1) % n, (r + 1 - s) % n, bufs[r][span((r + 1 - s) % n)].copy()) for r in range(n)]
        for dst, c, payload in msgs:
            bufs[dst][span(c)] = payload
    return bufs


# ---- closed form ---------------------------------------------------------------------
def fold_allreduce(x, op):
    """Element e of chunk c: FIN(((x_c + x_{c+1}) + ...) + x_{c+N-1}), identical on
    every rank."""
    n = len(x)
    count = x[0].size
    starts, sizes = partition_ref(count, n)
    out = np.empty_like(x[0])
    for c in range(n):
        sl = slice(starts[c], starts[c] + sizes[c])
        acc = x[c][sl].copy()
        for k in range(1, n):
            acc = add_ref(acc, x[(c + k) % n][sl])
        if op == "average":
            acc = div_ref(acc, n)
        out[sl] = acc
    return [out.copy() for _ in range(n)]


# ---- golden fixtures -----------------------------------------------------------------
def read_ring_golden():
    states, counters = {}, {}
    cur = None
    with open(os.path.join(GOLDEN, "ring_n3_count7.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            head, *rest = line.split()
            if head == "state":
                cur = rest[0]
                states[cur] = []
            elif head in ("sent", "recvd"):
                counters[head] = [int(v) for v in rest]
                cur = None
            else:
                states[cur].append([float(v) for v in line.split()])
    return {k: np.array(v, dtype=np.float32) for k, v in states.items()}, counters


def read_rounding_golden():
    rows = []
    with open(os.path.join(GOLDEN, "rounding.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def f32_bits(h):
    return np.array([int(h, 16)], dtype=np.uint32).view(np.float32)


def f16_bits(h):
    return np.array([int(h, 16)], dtype=np.uint16).view(np.float16)


def bits_equal(a, b):
    a, b = np.asarray(a), np.asarray(b)
    if a.dtype != b.dtype or a.shape != b.shape:
        return False
    u = {2: np.uint16, 4: np.uint32, 8: np.uint64}[a.dtype.itemsize]
    return bool(np.array_equal(a.view(u), b.view(u)))


# ---- pins as predicates over a ring module (used directly and for mutants) -----------
def _rng_inputs(rng, n, count, dtype, kind):
    if kind == "random":
        x = rng.standard_normal((n, count)) * rng.choice([1e-3, 1.0, 1e3], size=(n, count))
    elif kind == "int":
        x = rng.integers(-100, 101, size=(n, count)).astype(np.float64)
    return x.astype(dtype)


def pin_bruteforce(ring_mod, ns=range(1, 8), seed=0):
    """Oracle == mailbox simulation == closed-form fold, bitwise, tiny N and count."""
    rng = np.random.default_rng(seed)
    for dtype in (np.float32, np.float16):
        for n in ns:
            for count in range(0, 3 * n + 3):
                for op in ("sum", "average"):
                    x = _rng_inputs(rng, n, count, dtype, "random")
                    got = ring_mod.ring_allreduce(x.copy(), op)
                    mb = mailbox_allreduce(list(x), op)
                    fd = fold_allreduce(list(x), op)
                    for r in range(n):
                        if not (bits_equal(got[r], mb[r]) and bits_equal(got[r], fd[r])):
                            return False
    return True


def pin_golden_states(ring_mod):
    """The hand-worked N=3 example: final states for SUM and AVERAGE, and traffic."""
    states, counters = read_ring_golden()
    x = states["initial"].copy()
    tr = ring_mod.new_traffic(3)
    got = ring_mod.ring_allreduce(x, "sum", traffic=tr)
    if not bits_equal(got, states["ag1"]):
        return False
    if list(tr["sent"]) != counters["sent"] or list(tr["recvd"]) != counters["recvd"]:
        return False
    got = ring_mod.ring_allreduce(states["initial"].copy(), "average")
    return bits_equal(got, states["avg_final"])


def pin_exact_integers(ring_mod, seed=1):
    """Small integers: SUM is the exact integer sum, AVERAGE with N a power of two is
    the exact sum / N, whatever the order."""
    rng = np.random.default_rng(seed)
    for dtype in (np.float32, np.float16):
        for n in (1, 2, 3, 4, 5, 8):
            count = 4 * n + 3
            x = rng.integers(-100, 101, size=(n, count)) if dtype == np.float32 else rng.integers(-60, 61, size=(n, count))
            exact = x.sum(axis=0)
            got = ring_mod.ring_allreduce(x.astype(dtype), "sum")
            if not all(np.array_equal(got[r].astype(np.float64), exact) for r in range(n)):
                return False
            if n & (n - 1) == 0:
                got = ring_mod.ring_allreduce(x.astype(dtype), "average")
                if not all(np.array_equal(got[r].astype(np.float64), exact / n) for r in range(n)):
                    return False
    return True


def pin_one_hot(ring_mod, seed=2):
    """Only rank e mod N is nonzero at element e: every rank ends with that value
    (SUM) or that value / N (AVERAGE), which pins the routing of every chunk."""
    rng = np.random.default_rng(seed)
    for dtype in (np.float32, np.float16):
        for n in (2, 3, 5, 6):
            count = 5 * n + 2
            v = (rng.standard_normal(count) + 2.0).astype(dtype)
            x = np.zeros((n, count), dtype=dtype)
            for e in range(count):
                x[e % n, e] = v[e]
            got = ring_mod.ring_allreduce(x.copy(), "sum")
            if not all(bits_equal(got[r], v) for r in range(n)):
                return False
            got = ring_mod.ring_allreduce(x.copy(), "average")
            want = div_ref(v, n)
            if not all(bits_equal(got[r], want) for r in range(n)):
                return False
    return True


def pin_rank_bits(ring_mod):
    """x_r = 2^r: the sum is exactly 2^N - 1, so every rank is counted exactly once."""
    for n, dtype in ((1, np.float32), (7, np.float32), (20, np.float32), (10, np.float16)):
        count = 3 * n + 1
        x = np.stack([np.full(count, 2.0 ** r, dtype=dtype) for r in range(n)])
        got = ring_mod.ring_allreduce(x, "sum")
        if not np.all(got.astype(np.float64) == 2.0 ** n - 1):
            return False
    return True


def pin_order(ring_mod):
    """2^24 at rank c and 1.0 elsewhere for the elements of chunk c (binary32).  The
    ring's fold starts at rank c, so every +1 is a tie that rounds back to 2^24; a fold
    that adds two or more ones before reaching rank c ends at 2^24 + 2 or more."""
    for n in (3, 4, 5, 8):
        count = 3 * n + 2
        starts, sizes = partition_ref(count, n)
        x = np.ones((n, count), dtype=np.float32)
        for c in range(n):
            x[c, starts[c] : starts[c] + sizes[c]] = 2.0 ** 24
        got = ring_mod.ring_allreduce(x, "sum")
        if not np.all(got == np.float32(2.0 ** 24)):
            return False
    return True


def pin_traffic(ring_mod):
    """Check (3): rank r sends every chunk but (r+1) in the adding half and every chunk
    but (r+2) in the replacing half, so sent_r = 2*count - len_{r+1} - len_{r+2} and
    received_r = 2*count - len_r - len_{r+1}; in total 2(N-1)*count, which is exactly
    2(N-1)/N of the buffer per rank when N divides count."""
    for n in (1, 2, 3, 4, 7):
        for count in (0, 1, n - 1, 4 * n, 4 * n + 3):
            if count < 0:
                continue
            _, sizes = partition_ref(count, n)
            tr = ring_mod.new_traffic(n)
            ring_mod.ring_allreduce(np.ones((n, count), np.float32), "sum", traffic=tr)
            for r in range(n):
                if n == 1:
                    want_s = want_r = 0
                else:
                    want_s = 2 * count - sizes[(r + 1) % n] - sizes[(r + 2) % n]
                    want_r = 2 * count - sizes[r] - sizes[(r + 1) % n]
                if tr["sent"][r] != want_s or tr["recvd"][r] != want_r:
                    return False
            if int(tr["sent"].sum()) != 2 * (n - 1) * count:
                return False
            if count % n == 0 and not all(int(s) * n == 2 * (n - 1) * count for s in tr["sent"]):
                return False
    return True


def pin_columns(ring_mod, seed=3):
    """The column-subset form equals the whole run restricted to those columns."""
    rng = np.random.default_rng(seed)
    for dtype in (np.float32, np.float16):
        for n in (3, 4, 6):
            count = 11 * n + 5
            x = _rng_inputs(rng, n, count, dtype, "random")
            whole = ring_mod.ring_allreduce(x.copy(), "average")
            elems = np.sort(rng.choice(count, size=count // 3, replace=False))
            part = ring_mod.ring_allreduce(x[:, elems].copy(), "average", count=count, elems=elems)
            if not bits_equal(part, whole[:, elems]):
                return False
    return True


RING_PINS = [pin_bruteforce, pin_golden_states, pin_exact_integers, pin_one_hot, pin_rank_bits, pin_order, pin_traffic, pin_columns]


# ---- check (2): the bound on the distance to the binary64 sum -------------------------
def check2_coefficients(n, op, buffer, cast_in):
    """(c, eta) such that check (2) holds as |result - ref| <= c * A + eta per element.

    ref is the binary64 sum of the rank inputs x_r (the uncast binary32 values), divided
    by N for AVERAGE; A = sum_r |x_r| divided by D (D = N for AVERAGE, 1 for SUM).
    buffer: "f32" or "f16", the type the ring adds in; cast_in: the inputs are rounded to
    binary16 on the way in (fp16 compression of binary32 gradients).

    Derivation (reading R13: Higham's recursive-summation bound).  u is the buffer
    type's unit roundoff (2^-24 or 2^-11) and g = (N-1)u / (1 - (N-1)u) bounds the
    relative error of N-1 additions done one after the other: |s - S'| <= g * T' for
    the computed sum s, the exact sum S' and T' = sum |x'_r| of the values the ring
    adds.  Addition keeps fl(a+b) = (a+b)(1+d) with |d| <= u also under gradual
    underflow (a sum of subnormals is exact), so no absolute term enters there.
      * Rounding the inputs to binary16: x' = x(1+d) + e with |d| <= u and
        |e| <= 2^-25 (half the subnormal spacing), so |S' - S| <= u T + N 2^-25 and
        T' <= (1+u) T + N 2^-25.  Without the cast x' = x: u_c = 0, e = 0.
      * SUM: |s - S| <= g T' + |S' - S| <= T (u_c + g(1+u_c)) + N e (1 + g).
      * AVERAGE: the one division by N rounds once, |fl(s/N) - s/N| <= u |s|/N + h, with
        h = half the smallest subnormal of the buffer type (2^-150, 2^-25), and
        |s| <= (1+g) T'.  So |fl(s/N) - S/N| <= (T/N)(u_c + (g + u(1+g))(1+u_c))
        + e (1 + g + u(1+g)) + h.
    """
    u = 2.0 ** -24 if buffer == "f32" else 2.0 ** -11
    g = (n - 1) * u / (1 - (n - 1) * u)
    uc = 2.0 ** -11 if cast_in else 0.0
    e = 2.0 ** -25 if cast_in else 0.0
    if op == "sum":
        return uc + g * (1 + uc), n * e * (1 + g)
    h = 2.0 ** -150 if buffer == "f32" else 2.0 ** -25
    return uc + (g + u * (1 + g)) * (1 + uc), e * (1 + g + u * (1 + g)) + h
