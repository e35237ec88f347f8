"""CPU models of the elements each kernel launch writes and reads (test helper).

Each function replays one launcher's grid and its kernel's index arithmetic (block and
lane to ring chunk, tile, vector and rank slot) and returns, per rank, how many times
each element is written, and read where the check needs it.  The models are written
from the kernels in paper_1802_05799_amd/csrc; `Knobs` holds the few index choices a
planted mistake changes, so the tests can show that the checks catch such a mistake.

Conventions: positions are element indices of a rank's buffer (or of a tensor); the
alignment of a pointer enters only through its byte address modulo 16 (`mis`).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass
class Knobs:
    lane_shift: int = 0  # added to every lane's vector index (0 in the kernels)
    pair_split: int = 0  # added to the column where the second ring of a pair starts
    pair_column_shift: int = 0  # added to the second ring's own column index (0 in the kernels)
    chunk_tile_skip: int = 0  # tiles of a chunk skipped at its start (fused copies)
    skip_slot: int = 0  # the slot the fused copy-in leaves out (the sender: 0)
    receiver_from: int = -1  # the fused copy-out reads rank `receiver + this` (the sender: -1)
    replace_sender: int = -1  # replacing step s into the tensors reads rank `chunk + s + this` (-1)
    rs_ag_next: int = 0  # the fused step into the tensors also writes rank `chunk + this` (0)
    tile_block_stride: int = 0  # block b of a replacing step takes tiles b*this + j (0: tiles per block)
    add_sender: int = 0  # adding step s from the tensors: the sender of chunk c is rank c+s+this (0)
    fused_own_from_buffer: bool = False  # the fused step reads the owner's value from its buffer (False)
    xcd_shift: int = 0  # added to a block's XCD in tile_block() (0)
    bucket_end_shift: int = 0  # added to each bucket's first launch tile in ring_bucket() (0)


K = Knobs()
STREAM_BYTES = 128 << 20  # a ring step streams when a rank buffer is at least this large


def add(arr, idx, what="write"):
    """arr[idx] += 1 for every index (repeats counted), refusing indices outside arr: a
    model that steps outside a buffer is a caught mistake, not a wrap-around."""
    idx = np.asarray(idx, np.int64).reshape(-1)
    if idx.size and (idx.min() < 0 or idx.max() >= arr.size):
        raise IndexError(f"{what} outside the buffer: [{idx.min()}, {idx.max()}] of {arr.size}")
    np.add.at(arr, idx, 1)


def chunk(c, q, rem):
    return c * q + min(c, rem), q + (1 if c < rem else 0)


def head_elems(mis, esize, length):
    """Elements before the first 16-byte boundary (mis = address mod 16)."""
    h = (16 - mis) // esize if mis else 0
    return min(h, length)


@dataclass(frozen=True)
class Policy:
    U: int
    BS: int
    WAVE: bool = False


# the launch shapes of ring_kernels.hip (only U, BS and the lane layout decide which
# elements a lane touches; the cache hints do not)
RS_CACHED, RS_STREAM = Policy(2, 256), Policy(1, 64)
AG_CACHED, AG_STREAM, AG_LAST = Policy(2, 512), Policy(1, 64), Policy(2, 512)
RSAG_CACHED, RSAG_STREAM = Policy(1, 256), Policy(1, 64)
C16_CACHED, C16_RS_STREAM, C16_AG_STREAM = Policy(2, 256), Policy(1, 64), Policy(2, 256)


def streams(q, n, esize):
    return (q + 1) * n * esize >= STREAM_BYTES


def step_grid_x(q, rem, V, U, BS):
    longest = q + (1 if rem else 0)
    vecs = longest // V + 2
    bx = (vecs + BS * U - 1) // (BS * U)
    return min(max(bx, 1), 1 << 20)


def lane_vecs(blk, P, k=K):
    """Vector index of every (lane, u) of a block whose span starts at vector blk."""
    t = np.arange(P.BS, dtype=np.int64)[:, None]
    u = np.arange(P.U, dtype=np.int64)[None, :]
    if P.WAVE:
        idx = blk + (t >> 6) * 64 * P.U + u * 64 + (t & 63)
    else:
        idx = blk + u * P.BS + t
    return (idx + k.lane_shift).reshape(-1)


def body_elements(length, head, V, P, bx, gx, guard_whole=True, k=K):
    """Chunk-local elements one block of a ring step body touches (head and tail
    element by element, the rest as vectors), with repetition."""
    nvec = (length - head) // V
    tail = head + nvec * V
    gtid = bx * P.BS + np.arange(P.BS, dtype=np.int64)
    gth = gx * P.BS
    out = []
    for first, stop in ((0, head), (tail, length)):
        e = first + gtid
        while (e < stop).any():
            out.append(e[e < stop])
            e = e + gth
    blk = bx * P.BS * P.U
    while blk < nvec:
        idx = lane_vecs(blk, P, k)
        if not (guard_whole and blk + P.BS * P.U <= nvec):  # the whole-span branch has no per-vector guard
            idx = idx[idx < nvec]
        out.append((head + idx[:, None] * V + np.arange(V)[None, :]).reshape(-1))
        blk += gx * P.BS * P.U
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def ring_step(kind, n, count, step, esize, mis=None, vec_ok=True, policy=None, k=K):
    """One launch of rs_step_kernel ("rs"), ag_step_kernel ("ag") or rs_ag_step_kernel
    ("rs_ag", adding step N-2 with replacing step 0).  mis[r]: rank r's buffer address
    mod 16.  Returns (writes, sender_reads, own_reads) as (n, count) counts.  (With
    N = 2 the fused step's sender is the rank it also writes, element by element in the
    same lane, which reads before it writes.)"""
    mis = mis or [0] * n
    q, rem = divmod(count, n)
    V = 16 // esize
    if policy is None:
        st = streams(q, n, esize)
        if kind == "rs":
            policy = RS_STREAM if st else RS_CACHED
        elif kind == "ag":
            policy = AG_STREAM if st else (AG_LAST if step == n - 3 else AG_CACHED)
        else:
            policy = RSAG_STREAM if st else RSAG_CACHED
    gx = step_grid_x(q, rem, V, policy.U, policy.BS)
    writes = np.zeros((n, count), np.int64)
    sreads = np.zeros((n, count), np.int64)
    oreads = np.zeros((n, count), np.int64)
    for c in range(n):
        start, length = chunk(c, q, rem)
        if kind == "rs":
            snd = (c + step) % n
            dsts, own = [(snd + 1) % n], (snd + 1) % n
        elif kind == "ag":
            snd = (c + step + n - 1) % n
            dsts, own = [(snd + 1) % n], None
        else:
            snd = (c + n - 2) % n
            own = (snd + 1) % n
            dsts = [own, c]
        d0 = dsts[0]
        head = head_elems((mis[d0] + start * esize) % 16, esize, length) if vec_ok else length
        for bx in range(gx):
            e = start + body_elements(length, head, V, policy, bx, gx, k=k)
            for d in dsts:
                add(writes[d], e)
            add(sreads[snd], e, "read")
            if own is not None:
                add(oreads[own], e, "read")
    return writes, sreads, oreads


def ring_pair_step(kind, n, counts, step, esize, k=K):
    """One launch of a two-ring pair kernel: ring 0's columns of blocks, then ring 1's.
    Returns the writes per ring, (2, n, count_i) as a list of two arrays."""
    qs = [divmod(c, n) for c in counts]
    V = 16 // esize
    longer = 0 if qs[0][0] >= qs[1][0] else 1
    st = streams(qs[longer][0], n, esize)
    policy = {"rs": RS_STREAM if st else RS_CACHED,
              "ag": AG_STREAM if st else (AG_LAST if step == n - 3 else AG_CACHED),
              "rs_ag": RSAG_STREAM if st else RSAG_CACHED}[kind]
    g = [step_grid_x(q, rem, V, policy.U, policy.BS) for q, rem in qs]
    x0 = g[0] + k.pair_split
    writes = [np.zeros((n, c), np.int64) for c in counts]
    for col in range(g[0] + g[1]):
        z = 1 if col >= x0 else 0
        bx, gx = (col - x0, g[0] + g[1] - x0) if z else (col, x0)
        if z:
            bx += k.pair_column_shift
        q, rem = qs[z]
        for c in range(n):
            start, length = chunk(c, q, rem)
            if kind == "rs":
                dsts = [(c + step + 1) % n]
            elif kind == "ag":
                dsts = [(c + step) % n]
            else:
                dsts = [(c + n - 1) % n, c]
            head = head_elems((start * esize) % 16, esize, length)  # fusion buffers are 16-byte aligned
            e = start + body_elements(length, head, V, policy, bx, gx, k=k)
            for d in dsts:
                add(writes[z][d], e)
    return writes


def c16_step(kind, n, count, step, k=K):
    """Compressed ring: rs_step_c16_kernel ("rs": writes the receiver's binary16 wire
    copy), ag_first_c16_kernel ("ag0": writes the owner's and the receiver's binary32
    values) and rs_ag_step_c16_kernel ("rs_ag": writes the owner's and rank c's binary32
    values).  Binary32 buffers and the 256-byte aligned wire are 16-byte aligned.
    Returns (x_writes, wire_writes) as (n, count) counts."""
    q, rem = divmod(count, n)
    st = streams(q, n, 4)
    xw = np.zeros((n, count), np.int64)
    ww = np.zeros((n, count), np.int64)
    for c in range(n):
        start, length = chunk(c, q, rem)
        if kind == "rs":
            P, V, es = (C16_RS_STREAM if st else C16_CACHED), 8, 2
            snd = (c + step) % n
            targets = [(ww, (snd + 1) % n)]
        elif kind == "ag0":
            P, V, es = (C16_AG_STREAM if st else C16_CACHED), 4, 4
            snd = (c + n - 1) % n
            targets = [(xw, snd), (xw, (snd + 1) % n)]
        else:
            P, V, es = (C16_RS_STREAM if st else C16_CACHED), 4, 4
            snd = (c + n - 2) % n
            targets = [(xw, (snd + 1) % n), (xw, c)]
        gx = step_grid_x(q, rem, V, P.U, P.BS)
        head = head_elems((start * es) % 16, es, length)
        for bx in range(gx):
            e = start + body_elements(length, head, V, P, bx, gx, guard_whole=False, k=k)
            for arr, r in targets:
                add(arr[r], e)
    return xw, ww


# ---- the copy kernels (fusion_kernels.hip) -----------------------------------------------
@dataclass(frozen=True)
class CopyCfg:
    POS: int
    RB: int
    RPB: int
    BS: int = 256

    @property
    def tile_vecs(self):
        return self.BS * self.POS


PACK_CFG = CopyCfg(2, 2, 2)
UNPACK_CFG = CopyCfg(2, 1, 2)
SMALL_CFG = CopyCfg(1, 1, 0)
BCAST_CFG = CopyCfg(2, 1, 2)


def vec_elems(tensor_es, buf_es):
    return 4 if 4 in (tensor_es, buf_es) else 8


def ranks_per_block(cfg, n):
    return cfg.RPB if 0 < cfg.RPB < n else n


def copy_grid(cfg, ring, count, V, n):
    rpb = ranks_per_block(cfg, n)
    groups = (n + rpb - 1) // rpb
    tile = cfg.tile_vecs * V
    if not ring:  # (tiles, rank groups)
        return (count + tile - 1) // tile, groups, 1
    longest = count // n + (1 if count % n else 0)
    return (longest + tile - 1 + tile - 1) // tile, n, groups


class Layout:
    """A bucket's tensors in its buffer: offsets and ends, and the lookup of the tensor
    owning a buffer position (the last tensor starting at or before it)."""

    def __init__(self, numel, offset):
        self.off = np.asarray(offset, np.int64)
        self.end = self.off + np.asarray(numel, np.int64)

    def lookup(self, p):
        return np.searchsorted(self.off, p, side="right") - 1


def block_span(ring, tile, count, n, rpb, q, rem, group, bx, c, k=K):
    if ring:
        cs, length = chunk(c, q, rem)
        ce = cs + length
        p0 = (cs & ~(tile - 1)) + (bx + k.chunk_tile_skip) * tile
        p1 = min(p0 + tile, ce)
    else:
        cs, ce = 0, count
        p0 = bx * tile
        p1 = min(p0 + tile, count)
    rbeg = group * rpb
    return p0, p1, cs, ce, rbeg, min(rbeg + rpb, n)


def tile_positions(cfg, p0, V, k=K):
    t = np.arange(cfg.BS, dtype=np.int64)[:, None]
    u = np.arange(cfg.POS, dtype=np.int64)[None, :]
    return (p0 + (u * cfg.BS + t + k.lane_shift) * V).reshape(-1)


def classify(lay, p, V, p1, cs, ce):
    """0 none, 1 whole vector of one tensor, 2 padding only, 3 element by element."""
    if p >= p1 or p + V <= cs:
        return 0
    j = lay.lookup(p)
    end = lay.end[j] if j >= 0 else -(1 << 62)
    if p >= cs and p + V <= ce:
        if j >= 0 and p + V <= end:
            return 1
        if p >= end and lay.lookup(p + V - 1) == j:
            return 2
    return 3


def whole_tile(lay, p0, tile, cs, ce):
    if p0 < cs or p0 + tile > ce:
        return False
    j0, j1 = lay.lookup(p0), lay.lookup(p0 + tile - 1)
    return j0 == j1 and j0 >= 0 and lay.off[j0] <= p0 and p0 + tile <= lay.end[j0]


def copy_launch(kind, n, count, numel, offset, tensor_es, buf_es, ring, skip_sender=False, cfg=None, blocks=None,
                k=K):
    """One launch of pack_kernel ("pack") or unpack_kernel ("unpack"), plain or fused
    with a ring step.  blocks: optional list of (bx, y, z) to replay (a pair launch's
    share); otherwise the whole grid.  Returns (buf_writes (n, count), tensor_writes
    list per rank of per-tensor arrays, buf_reads (n, count))."""
    cfg = cfg or (PACK_CFG if kind == "pack" else UNPACK_CFG)
    V = vec_elems(tensor_es, buf_es)
    tile = cfg.tile_vecs * V
    lay = Layout(numel, offset)
    q, rem = divmod(count, n)
    rpb = ranks_per_block(cfg, n)
    gx, gy, gz = copy_grid(cfg, ring, count, V, n)
    bw = np.zeros((n, count), np.int64)
    br = np.zeros((n, count), np.int64)
    tw = [[np.zeros(m, np.int64) for m in numel] for _ in range(n)]
    if blocks is None:
        blocks = [(x, y, z) for x in range(gx) for y in range(gy) for z in range(gz)]
    for bx, y, z in blocks:
        c = y if ring else 0
        group = z if ring else y
        p0, p1, cs, ce, rbeg, rend = block_span(ring, tile, count, n, rpb, q, rem, group, bx, c, k)
        if p0 >= p1:
            continue
        rot = c if (ring and kind == "pack") else 0
        ranks = [(v + rot) % n for v in range(rbeg, rend)]
        if kind == "pack":
            written = [r for v, r in zip(range(rbeg, rend), ranks) if not (ring and skip_sender and v == k.skip_slot)]
        else:
            receiver = (c + n - 2) % n if ring else -1
        pos = tile_positions(cfg, p0, V, k)
        if whole_tile(lay, p0, tile, cs, ce):
            j = lay.lookup(p0)
            li = (pos - lay.off[j])[:, None] + np.arange(V)[None, :]
            for r in (written if kind == "pack" else ranks):
                if kind == "pack":
                    add(bw[r], pos[:, None] + np.arange(V)[None, :])
                else:
                    add(tw[r][j], li)
                    frm = (r + k.receiver_from) % n if r == receiver else r
                    add(br[frm], pos[:, None] + np.arange(V)[None, :], "read")
            continue
        for p in pos:
            cls = classify(lay, int(p), V, p1, cs, ce)
            if cls == 0:
                continue
            if cls in (1, 2):
                for r in (written if kind == "pack" else ranks):
                    if kind == "pack":
                        add(bw[r], np.arange(p, p + V))
                    elif cls == 1:
                        j = lay.lookup(p)
                        add(tw[r][j], np.arange(p - lay.off[j], p - lay.off[j] + V))
                        frm = (r + k.receiver_from) % n if r == receiver else r
                        add(br[frm], np.arange(p, p + V), "read")
                continue
            for e in range(int(p), int(p) + V):
                if e >= ce:
                    break
                if e < cs:
                    continue
                j = lay.lookup(e)
                inside = j >= 0 and e < lay.end[j]
                for r in (written if kind == "pack" else ranks):
                    if kind == "pack":
                        add(bw[r], [e])
                    elif inside:
                        add(tw[r][j], [e - lay.off[j]])
                        frm = (r + k.receiver_from) % n if r == receiver else r
                        add(br[frm], [e], "read")
    return bw, tw, br


def copy_pair_launch(kind, n, buckets, tensor_es, buf_es, k=K):
    """A pair kernel of the fused copies: bucket 0's chunk-tile columns, then bucket 1's.
    buckets: two (count, numel, offset).  Returns per bucket what copy_launch returns."""
    cfg = PACK_CFG if kind == "pack" else UNPACK_CFG
    V = vec_elems(tensor_es, buf_es)
    g = [copy_grid(cfg, True, b[0], V, n) for b in buckets]
    x0 = g[0][0] + k.pair_split
    gx, gy, gz = g[0][0] + g[1][0], n, g[0][2]
    per = [[], []]
    for col in range(gx):
        b = 1 if col >= x0 else 0
        for y in range(gy):
            for z in range(gz):
                per[b].append((col - b * x0, y, z))
    return [copy_launch(kind, n, *buckets[b], tensor_es, buf_es, True, skip_sender=True, blocks=per[b], k=k)
            for b in range(2)]


def small_cycle_threads(n, count, numel, offset, V, k=K):
    """small_cycle_kernel: per buffer position, the thread that takes it through the
    copy-in, every ring step and the copy-out (-1 for padding that no thread touches),
    and per rank and tensor how often each tensor element is written back."""
    cfg = SMALL_CFG
    tile = cfg.tile_vecs * V
    lay = Layout(numel, offset)
    owner = np.full(count, -1, np.int64)
    clash = False
    tw = [[np.zeros(m, np.int64) for m in numel] for _ in range(n)]
    blocks = (count + tile - 1) // tile
    for bx in range(blocks):
        p0 = bx * tile
        p1 = min(p0 + tile, count)
        for t in range(cfg.BS):
            p = p0 + (t + k.lane_shift) * V
            cls = classify(lay, p, V, p1, 0, count)
            tid = bx * cfg.BS + t
            if cls == 1:
                j = lay.lookup(p)
                clash |= bool((owner[p : p + V] >= 0).any())
                owner[p : p + V] = tid
                for r in range(n):
                    add(tw[r][j], np.arange(p - lay.off[j], p - lay.off[j] + V))
            elif cls == 3:
                for e in range(p, min(p + V, count)):
                    j = lay.lookup(e)
                    if j < 0 or e >= lay.end[j]:
                        continue
                    clash |= bool(owner[e] >= 0)
                    owner[e] = tid
                    for r in range(n):
                        add(tw[r][j], [e - lay.off[j]])
    return owner, clash, tw


def chain_threads(count, V, n, fold=False, k=K):
    """chain_kernel (or, with fold, fold_kernel's grid): how many threads take each
    element (grid-stride over V-element vectors, one thread per vector)."""
    nv = (count + V - 1) // V
    if fold:
        blocks = min(max((count // 4 + 256) // 256, 1), 1 << 20)
    else:
        blocks = min(max((nv + 255) // 256, 1), 65536)
    hits = np.zeros(count, np.int64)
    i = np.arange(blocks * 256, dtype=np.int64) + k.lane_shift
    while (i < nv).any():
        for e0 in (i[i < nv] * V):
            add(hits, np.arange(e0, min(e0 + V, count)))
        i = i + blocks * 256
    return hits


def bcast_step(n, nbytes, root, step, k=K):
    """bcast_step_kernel: (writes, reads) per rank over the buffer's bytes."""
    units = (nbytes + 15) // 16
    q, rem = divmod(units, n)
    w = np.zeros((n, nbytes), np.int64)
    rd = np.zeros((n, nbytes), np.int64)
    longest = q + (1 if rem else 0)
    gx = min(max((longest + 256 * 2 - 1) // (256 * 2), 1), 1 << 20)
    for kk in range(n - 1):
        j = step - kk
        if j < 0 or j >= n:
            continue
        src, dst = (root + kk) % n, (root + kk + 1) % n
        u0, cnt = chunk(j, q, rem)
        lo, hi = min(u0 * 16, nbytes), min((u0 + cnt) * 16, nbytes)
        full = (hi - lo) // 16
        for bx in range(gx):
            base = bx * 256 * 2 + np.arange(256) + k.lane_shift
            while (base < full).any():
                for u in range(2):
                    idx = base + u * 256
                    idx = idx[idx < full]
                    b = (lo + idx[:, None] * 16 + np.arange(16)[None, :]).reshape(-1)
                    add(w[dst], b)
                    add(rd[src], b, "read")
                base = base + gx * 256 * 2
            e = lo + full * 16 + bx * 256 + np.arange(256)
            e = e[e < hi]
            add(w[dst], e)
            add(rd[src], e, "read")
    return w, rd


def bcast_tensors_step(n, nbytes, root, step, k=K):
    """bcast_tensors_step_kernel over the tensors' virtual byte space (16-byte aligned
    starts).  Returns (writes, reads) per rank, per tensor byte arrays."""
    starts, end = [], 0
    for b in nbytes:
        s = -(-end // 16) * 16
        starts.append(s)
        end = s + b
    total = end
    lay = Layout(nbytes, starts)
    units = (total + 15) // 16
    q, rem = divmod(units, n)
    w = [[np.zeros(b, np.int64) for b in nbytes] for _ in range(n)]
    rd = [[np.zeros(b, np.int64) for b in nbytes] for _ in range(n)]
    tile = BCAST_CFG.tile_vecs * 16
    gx = max((((q + (1 if rem else 0)) * 16) + tile - 1) // tile, 1)
    for kk in range(n - 1):
        j = step - kk
        if j < 0 or j >= n:
            continue
        src, dst = (root + kk) % n, (root + kk + 1) % n
        u0, cnt = chunk(j, q, rem)
        lo, hi = min(u0 * 16, total), min((u0 + cnt) * 16, total)
        for bx in range(gx):
            p0 = lo + bx * tile
            if p0 >= hi:
                continue
            p1 = min(p0 + tile, hi)
            for p in tile_positions(BCAST_CFG, p0, 16, k):
                if p >= p1:
                    continue
                t = lay.lookup(p)
                if t < 0 or p >= lay.end[t]:
                    continue
                stop = min(p + 16, lay.end[t], p1)
                add(w[dst][t], np.arange(p - starts[t], stop - starts[t]))
                add(rd[src][t], np.arange(p - starts[t], stop - starts[t]), "read")
    return w, rd


# ---- the fused copies driven by tile tables (pack_tiles_kernel, unpack_tiles_kernel) ----
def tile_lanes(length, V, aligned, U=1):
    """Element indices (tile-relative) each lane of a 256-thread block takes, with repetition:
    U V-element vectors per lane, 256 vectors apart (the lane holding the last, partial
    vector finishes it element by element), or, when the copies are not vector-aligned,
    elements strided by the block."""
    out = []
    for t in range(256):
        if aligned:
            for u in range(U):
                i = (u * 256 + t) * V
                out.extend(range(i, min(i + V, length)) if i < length else [])
        else:
            out.extend(range(t, length, 256))
    return np.asarray(out, np.int64)


def tiled_copy(kind, n, count, numel, tiles, V, aligned=True, U=1, k=K):
    """pack_tiles_kernel ("pack": grid (tiles, n-1 slots), slot y = rank chunk+1+y) or
    unpack_tiles_kernel ("unpack": grid (tiles, n ranks), the chunk's last-step receiver
    reading its sender's buffer).  tiles: (pos, li, tensor, len, chunk) rows.
    Returns (buf_writes (n, count), tensor_writes per rank and tensor, buf_reads (n, count))."""
    bw = np.zeros((n, count), np.int64)
    br = np.zeros((n, count), np.int64)
    tw = [[np.zeros(m, np.int64) for m in numel] for _ in range(n)]
    for pos, li, t, length, c in tiles:
        assert length <= 256 * U * V, "a tile longer than a block takes"
        e = tile_lanes(length, V, aligned, U) + k.lane_shift
        if kind == "pack":
            for y in range(n - 1):
                r = (c + 1 + y) % n
                add(bw[r], pos + e)
        else:
            rc = (c - 2) % n
            for r in range(n):
                frm = (r + k.receiver_from) % n if r == rc else r
                add(tw[r][t], li + e)
                add(br[frm], pos + e, "read")
    return bw, tw, br


# ---- replacing steps into the tensors (rs_ag_tiles_kernel, ag_tiles_kernel) -----------
def tiled_replace(kind, n, count, numel, tiles, V, step=0, aligned=True, U=1, k=K, tpb=2):
    """rs_ag_tiles_kernel ("rs_ag": adding step N-2 and replacing step 0, from the owner's
    and sender's buffers into the owner's and rank c's tensors; grid (tiles)) or
    ag_tiles_kernel ("ag": replacing step `step`, rank c-1+step's tensors into rank
    c+step's; grid (ceil(tiles / tpb)), block b taking tiles b*tpb .. b*tpb+tpb-1), over
    the copy-out's tiles (padding tiles skipped).
    Returns (tensor_writes, tensor_reads per rank and tensor, buf_reads (n, count))."""
    tw = [[np.zeros(m, np.int64) for m in numel] for _ in range(n)]
    tr = [[np.zeros(m, np.int64) for m in numel] for _ in range(n)]
    br = np.zeros((n, count), np.int64)
    order = block_tiles(len(tiles), 1 if kind == "rs_ag" else tpb, 0 if kind == "rs_ag" else k.tile_block_stride, k)
    for g in order:
        pos, li, t, length, c = tiles[g]
        assert length <= 256 * U * V, "a tile longer than a block takes"
        if t < 0:
            continue
        e = tile_lanes(length, V, aligned, U) + k.lane_shift
        if kind == "rs_ag":
            own = (c - 1) % n
            snd = (own - 1) % n
            add(br[own], pos + e, "read")
            add(br[snd], pos + e, "read")
            add(tw[own][t], li + e)
            add(tw[(c + k.rs_ag_next) % n][t], li + e)
        else:
            snd = (c + step + k.replace_sender) % n
            add(tr[snd][t], li + e, "read")
            add(tw[(snd + 1) % n][t], li + e)
    return tw, tr, br


# ---- the whole cycle with the adding steps from the tensors, as data -------------------
def tile_block(b, grid, k=K):
    """tile_block(): the blocks of one XCD (b mod 8) take one contiguous run."""
    q, r = divmod(grid, 8)
    x = (b + k.xcd_shift) % 8
    return x * q + min(x, r) + b // 8


def block_tiles(ntiles, tpb, stride=0, k=K):
    """Tile indices in the order a grid of ceil(ntiles / tpb) blocks takes them, block b
    taking tiles tile_block(b)*tpb + j (with a planted stride, *stride + j)."""
    st = stride or tpb
    grid = -(-ntiles // tpb)
    return [g for b in range(grid) for g in (tile_block(b, grid, k) * st + j for j in range(tpb)) if g < ntiles]


class Launch:
    """Reads and writes of one launch on named arrays, applied after the launch, with the
    check that no element is both read and written by it (no order between its blocks)."""

    def __init__(self):
        self.reads, self.writes = [], []

    def read(self, arr, idx):
        self.reads.append((id(arr), arr, np.asarray(idx, np.int64)))
        return arr[idx]

    def write(self, arr, idx, val):
        self.writes.append((id(arr), arr, np.asarray(idx, np.int64), np.asarray(val)))

    def commit(self):
        written = {}
        for key, arr, idx, _ in self.writes:
            m = written.setdefault(key, np.zeros(arr.size, np.int64))
            np.add.at(m, idx, 1)
        for m in written.values():
            assert (m <= 1).all(), "an element written twice by one launch"
        for key, arr, idx in self.reads:
            if key in written:
                assert not written[key][idx].any(), "an element read and written by one launch"
        for _, arr, idx, val in self.writes:
            arr[idx] = val


def ring_bucket(ends, g, k=K):
    """ring_bucket(): the bucket whose tiles [ends[b-1], ends[b]) hold the launch's tile g."""
    b = 0
    for i in range(1, len(ends)):
        if g >= ends[i - 1] + k.bucket_end_shift:
            b = i
    return b, g - (ends[b - 1] if b else 0)


def dataflow_cycle(n, count, numel, tin, tout, V, U=1, aligned=True, k=K, tpb=2):
    """dataflow_group for one bucket; returns its ranks' tensors."""
    return dataflow_group(n, [(count, numel, tin, tout)], V, U, aligned, k, tpb)[0]


def dataflow_group(n, buckets, V, U=1, aligned=True, k=K, tpb=2):
    """The cycle with HVDX_TILED_REPLACE_IN_TENSORS | HVDX_TILED_ADD_FROM_TENSORS of one to
    four buckets (count, numel, copy-in tiles, copy-out tiles) sharing every launch, on
    values that record which ranks' inputs they hold (bit r for rank r): add_tiles_kernel
    for adding steps 0..N-3 over the copy-in tiles, rs_ag_tiles_kernel<..., OWN_T> and
    ag_tiles_kernel over the copy-out tiles, each launch's reads and writes replayed from
    the kernels' index arithmetic (the launch's tiles are the buckets' tables one after
    another).  Checks that no launch reads what it writes, that each adding step reads a
    rank's own elements while they still hold its input, that no value is counted twice,
    that the fused step completes every sum and that the replacing steps forward only
    complete sums.  Returns every bucket's ranks' tensors."""
    full = (1 << n) - 1
    T = [[[np.full(m, 1 << r, np.int64) for m in numel] for r in range(n)] for _, numel, _, _ in buckets]
    B = [[np.zeros(count, np.int64) for _ in range(n)] for count, _, _, _ in buckets]

    def launch_tiles(which, per_block):
        tabs = [bk[2] if which == "in" else bk[3] for bk in buckets]
        ends = list(np.cumsum([len(t) for t in tabs]))
        for g in block_tiles(int(ends[-1]), per_block, k.tile_block_stride if per_block > 1 else 0, k):
            b, loc = ring_bucket(ends, g, k)
            if loc >= len(tabs[b]):
                raise IndexError(f"tile {loc} of bucket {b} past its table")
            yield b, tabs[b][loc]

    for step in range(n - 2):
        L = Launch()
        for b, (pos, li, t, length, c) in launch_tiles("in", tpb):
            if t < 0:
                continue
            e = tile_lanes(length, V, aligned, U) + k.lane_shift
            snd = (c + step + k.add_sender) % n
            rcv = (snd + 1) % n
            own = L.read(T[b][rcv][t], li + e)
            assert (own == 1 << rcv).all(), f"step {step}: rank {rcv}'s own elements no longer its input"
            sent = L.read(T[b][snd][t], li + e) if step == 0 else L.read(B[b][snd], pos + e)
            assert not (own & sent).any(), f"step {step}: a rank's value counted twice"
            L.write(B[b][rcv], pos + e, own | sent)
        L.commit()
    L = Launch()
    for b, (pos, li, t, length, c) in launch_tiles("out", 1):
        e = tile_lanes(length, V, aligned, U) + k.lane_shift
        own = (c - 1) % n
        snd = (own - 1) % n
        # the owner's elements: each read and then overwritten by the same lane, so not a
        # read of the launch's own output (kept out of the race check)
        mine = B[b][own][pos + e] if k.fused_own_from_buffer else T[b][own][t][li + e]
        sent = L.read(B[b][snd], pos + e)
        assert not (mine & sent).any() and ((mine | sent) == full).all(), "the fused step's sum is not complete"
        L.write(T[b][own][t], li + e, mine | sent)
        L.write(T[b][c][t], li + e, mine | sent)
    L.commit()
    for step in range(1, n - 1):
        L = Launch()
        for b, (pos, li, t, length, c) in launch_tiles("out", tpb):
            e = tile_lanes(length, V, aligned, U) + k.lane_shift
            snd = (c + step + k.replace_sender) % n
            v = L.read(T[b][snd][t], li + e)
            assert (v == full).all(), f"replacing step {step} forwards an incomplete sum"
            L.write(T[b][(snd + 1) % n][t], li + e, v)
        L.commit()
    return T
