"""Which elements every kernel launch writes (CPU models of the launchers' grids and the
kernels' index arithmetic, tests/_writesets.py): in each ring step every element of a
receiving chunk is written exactly once and nothing else is (paper section 3: one
message per chunk and step, so one writer per element), no element is both read as a
sender's value and written in the same step, the copies write every buffer or tensor
element once, and the broadcast chain writes each byte of a link's chunk once.  Each
check also rejects a planted index mistake."""
import numpy as np
import pytest

import _writesets as W

RING_CASES = [(2, 1), (2, 37), (3, 7), (3, 1001), (4, 3), (5, 4 * 5 + 3), (7, 32781), (8, 4096 * 8 + 13),
              (13, 100003)]


def owner_mask(kind, n, count, step):
    """(n, count) 1 where the paper's schedule writes in this step (reading R1)."""
    q, rem = divmod(count, n)
    m = np.zeros((n, count), np.int64)
    for c in range(n):
        s, length = W.chunk(c, q, rem)
        if kind == "rs":
            m[(c + step + 1) % n, s : s + length] += 1
        elif kind == "ag":
            m[(c + step) % n, s : s + length] += 1
        else:
            m[(c + n - 1) % n, s : s + length] += 1
            m[c, s : s + length] += 1
    return m


def check_ring(kind, n, count, step, esize, **kw):
    writes, sreads, oreads = W.ring_step(kind, n, count, step, esize, **kw)
    want = owner_mask(kind, n, count, step)
    if not np.array_equal(writes, want):
        return "writes"
    if n >= 3 and ((writes > 0) & (sreads > 0)).any():
        return "read as a sender and written in one step"
    if kind != "ag" and not np.array_equal(oreads > 0, owner_mask("rs", n, count, step if kind == "rs" else n - 2) > 0):
        return "own reads"
    return None


@pytest.mark.parametrize("esize", [4, 2], ids=["binary32", "binary16"])
@pytest.mark.parametrize("kind", ["rs", "ag", "rs_ag"])
def test_ring_steps_write_each_receiving_element_once(kind, esize):
    for n, count in RING_CASES:
        steps = [n - 2] if kind == "rs_ag" else sorted({0, (n - 2) // 2, n - 2, max(n - 3, 0)})
        for step in steps:
            assert check_ring(kind, n, count, step, esize) is None, (n, count, step)


@pytest.mark.parametrize("policy", [W.RS_CACHED, W.RS_STREAM, W.AG_CACHED, W.RSAG_CACHED, W.Policy(4, 256),
                                    W.Policy(2, 512, True)], ids=str)
def test_every_launch_shape_and_alignment(policy):
    """Each shape the launchers use (and two wider ones) on unaligned chunk starts, on
    misaligned buffers (vectors then start after a scalar head), and on buffers the
    kernels must treat element by element."""
    for n, count in ((3, 4099), (5, 70001), (8, 3 * 2048 + 5)):
        for mis, vec_ok in (([0] * n, True), ([4 * (r % 4) for r in range(n)], True), ([2] * n, False)):
            for kind in ("rs", "ag", "rs_ag"):
                step = n - 2 if kind == "rs_ag" else 1
                assert check_ring(kind, n, count, step, 4, mis=mis, vec_ok=vec_ok, policy=policy) is None


def test_streaming_shape_is_picked_by_rank_buffer_bytes():
    """(q+1) * N * esize >= 128 MiB: VGG-16's fc6 streams at 32 and 64 ranks, the fusion
    buffers of the workloads do not."""
    for n, es in ((2, 4), (32, 4), (64, 2)):
        edge = (128 << 20) // (n * es) - 1  # the smallest q that streams
        assert W.streams(edge, n, es) and not W.streams(edge - 1, n, es)
    assert W.streams(102760448 // 32, 32, 4) and W.streams(102760448 // 64, 64, 4)
    assert not W.streams(16489448 // 8, 8, 4) and not W.streams(16777216 // 32, 32, 4)


def test_two_ring_launches_split_columns():
    for n, counts in ((3, (1000, 37)), (8, (4096 * 8 + 13, 100003)), (8, (3, 5)), (13, (70001, 70001)),
                      (5, (2 << 16, 1))):
        for kind, step in (("rs", 1), ("ag", 1), ("ag", n - 3), ("rs_ag", n - 2)):
            got = W.ring_pair_step(kind, n, counts, step, 4)
            for z in range(2):
                assert np.array_equal(got[z], owner_mask(kind, n, counts[z], step)), (n, counts, kind, z)


@pytest.mark.parametrize("kind", ["rs", "ag0", "rs_ag"])
def test_compressed_ring_steps(kind):
    for n, count in ((2, 37), (3, 1001), (4, 8 * 4096 + 5), (8, 70001)):
        step = {"rs": 1 % (n - 1), "ag0": 0, "rs_ag": n - 2}[kind]
        xw, ww = W.c16_step(kind, n, count, step)
        if kind == "rs":
            assert np.array_equal(ww, owner_mask("rs", n, count, step)) and not xw.any()
        elif kind == "ag0":  # owner c-1 and receiver c
            want = owner_mask("ag", n, count, 0) + owner_mask("ag", n, count, n - 1 if n > 1 else 0) * 0
            own = np.zeros_like(want)
            q, rem = divmod(count, n)
            for c in range(n):
                s, length = W.chunk(c, q, rem)
                own[(c - 1) % n, s : s + length] += 1
            assert np.array_equal(xw, want + own) and not ww.any()
        else:
            assert np.array_equal(xw, owner_mask("rs_ag", n, count, n - 2)) and not ww.any()


def plan(numel, esize, align):
    offs, count = [], 0
    a = align // esize
    for m in numel:
        s = -(-count // a) * a
        offs.append(s)
        count = s + m
    return offs, count


COPY_LAYOUTS = [
    [7, 64, 100, 1000, 4608, 4096, 513, 10000],  # the tiny workload's tensors
    [2048 * 3, 5, 4096 * 2 + 3, 1, 9000],
    [33] * 90 + [12000],  # more tensors in one tile than the LDS table holds
    [0, 17, 0, 4096, 2],  # empty tensors
]


@pytest.mark.parametrize("esizes", [(4, 4), (4, 2), (2, 2)], ids=["f32", "f32-to-f16", "f16"])
def test_copies_write_every_element_once(esizes):
    te, be = esizes
    for numel in COPY_LAYOUTS:
        for align in (16, be):  # the plan's 16-byte offsets, and unaligned ones (edge path)
            offset, count = plan(numel, be, align)
            for n in (1, 3, 5):
                bw, _, _ = W.copy_launch("pack", n, count, numel, offset, te, be, ring=False)
                assert (bw == 1).all(), ("pack", numel[:3], align, n)
                _, tw, _ = W.copy_launch("unpack", n, count, numel, offset, te, be, ring=False)
                assert all((x == 1).all() for row in tw for x in row), ("unpack", numel[:3], align, n)
                if n < 3:
                    continue
                q, rem = divmod(count, n)
                for skip in (False, True):
                    bw, _, _ = W.copy_launch("pack", n, count, numel, offset, te, be, ring=True, skip_sender=skip)
                    want = np.ones((n, count), np.int64)
                    if skip:  # the sender of chunk c (rank c) does not store its own copy
                        for c in range(n):
                            s, length = W.chunk(c, q, rem)
                            want[c, s : s + length] = 0
                    assert np.array_equal(bw, want), ("pack_rs", numel[:3], align, n, skip)
                _, tw, br = W.copy_launch("unpack", n, count, numel, offset, te, be, ring=True)
                assert all((x == 1).all() for row in tw for x in row), ("ag_unpack", numel[:3], align, n)
                # rank c-2 takes chunk c from its sender, rank c-3; no rank reads its own copy of it
                for c in range(n):
                    s, length = W.chunk(c, q, rem)
                    rcv = (c + n - 2) % n
                    assert not br[rcv, s : s + length].any(), ("ag_unpack reads the receiver", c)


def test_two_buffer_copies():
    b0 = [4096 * 2 + 3, 5, 700]
    b1 = [33] * 70 + [5000]
    for n in (3, 8):
        buckets = []
        for numel in (b0, b1):
            offset, count = plan(numel, 4, 16)
            buckets.append((count, numel, offset))
        for kind in ("pack", "unpack"):
            got = W.copy_pair_launch(kind, n, buckets, 4, 4)
            for (count, numel, offset), (bw, tw, _) in zip(buckets, got):
                if kind == "pack":
                    q, rem = divmod(count, n)
                    want = np.ones((n, count), np.int64)
                    for c in range(n):
                        s, length = W.chunk(c, q, rem)
                        want[c, s : s + length] = 0
                    assert np.array_equal(bw, want), (kind, n)
                else:
                    assert all((x == 1).all() for row in tw for x in row), (kind, n)


def test_small_cycle_one_thread_per_element():
    for numel in COPY_LAYOUTS[:2] + [[3, 1, 2]]:
        for be in (4, 2):
            offset, count = plan(numel, be, 16)
            for n in (2, 4, 7):
                owner, clash, tw = W.small_cycle_threads(n, count, numel, offset, W.vec_elems(4, be))
                assert not clash
                assert all((x == 1).all() for row in tw for x in row)
                inside = np.zeros(count, bool)
                for o, m in zip(offset, numel):
                    inside[o : o + m] = True
                assert (owner[inside] >= 0).all()


def test_one_launch_ring_and_fold_one_thread_per_element():
    for count in (1, 3, 4, 5, 1001, 65536 * 4 + 7, 256 * 4 * 3 + 1):
        assert (W.chain_threads(count, 4, 3) == 1).all()
        assert (W.chain_threads(count, 8, 5) == 1).all()
        assert (W.chain_threads(count, 4, 5, fold=True) == 1).all()


def test_broadcast_steps():
    for n, nbytes, root in ((2, 1, 1), (3, 40, 1), (4, 1000, 3), (7, 4099, 2), (8, 70001, 0)):
        total = np.zeros((n, nbytes), np.int64)
        for step in range(2 * n - 2):
            w, rd = W.bcast_step(n, nbytes, root, step)
            assert not ((w > 0) & (rd > 0)).any()  # a link's chunk is not what the next link sends now
            assert w.max(initial=0) <= 1
            total += w
        want = np.ones((n, nbytes), np.int64)
        want[root] = 0
        assert np.array_equal(total, want)


def test_tensor_broadcast_steps():
    for n, sizes, root in ((3, [10, 20], 1), (4, [4096, 100, 70001, 3, 0, 12288], 2), (5, [8192] * 3 + [7], 4)):
        total = [np.zeros((n, b), np.int64) for b in sizes]
        for step in range(2 * n - 2):
            w, rd = W.bcast_tensors_step(n, sizes, root, step)
            for t in range(len(sizes)):
                assert not any(((w[r][t] > 0) & (rd[r][t] > 0)).any() for r in range(n))
                for r in range(n):
                    total[t][r] += w[r][t]
        for t, b in enumerate(sizes):
            want = np.ones((n, b), np.int64)
            want[root] = 0
            assert np.array_equal(total[t], want), t


def test_buffers_past_2_to_31_elements():
    """The 2^31 + 4099-element rank buffers of the large GPU tests: grid sizes stay in
    range, and the vector spans of the first, middle and last blocks of each launch
    (streaming shape, grid capped at 2^20 blocks, several passes per block) are disjoint
    and tile [0, nvec) in the order the grid-stride loop takes them."""
    count, n = (1 << 31) + 4099, 3
    q, rem = divmod(count, n)
    for P in (W.RS_STREAM, W.AG_STREAM, W.RSAG_STREAM):
        gx = W.step_grid_x(q, rem, 4, P.U, P.BS)
        assert 1 <= gx <= 1 << 20
        for c in range(n):
            start, length = W.chunk(c, q, rem)
            head = W.head_elems((start * 4) % 16, 4, length)
            nvec = (length - head) // 4
            span = P.BS * P.U
            ntiles = -(-nvec // span)
            passes = -(-ntiles // gx)
            assert passes > 1 and start + length <= count < 1 << 62
            seen = []
            for bx in (0, 1, gx // 2, gx - 1):
                tiles = [bx + i * gx for i in range(passes) if bx + i * gx < ntiles]
                for tl in tiles:
                    seen.append((tl * span, min((tl + 1) * span, nvec)))
            seen.sort()
            assert all(a[1] <= b[0] for a, b in zip(seen, seen[1:]))
            assert seen[-1][1] <= nvec
    # the fused copy of one such tensor: tiles of 2048 elements, a grid that fits a 32-bit x
    V = 4
    tile = W.PACK_CFG.tile_vecs * V
    gx, gy, gz = W.copy_grid(W.PACK_CFG, True, count, V, n)
    assert gx < 1 << 31 and (gy, gz) == (n, 2)
    for c in range(n):  # the chunk's tiles, from the one holding its first element, reach its end
        cs, length = W.chunk(c, q, rem)
        assert (cs & ~(tile - 1)) + gx * tile >= cs + length


# ---- planted mistakes: each must be rejected ----------------------------------------------
def test_planted_lane_shift_is_caught():
    bad = W.Knobs(lane_shift=1)
    with pytest.raises((AssertionError, IndexError)):
        w, _, _ = W.ring_step("rs", 3, 4099, 1, 4, k=bad)
        assert np.array_equal(w, owner_mask("rs", 3, 4099, 1))


def test_pair_split_point_only_moves_work():
    """Any split of the columns covers both rings (each ring's grid-stride loop spans its
    own columns); an off-by-one in the second ring's own column index does not."""
    counts = (4096 * 8 * 9 + 13, 100003)
    for split in (-1, 1):
        got = W.ring_pair_step("ag", 8, counts, 1, 4, k=W.Knobs(pair_split=split))
        assert all(np.array_equal(got[z], owner_mask("ag", 8, c, 1)) for z, c in enumerate(counts))
    got = W.ring_pair_step("ag", 8, counts, 1, 4, k=W.Knobs(pair_column_shift=1))
    assert not all(np.array_equal(got[z], owner_mask("ag", 8, c, 1)) for z, c in enumerate(counts))


def test_planted_chunk_tile_skip_is_caught():
    numel = COPY_LAYOUTS[1]
    offset, count = plan(numel, 4, 16)
    bw, _, _ = W.copy_launch("pack", 3, count, numel, offset, 4, 4, ring=True, k=W.Knobs(chunk_tile_skip=1))
    assert not (bw == 1).all()


def test_planted_wrong_skipped_slot_is_caught():
    numel = COPY_LAYOUTS[0]
    offset, count = plan(numel, 4, 16)
    bw, _, _ = W.copy_launch("pack", 4, count, numel, offset, 4, 4, ring=True, skip_sender=True,
                             k=W.Knobs(skip_slot=1))
    q, rem = divmod(count, 4)
    s, length = W.chunk(0, q, rem)
    assert bw[0, s : s + length].any()  # the sender's own chunk is now stored: caught


def test_planted_copy_out_from_the_receiver_is_caught():
    numel = COPY_LAYOUTS[0]
    offset, count = plan(numel, 4, 16)
    _, _, br = W.copy_launch("unpack", 4, count, numel, offset, 4, 4, ring=True, k=W.Knobs(receiver_from=0))
    q, rem = divmod(count, 4)
    s, length = W.chunk(2, q, rem)
    assert br[0, s : s + length].any()  # rank 0 receives chunk 2 and reads its own copy: caught


# ---- tile-driven fused copies ----------------------------------------------------------
def lane_vectors(te, be):
    """Vectors per lane of the built tile kernels: a tile is what 256 lanes move."""
    import paper_1802_05799_amd as hv

    return hv.hvdx_fuse_tile_elems(0 if te == 4 else 1, 0 if be == 4 else 1) // (256 * W.vec_elems(te, be))


def tiles_of(numel, offset, count, te, be, n, direction):
    import paper_1802_05799_amd as hv

    arr, k = hv.hvdx_fuse_copy_tiles(numel, offset, count, 0 if te == 4 else 1, 0 if be == 4 else 1, n, direction)
    return [(x.pos, x.li, x.tensor, x.len, x.chunk) for x in arr[:k]]


@pytest.mark.parametrize("esizes", [(4, 4), (4, 2), (2, 2)], ids=["f32", "f32-to-f16", "f16"])
def test_tiled_copies_write_every_element_once(esizes):
    import paper_1802_05799_amd as hv

    te, be = esizes
    V = W.vec_elems(te, be)
    for numel in COPY_LAYOUTS + [[4096 * 3 + 1, 7, 2 * 4096 * 2]]:
        for align in (16, be):
            offset, count = plan(numel, be, align)
            for n in (3, 5, 8):
                q, rem = divmod(count, n)
                tin = tiles_of(numel, offset, count, te, be, n, hv.COPY_IN)
                tout = tiles_of(numel, offset, count, te, be, n, hv.COPY_OUT)
                U = lane_vectors(te, be)
                for aligned in (True, False):
                    bw, _, _ = W.tiled_copy("pack", n, count, numel, tin, V, aligned, U)
                    want = np.ones((n, count), np.int64)
                    for c in range(n):  # the sender of chunk c stores nothing there
                        s, length = W.chunk(c, q, rem)
                        want[c, s : s + length] = 0
                    assert np.array_equal(bw, want), ("pack", numel[:3], align, n, aligned)
                    _, tw, br = W.tiled_copy("unpack", n, count, numel, tout, V, aligned, U)
                    assert all((x == 1).all() for row in tw for x in row), ("unpack", numel[:3], align, n)
                    for c in range(n):
                        s, length = W.chunk(c, q, rem)
                        assert not br[(c - 2) % n, s : s + length].any()


def test_planted_tiled_lane_shift_is_caught():
    import paper_1802_05799_amd as hv

    numel = COPY_LAYOUTS[1]
    offset, count = plan(numel, 4, 16)
    tout = tiles_of(numel, offset, count, 4, 4, 3, hv.COPY_OUT)
    with pytest.raises((AssertionError, IndexError)):
        _, tw, _ = W.tiled_copy("unpack", 3, count, numel, tout, 4, True, k=W.Knobs(lane_shift=1))
        assert all((x == 1).all() for row in tw for x in row)


# ---- replacing steps delivered into the tensors -----------------------------------------
def replace_phase(n, count, numel, offset, tiles, V, aligned, U, k=W.K):
    """Runs the fused step and replacing steps 1..N-2 into the tensors on a model of which
    tensor elements hold their final value; checks each launch on the way.  Returns the
    final-value map."""
    q, rem = divmod(count, n)
    tw, _, br = W.tiled_replace("rs_ag", n, count, numel, tiles, V, aligned=aligned, U=U, k=k)
    for c in range(n):  # chunk c is read from its owner c-1 and sender c-2 only
        s, length = W.chunk(c, q, rem)
        readers = {r for r in range(n) if br[r, s : s + length].any()}
        assert readers <= {(c - 1) % n, (c - 2) % n}, (c, readers)
    assert all((x <= 1).all() for row in tw for x in row), "an element written twice by the fused step"
    final = [[x > 0 for x in row] for row in tw]
    for step in range(1, n - 1):
        tw, tr, _ = W.tiled_replace("ag", n, count, numel, tiles, V, step, aligned, U, k)
        for r in range(n):
            for t in range(len(numel)):
                assert not (tr[r][t] > 0)[~final[r][t]].any(), f"step {step} forwards what rank {r} lacks"
                assert not ((tw[r][t] > 0) & (tr[r][t] > 0)).any(), f"step {step} reads what it writes"
                assert not ((tw[r][t] > 0) & final[r][t]).any(), f"step {step} writes rank {r} twice"
                assert (tw[r][t] <= 1).all()
                final[r][t] |= tw[r][t] > 0
    return final


@pytest.mark.parametrize("esize", [4, 2], ids=["f32", "f16"])
def test_replacing_into_tensors_delivers_every_element_once(esize):
    import paper_1802_05799_amd as hv

    V = W.vec_elems(esize, esize)
    for numel in COPY_LAYOUTS + [[4096 * 3 + 1, 7, 2 * 4096 * 2]]:
        for align in (16, esize):
            offset, count = plan(numel, esize, align)
            for n in (3, 4, 7):
                tout = tiles_of(numel, offset, count, esize, esize, n, hv.COPY_OUT)
                for aligned in (True, False):
                    final = replace_phase(n, count, numel, offset, tout, V, aligned, 1)
                    assert all(x.all() for row in final for x in row), (numel[:3], align, n, aligned)


@pytest.mark.parametrize("knobs", [W.Knobs(replace_sender=0), W.Knobs(rs_ag_next=1), W.Knobs(lane_shift=1),
                                   W.Knobs(tile_block_stride=1)],
                         ids=["sender", "next-rank", "lane", "tiles-per-block"])
def test_planted_replacing_mistakes_are_caught(knobs):
    import paper_1802_05799_amd as hv

    numel = COPY_LAYOUTS[1]
    offset, count = plan(numel, 4, 16)
    tout = tiles_of(numel, offset, count, 4, 4, 5, hv.COPY_OUT)
    with pytest.raises((AssertionError, IndexError)):
        final = replace_phase(5, count, numel, offset, tout, 4, True, 1, knobs)
        assert all(x.all() for row in final for x in row)


# ---- the cycle with the adding steps from the tensors, as data --------------------------
@pytest.mark.parametrize("esizes", [(4, 4), (4, 2), (2, 2)], ids=["f32", "f32-to-f16", "f16"])
def test_cycle_from_and_into_tensors_sums_every_input_once(esizes):
    import paper_1802_05799_amd as hv

    te, be = esizes
    V = W.vec_elems(te, be)
    U = lane_vectors(te, be)
    for numel in COPY_LAYOUTS + [[4096 * 3 + 1, 7, 2 * 4096 * 2]]:
        for align in (16, be):
            offset, count = plan(numel, be, align)
            for n in (3, 4, 7):
                tin = tiles_of(numel, offset, count, te, be, n, hv.COPY_IN)
                tout = tiles_of(numel, offset, count, te, be, n, hv.COPY_OUT)
                for aligned in (True, False):
                    T = W.dataflow_cycle(n, count, numel, tin, tout, V, U, aligned)
                    full = (1 << n) - 1
                    assert all((x == full).all() for row in T for x in row), (numel[:3], align, n, aligned)


@pytest.mark.parametrize("knobs", [W.Knobs(add_sender=1), W.Knobs(fused_own_from_buffer=True),
                                   W.Knobs(replace_sender=0), W.Knobs(tile_block_stride=1), W.Knobs(lane_shift=1),
                                   W.Knobs(xcd_shift=1)],
                         ids=["adding-sender", "own-from-buffer", "replacing-sender", "tiles-per-block", "lane",
                              "xcd-runs"])
def test_planted_cycle_mistakes_are_caught(knobs):
    import paper_1802_05799_amd as hv

    numel = COPY_LAYOUTS[1]
    offset, count = plan(numel, 4, 16)
    tin = tiles_of(numel, offset, count, 4, 4, 5, hv.COPY_IN)
    tout = tiles_of(numel, offset, count, 4, 4, 5, hv.COPY_OUT)
    with pytest.raises((AssertionError, IndexError)):
        T = W.dataflow_cycle(5, count, numel, tin, tout, 4, 1, True, knobs)
        assert all((x == 31).all() for row in T for x in row)


def test_xcd_block_order_is_a_bijection():
    for grid in list(range(1, 70)) + [4099, (1 << 20) + 3]:
        assert sorted(W.tile_block(b, grid) for b in range(grid)) == list(range(grid))


def test_buckets_sharing_every_launch_each_sum_their_own_inputs():
    """Up to four buckets (as FusedAllreduce groups them) in every launch of the ring on
    the tensors: each tile finds its bucket from the running tile counts."""
    import paper_1802_05799_amd as hv

    layouts = [COPY_LAYOUTS[1], [4096 * 3 + 1, 7, 2 * 4096 * 2], [5, 1, 3000], COPY_LAYOUTS[0]]
    for te, be in ((4, 4), (4, 2)):
        V, U = W.vec_elems(te, be), lane_vectors(te, be)
        for nb in (2, 3, 4):
            for n in (3, 5):
                bk = []
                for numel in layouts[:nb]:
                    offset, count = plan(numel, be, 16)
                    bk.append((count, numel, tiles_of(numel, offset, count, te, be, n, hv.COPY_IN),
                               tiles_of(numel, offset, count, te, be, n, hv.COPY_OUT)))
                Ts = W.dataflow_group(n, bk, V, U)
                full = (1 << n) - 1
                assert all((x == full).all() for T in Ts for row in T for x in row), (te, be, nb, n)


def test_planted_bucket_boundary_is_caught():
    import paper_1802_05799_amd as hv

    bk = []
    for numel in (COPY_LAYOUTS[1], [5, 1, 3000]):
        offset, count = plan(numel, 4, 16)
        bk.append((count, numel, tiles_of(numel, offset, count, 4, 4, 4, hv.COPY_IN),
                   tiles_of(numel, offset, count, 4, 4, 4, hv.COPY_OUT)))
    with pytest.raises((AssertionError, IndexError)):
        Ts = W.dataflow_group(4, bk, 4, 1, True, W.Knobs(bucket_end_shift=1))
        assert all((x == 15).all() for T in Ts for row in T for x in row)
