"""GPU broadcast chain against the oracle: every step's state, the final bytes, edges."""
import numpy as np
import pytest
import torch

import paper_1802_05799_amd as hv
from _gpu import assert_bits_equal, say
from oracle import broadcast

pytestmark = pytest.mark.gpu


def rank_buffers(x, offset=0, guard=64):
    """One byte buffer per row of x, each `offset` bytes into an allocation with guards."""
    bases, views = [], []
    for row in x:
        base = torch.full((row.size + offset + 2 * guard,), 0xA5, dtype=torch.uint8, device="cuda")
        v = base[guard + offset : guard + offset + row.size]
        v.copy_(torch.from_numpy(row))
        bases.append(base)
        views.append(v)
    return bases, views


@pytest.mark.parametrize("offset", [0, 3])
def test_broadcast_steps_and_result(offset):
    rng = np.random.default_rng(400)
    for n, nbytes, root in ((2, 1, 0), (3, 40, 1), (4, 1000, 3), (7, 4099, 2), (8, 1 << 20, 0), (16, 12345, 9),
                            (64, 100003, 63), (128, 70000, 5)):
        say(f"broadcast n={n} nbytes={nbytes} root={root} offset={offset}")
        x = rng.integers(0, 256, size=(n, nbytes), dtype=np.uint8)
        bases, views = rank_buffers(x, offset)
        ptrs = [v.data_ptr() for v in views]

        def gpu_step(s, want):  # one GPU step per oracle step, compared at once
            hv.hvdx_broadcast_step(ptrs, n, nbytes, root, s)
            torch.cuda.synchronize()
            assert_bits_equal(np.stack([v.cpu().numpy() for v in views]), want, f"step {s}")

        broadcast.chain_broadcast(x.copy(), root, observe=gpu_step)
        for b in bases:  # guards untouched
            g = b.cpu().numpy()
            assert np.all(g[: 64 + offset] == 0xA5) and np.all(g[64 + offset + nbytes :] == 0xA5)
        # the whole call from fresh inputs
        bases, views = rank_buffers(x, offset)
        hv.hvdx_broadcast([v.data_ptr() for v in views], n, nbytes, root)
        torch.cuda.synchronize()
        assert_bits_equal(np.stack([v.cpu().numpy() for v in views]), np.broadcast_to(x[root], x.shape).copy())


def test_broadcast_tensors_helper():
    rng = np.random.default_rng(401)
    shapes = [(7,), (3, 3, 16, 32), (1000,), (2048, 1000), (1,)]
    for dtype in (torch.float32, torch.float16):
        per_rank = [[torch.from_numpy(rng.standard_normal(s).astype(np.float32)).to(dtype).cuda() for s in shapes]
                    for _ in range(5)]
        want = [t.clone() for t in per_rank[2]]
        hv.broadcast_(per_rank, root=2)
        torch.cuda.synchronize()
        for r in range(5):
            for t, w in zip(per_rank[r], want):
                assert torch.equal(t.view(torch.int16 if dtype == torch.float16 else torch.int32),
                                   w.view(torch.int16 if dtype == torch.float16 else torch.int32))


# ---- many tensors in one call: hvdx_broadcast_tensors (reading B2) ---------------------
def tensor_views(x_rows, sizes, offsets, guard=48):
    """Rank r's tensors as uint8 views, tensor t `offsets[t]` bytes past a 256-byte
    aligned start inside its own guarded allocation.  Returns (bases, views)."""
    bases, views = [], []
    for row in x_rows:
        rb, rv = [], []
        for a, s, off in zip(row, sizes, offsets):
            base = torch.full((s + off + 2 * guard,), 0x5A, dtype=torch.uint8, device="cuda")
            v = base[guard + off : guard + off + s]
            if s:
                v.copy_(torch.from_numpy(a))
            rb.append(base)
            rv.append(v)
        bases.append(rb)
        views.append(rv)
    return bases, views


def host_state(views):
    """Every rank's tensors on the host, moved in one copy."""
    flat = [v for row in views for v in row]
    allb = torch.cat(flat).cpu().numpy() if flat else np.zeros(0, np.uint8)
    out, at = [], 0
    for row in views:
        rr = []
        for v in row:
            rr.append(allb[at : at + v.numel()])
            at += v.numel()
        out.append(rr)
    return out


TENSOR_CASES = [
    # (ranks, tensor sizes in bytes, byte offset of each tensor in its allocation, root)
    (2, [1], [0], 1),
    (3, [10, 20], [0, 0], 1),  # the hand-worked case of the oracle's golden file
    (3, [5, 16, 0, 33, 1], [0, 0, 0, 0, 0], 0),  # an empty tensor; units shared by no two tensors
    (4, [4096, 100, 70001, 3, 0, 12288], [0, 0, 0, 0, 0, 0], 2),
    (5, [4096, 100, 70001, 3, 12288], [1, 4, 8, 3, 12], 4),  # unaligned copies: the byte path
    (8, [8192] * 6 + [16, 1 << 18, 7], [0] * 9, 0),  # whole tiles inside one tensor
    (13, [30000, 40000, 123, 8191, 8193], [0, 0, 0, 0, 0], 7),
    (128, [5000, 64, 100000, 9], [0, 0, 0, 0], 127),
]


@pytest.mark.parametrize("case", range(len(TENSOR_CASES)))
def test_broadcast_tensors_steps_and_result(case):
    n, sizes, offsets, root = TENSOR_CASES[case]
    say(f"tensor broadcast case {case}: n={n} sizes={sizes[:6]} offsets={offsets[:6]} root={root}")
    rng = np.random.default_rng(900 + case)
    x = [[rng.integers(0, 256, size=s, dtype=np.uint8) for s in sizes] for _ in range(n)]
    bases, views = tensor_views(x, sizes, offsets)
    tb = hv.TensorBroadcast(views)
    assert tb.total == broadcast.tensor_layout(sizes)[1]

    def gpu_step(s, want):
        tb.step(root, s)
        torch.cuda.synchronize()
        got = host_state(views)
        for r in range(n):
            for t in range(len(sizes)):
                assert_bits_equal(got[r][t], want[r][t], f"step {s} rank {r} tensor {t}")

    broadcast.chain_broadcast_tensors([[a.copy() for a in row] for row in x], root, observe=gpu_step)
    for r in range(n):  # guard bytes around every tensor untouched
        for t, (s, off) in enumerate(zip(sizes, offsets)):
            g = bases[r][t].cpu().numpy()
            assert np.all(g[: 48 + off] == 0x5A) and np.all(g[48 + off + s :] == 0x5A), (r, t)
    # the whole call from fresh inputs
    bases, views = tensor_views(x, sizes, offsets)
    hv.TensorBroadcast(views)(root)
    torch.cuda.synchronize()
    got = host_state(views)
    for r in range(n):
        for t in range(len(sizes)):
            assert_bits_equal(got[r][t], x[root][t], f"whole call rank {r} tensor {t}")


def test_broadcast_resnet50_parameters():
    """broadcast_ over ResNet-50's 161 parameter tensors of 8 ranks (one chain for all),
    every byte against the root's."""
    from workloads import configs
    from workloads import gpu as wgpu

    w = configs.get("resnet50")
    say("tensor broadcast: resnet50 parameters, 8 ranks")
    per_rank, storage, starts = wgpu.make_rank_tensors(w)
    want = storage[3].clone()
    hv.broadcast_(per_rank, root=3)
    torch.cuda.synchronize()
    numel = w.numel()
    for r in range(w.nranks):
        for s, m in zip(starts, numel):
            if not torch.equal(storage[r][s : s + m].view(torch.int32), want[s : s + m].view(torch.int32)):
                raise AssertionError(f"rank {r} tensor at {s} differs")
    # rank storages outside the tensors (the 256-byte alignment gaps) stay zero
    mask = torch.ones_like(storage[0], dtype=torch.bool)
    for s, m in zip(starts, numel):
        mask[s : s + m] = False
    assert all(bool((x[mask] == 0).all()) for x in storage)
