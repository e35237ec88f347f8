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
