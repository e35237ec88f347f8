"""Timeline host logic: the per-rank chunk labels follow the ring schedule, and the
C entry points refuse misuse without touching the GPU."""
import pytest

import paper_1802_05799_amd as hv
from oracle import ring
from paper_1802_05799_amd.timeline import chunks_of_step


def test_chunk_labels_follow_the_oracle_schedule():
    for n in (2, 3, 5, 8, 17):
        for s in range(n - 1):
            for r in range(n):
                sent, recv = chunks_of_step(hv._lib.KERNEL_REDUCE_SCATTER, s, r, n)
                assert ring.rs_sender(sent, s, n) == r and ring.rs_receiver(sent, s, n) == (r + 1) % n
                assert ring.rs_receiver(recv, s, n) == r and ring.rs_sender(recv, s, n) == (r - 1) % n
                sent, recv = chunks_of_step(hv._lib.KERNEL_ALLGATHER, s, r, n)
                assert ring.ag_sender(sent, s, n) == r and ring.ag_receiver(sent, s, n) == (r + 1) % n
                assert ring.ag_receiver(recv, s, n) == r and ring.ag_sender(recv, s, n) == (r - 1) % n


def test_timeline_refuses_misuse():
    with pytest.raises(hv.HvdxError):
        hv.hvdx_timeline_end(4)  # nothing recording
    with pytest.raises(hv.HvdxError):
        hv.hvdx_timeline_begin(0)
    with pytest.raises(hv.HvdxError):
        hv.hvdx_timeline_begin(-5)


def test_broadcast_labels_follow_the_oracle_chain():
    import numpy as np

    from oracle import broadcast
    from paper_1802_05799_amd.timeline import broadcast_step_args

    for n in (2, 3, 5):
        for root in range(n):
            x = np.zeros((n, 16 * n), np.uint8)
            for r in range(n):
                x[r] = r + 1
            chunks = broadcast.chunk_bytes(16 * n, n)
            prev = x.copy()
            seen = []
            broadcast.chain_broadcast(x, root, observe=lambda s, b: seen.append(b.copy()))
            for s, cur in enumerate(seen):
                for r in range(n):
                    args = broadcast_step_args(s, r, root, n)
                    changed = [j for j, (lo, hi) in enumerate(chunks) if not np.array_equal(cur[r, lo:hi], prev[r, lo:hi])]
                    if changed:
                        assert args.get("recv chunk") == changed[0] and len(changed) == 1
                prev = cur
