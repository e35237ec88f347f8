"""The Tensor Fusion cycle replayed from a HIP graph, against the eager launches and the oracle.

Each case captures the cycle once, then several times: loads fresh inputs (eager
copies, with synchronizations), runs the eager cycle, reloads the same inputs,
replays the graph, and checks the replay bit for bit against the eager result and
the oracle's."""
import numpy as np
import pytest
import torch

import paper_1802_05799_amd as hv
from _gpu import assert_bits_equal, say
from oracle import allreduce

pytestmark = pytest.mark.gpu

GRAPH_CASES = [
    # (numel, nranks, threshold bytes, compress, op)
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 4, 64 << 20, False, "average"),  # the tiny workload
    ([7, 64, 100, 1000, 4608, 4096, 513, 10000], 3, 4096, True, "average"),  # buckets + compressed direct
    ([3000, 1, 2, 50000, 64, 64, 64, 128 * 1024, 9], 5, 40000, False, "sum"),
    ([1, 0, 33], 1, 64, True, "average"),  # one rank: copies and the compressed round trip
]


def load(dev, host):
    for r, row in enumerate(host):
        for t, x in enumerate(row):
            dev[r][t].copy_(torch.from_numpy(x))
    torch.cuda.synchronize()


def snapshot(dev):
    torch.cuda.synchronize()
    return [[x.cpu().numpy() for x in row] for row in dev]


@pytest.mark.parametrize("small_bytes", [0, hv.SMALL_BUCKET_BYTES], ids=["per-step", "one-launch"])
@pytest.mark.parametrize("case", range(len(GRAPH_CASES)))
def test_graph_replays_match_eager_and_oracle(case, small_bytes):
    numel, n, threshold, compress, op = GRAPH_CASES[case]
    say(f"graph case={case} n={n} threshold={threshold} compress={compress}")
    dev = [[torch.zeros(k, dtype=torch.float32, device="cuda") for k in numel] for _ in range(n)]
    ar = hv.FusedAllreduce(dev, op=op, compress=compress, threshold_bytes=threshold, small_bucket_bytes=small_bytes)
    graph = ar.capture()
    torch.cuda.synchronize()
    for rep in range(3):
        rng = np.random.default_rng(700 + 10 * case + rep)
        host = [[(rng.standard_normal(k) * 0.01).astype(np.float32) for k in numel] for _ in range(n)]
        load(dev, host)
        ar()
        eager = snapshot(dev)
        load(dev, host)
        graph.replay()
        got = snapshot(dev)
        want = allreduce.allreduce(host, op, compress=compress, threshold=threshold)
        for r in range(n):
            for t in range(len(numel)):
                assert_bits_equal(got[r][t], eager[r][t], f"replay {rep} vs eager, rank {r} tensor {t}")
                assert_bits_equal(got[r][t], want[r][t], f"replay {rep} vs oracle, rank {r} tensor {t}")


def test_graph_capture_leaves_no_timeline_records():
    dev = [[torch.zeros(1000, dtype=torch.float32, device="cuda")] for _ in range(4)]
    ar = hv.FusedAllreduce(dev)
    with hv.Timeline() as tl:
        graph = ar.capture()
        graph.replay()
        torch.cuda.synchronize()
    assert tl.records == [] and tl.dropped == 0
    with hv.Timeline() as tl:
        ar()
        torch.cuda.synchronize()
    assert len(tl.records) == len(ar.kernel_sequence())
