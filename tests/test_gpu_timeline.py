"""The timeline on the GPU: one record per launch, in launch order, and a Chrome trace."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import paper_1802_05799_amd as hv
from _gpu import say

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def tensors(n, numel, seed=0):
    g = np.random.default_rng(seed)
    return [[torch.from_numpy((g.standard_normal(k) * 0.01).astype(np.float32)).cuda() for k in numel] for _ in range(n)]


MODES = {"fused-boundary": (True, True, True), "fused-boundary-copy-in": (True, True, False),
         "fused-boundary-buffers": (True, False, False), "separate": (False, True, True)}


@pytest.mark.parametrize("mode", list(MODES))
def test_records_follow_launches(mode):
    fuse_boundary, into, add = MODES[mode]
    say(f"timeline records {mode}")
    per_rank = tensors(5, [7, 4000, 100, 30000, 5])
    ar = hv.FusedAllreduce(per_rank, op="average", threshold_bytes=40000, fuse_boundary=fuse_boundary,
                           small_bucket_bytes=0, replace_in_tensors=into, add_from_tensors=add)
    sid = torch.cuda.current_stream().cuda_stream
    launches = ar.kernel_sequence()
    with hv.Timeline(capacity=1000) as tl:
        ar(sid)
        ar(sid)
    assert tl.dropped == 0 and len(tl.records) == 2 * len(launches)
    code = {"pack": 0, "rs": 1, "ag": 2, "unpack": 3, "rs_ag": 6, "pack_rs": 8, "ag_unpack": 9}
    for rec, (kind, bi, s) in zip(tl.records, launches + launches):
        assert rec["kind"] == code[kind] and rec["step"] == s and rec["nranks"] == 5 and rec["launches"] == 1
        both = bi if isinstance(bi, tuple) else (bi,)  # a launch serving a pair of buckets counts both
        assert rec["count"] == sum(ar.buckets[x].count for x in both) and rec["duration_us"] > 0
    starts = [r["start_us"] for r in tl.records]
    assert starts[0] == 0 and starts == sorted(starts)
    trace = tl.chrome_trace()
    json.dumps(trace)
    ranks = {e["tid"] for e in trace["traceEvents"] if e["ph"] == "X"}
    assert ranks == set(range(6))  # GPU track + 5 ranks


def test_small_buckets_record_one_launch():
    """Buckets on the one-launch path: one record each, named for the whole cycle."""
    say("timeline records small buckets")
    per_rank = tensors(5, [7, 4000, 100, 30000, 5])
    ar = hv.FusedAllreduce(per_rank, op="average", threshold_bytes=40000)
    launches = ar.kernel_sequence()
    assert {k for k, _, _ in launches} == {"cycle_small", "ring_small"}
    with hv.Timeline(capacity=100) as tl:
        ar()
    code = {"cycle_small": hv._lib.KERNEL_CYCLE_SMALL, "ring_small": hv._lib.KERNEL_RING_SMALL}
    assert [r["kind"] for r in tl.records] == [code[k] for k, _, _ in launches]
    names = {e["name"] for e in tl.chrome_trace()["traceEvents"] if e["ph"] == "X" and e["tid"] == 0}
    assert names == {"copy in + whole ring + copy out (one launch)", "whole ring (one launch)"}


def test_capacity_counts_dropped_launches():
    per_rank = tensors(3, [1000, 2000])
    ar = hv.FusedAllreduce(per_rank, small_bucket_bytes=0)  # one launch per ring step
    with hv.Timeline(capacity=2) as tl:
        ar()
    assert len(tl.records) == 2 and tl.dropped == len(ar.kernel_sequence()) - 2


def test_environment_variable_writes_trace(tmp_path):
    path = tmp_path / "trace.json"
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "import torch, paper_1802_05799_amd as hv\n"
        "xs = [[torch.ones(1000, device='cuda'), torch.ones(77, device='cuda')] for _ in range(4)]\n"
        "ar = hv.FusedAllreduce(xs, small_bucket_bytes=0)\n"
        "ar(); ar(); torch.cuda.synchronize()\n" % ROOT
    )
    say("timeline env subprocess")
    env = dict(os.environ, HVDX_TIMELINE=str(path))
    subprocess.run([sys.executable, "-c", code], env=env, check=True, timeout=120)
    trace = json.loads(path.read_text())
    names = [e["name"] for e in trace["traceEvents"] if e["ph"] == "X" and e["tid"] == 0]
    # the adding steps read the tensors (no copy-in), the replacing steps write them (no copy-out)
    assert names == ["reduce-scatter 0", "reduce-scatter 1", "reduce-scatter + allgather 2", "allgather 1",
                     "allgather 2"] * 2


@pytest.mark.parametrize("mode", list(MODES))
def test_per_phase_records(mode):
    fuse_boundary, into, add = MODES[mode]
    per_rank = tensors(6, [7, 4000, 100, 30000, 5])
    ar = hv.FusedAllreduce(per_rank, op="average", threshold_bytes=40000, fuse_boundary=fuse_boundary,
                           small_bucket_bytes=0, replace_in_tensors=into, add_from_tensors=add)
    with hv.Timeline(capacity=100, per_phase=True) as tl:
        ar()
    got = [(r["kind"], r["step"], r["launches"]) for r in tl.records]
    want = []
    for bi, b in enumerate(ar.buckets):
        if b.slot > 0:  # ran together with an earlier bucket: that group's records cover it
            continue
        if fuse_boundary and not b.direct and add:  # steps 0-3 from the tensors, 4 + 0, steps 1-4 into them
            want += [(1, 0, 4), (6, 4, 1), (2, 1, 4)]
            continue
        if fuse_boundary and not b.direct and into:  # copy-in + step 0, steps 1-3, 4 + 0, steps 1-4
            want += [(8, 0, 1), (1, 1, 3), (6, 4, 1), (2, 1, 4)]
            continue
        if fuse_boundary and not b.direct:  # copy-in + step 0, steps 1-3, 4 + 0, steps 1-3, 4 + copy-out
            want += [(8, 0, 1), (1, 1, 3), (6, 4, 1), (2, 1, 3), (9, 4, 1)]
            continue
        if not b.direct:
            want.append((0, -1, 1))
        want += [(1, 0, 4), (6, 4, 1), (2, 1, 4)]
        if not b.direct:
            want.append((3, -1, 1))
    assert any(not b.direct for b in ar.buckets) and any(b.direct for b in ar.buckets)
    assert got == want
