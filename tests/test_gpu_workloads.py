"""The five workloads at full size through the whole Tensor Fusion cycle on the GPU.

Every element of every rank is compared bit for bit with the C oracle (oracle/csrc),
which runs the same allreduce over host copies of the same inputs: the plan, the copy
in, the ring of section 3 chunk by chunk, the copy out (section 7's steps 3-5).  The
rank storages are compared whole, so the gaps between the tensor views (which nothing
may write) are compared too.  On top of that, check (1) (every rank identical) and check
(2) (the distance to the binary64 sum of the inputs within the derived summation bound)
run on the device over every element.
"""
import numpy as np
import pytest
import torch

import _pins
import paper_1802_05799_amd as hv
from _gpu import assert_bits_equal, say
from oracle import fusion
from oracle import native
from workloads import configs, rng
from workloads import gpu as wgpu

pytestmark = pytest.mark.gpu


def test_gpu_generator_matches_numpy():
    for name in ("tiny", "resnet50", "vgg16"):
        w = configs.get(name)
        for r in (0, w.nranks - 1):
            x = torch.empty(70001, dtype=torch.float32, device="cuda")
            first = 123457 if name != "tiny" else 0
            wgpu.fill_(x, w.dist, w.key(r), first, w.sigma)
            want = rng.values(w.dist, w.key(r), np.arange(first, first + x.numel()), w.sigma)
            assert_bits_equal(x.cpu().numpy(), want, f"{name} rank {r}")


def oracle_storages(w, storage, starts, threshold):
    """Host copies of every rank's flat storage, reduced in place by the C oracle on all
    the host threads OpenMP is given (the tensors are views into the copies)."""
    numel = w.numel()
    host = [s.cpu().numpy() for s in storage]
    views = [[h[s : s + m] for s, m in zip(starts, numel)] for h in host]
    ws = np.empty(native.workspace_bytes(numel, w.nranks, np.float32, w.compress, threshold), dtype=np.uint8)
    native.allreduce(views, w.op, compress=w.compress, threshold=threshold, threads=native.max_threads(), out=views,
                     workspace=ws)
    del ws
    return host


def check_every_element(name, storage, host):
    for r in range(len(storage)):
        assert_bits_equal(storage[r].cpu().numpy(), host[r], f"{name} rank {r}")


def check2_on_device(w, storage, starts):
    """Check (2) over every element: |rank 0's result - binary64 sum of the inputs (/N)|
    within the derived bound, and within rel 1e-6*N for binary32."""
    n = w.nranks
    tmp = torch.zeros_like(storage[0])
    ref = torch.zeros(storage[0].shape, dtype=torch.float64, device="cuda")
    absum = torch.zeros_like(ref)
    for r in range(n):
        wgpu.fill_rank_flat_(tmp, w, r, starts)
        ref += tmp.double()
        absum += tmp.double().abs()
    d = n if w.op == "average" else 1
    ref /= d
    absum /= d
    err = (storage[0].double() - ref).abs()
    c, eta = _pins.check2_coefficients(n, w.op, "f16" if w.compress else "f32", cast_in=w.compress)
    bound = c * absum + eta
    assert bool((err <= bound).all()), float((err - bound).max())
    if not w.compress:
        assert bool((err <= 1e-6 * n * absum).all())


@pytest.mark.parametrize(
    "name,threshold,fuse_boundary,mode",
    [("tiny", 64 << 20, True, "tensors"), ("resnet50", 64 << 20, True, "tensors"),
     ("inceptionv3", 64 << 20, True, "tensors"), ("vgg16", 64 << 20, True, "tensors"),
     ("vgg16fp16", 64 << 20, True, "tensors"), ("resnet50", 0, True, "tensors"),
     ("inceptionv3", 1 << 20, True, "tensors"), ("resnet50", 64 << 20, True, "copy-in"),
     ("resnet50", 64 << 20, True, "buffers"), ("vgg16", 64 << 20, True, "buffers"),
     ("resnet50", 64 << 20, False, "tensors"), ("vgg16", 64 << 20, False, "tensors"),
     ("vgg16fp16", 64 << 20, False, "tensors")],
    ids=["tiny", "resnet50", "inceptionv3", "vgg16", "vgg16fp16", "resnet50-unfused", "inceptionv3-1MiB",
         "resnet50-copy-in", "resnet50-buffers", "vgg16-buffers", "resnet50-separate-boundary",
         "vgg16-separate-boundary", "vgg16fp16-separate-boundary"],
)
def test_full_workload(name, threshold, fuse_boundary, mode):
    """Threshold 0 is the unfused ablation: every tensor reduced by its own ring.  With
    fuse_boundary=False copy-in, ring and copy-out run as separate calls.  Mode "tensors"
    (the default) runs the fused buckets' adding steps from the tensors and their
    replacing steps into them; "copy-in" only the latter; "buffers" the ring in the
    fusion buffers between the copies."""
    w = configs.get(name)
    say(f"workload {name} threshold {threshold} fuse_boundary {fuse_boundary} mode {mode}: generate")
    per_rank, storage, starts = wgpu.make_rank_tensors(w)
    torch.cuda.synchronize()
    say(f"workload {name}: C oracle on {native.max_threads()} host threads")
    host = oracle_storages(w, storage, starts, threshold)
    say(f"workload {name}: allreduce")
    ar = hv.FusedAllreduce(per_rank, op=w.op, compress=w.compress, threshold_bytes=threshold,
                           fuse_boundary=fuse_boundary, replace_in_tensors=mode != "buffers",
                           add_from_tensors=mode == "tensors")
    plan = fusion.fuse_plan(w.numel(), 2 if w.compress else 4, threshold)
    assert [(b.count, b.direct) for b in plan] == [(b.count, b.direct) for b in ar.buckets]
    ar()
    torch.cuda.synchronize()

    say(f"workload {name}: every element of every rank against the oracle")
    check_every_element(name, storage, host)
    del host

    say(f"workload {name}: check 1")
    for r in range(1, w.nranks):
        assert torch.equal(storage[r].view(torch.int32), storage[0].view(torch.int32)), f"rank {r} differs"

    say(f"workload {name}: check 2")
    check2_on_device(w, storage, starts)
