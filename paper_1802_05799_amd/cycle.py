"""The Tensor Fusion cycle over N simulated ranks (paper section 7, steps 1-6).

`FusedAllreduce` is built once for a fixed set of gradient tensors (one list per
simulated rank, all in GPU memory) and then reduces them in place each time it is
called: every fusion buffer of the plan goes through the ring-allreduce of paper
section 3; a tensor larger than the buffer runs the ring in place on the rank tensors
themselves.  By default a fusion buffer's ring runs on the ranks' tensors: its adding
steps read each rank's own elements from the tensors (where a copy-in would take them
from), the buffers hold the partial sums received, and its replacing steps write the
tensors (where a copy-out would put them); the paper's copies are options.  Torch
provides the device memory and the stream; every step is a libhvdx kernel.

The fusion buffers are allocated once, at the size of the largest fused bucket
(at most the threshold, 64 MiB by default), and reused for every bucket, as the
paper's step 2 describes.  The descriptor arrays the kernels read (tensor pointers,
sizes, offsets, tile tables) are uploaded once at construction, so the tensors must
stay allocated and in place for the object's lifetime.

Buckets of at most `small_bucket_bytes` per rank (4 MiB by default) run their whole
cycle in one launch (hvdx_fuse_allreduce_small, hvdx_ring_allreduce_small): there a
ring step's launch costs more than its messages.  Fused buckets on the per-step path
run in groups, in plan order, every launch serving the whole group (up to four
buffers with the ring on the tensors, else two), each member after the first with
fusion buffers of its own.  Same bits either way.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import _lib as L
from . import timeline as _timeline

_TORCH_DTYPE = {L.FLOAT32: torch.float32, L.FLOAT16: torch.float16}
_HVDX_DTYPE = {torch.float32: L.FLOAT32, torch.float16: L.FLOAT16}
_OPS = {"sum": L.SUM, "average": L.AVERAGE}


@dataclass
class Bucket:
    tensors: list  # indices into the ready list
    offsets: list  # element offsets in the buffer
    count: int  # buffer elements
    direct: bool  # reduced in place without a copy
    numel_dev: torch.Tensor | None = None
    offset_dev: torch.Tensor | None = None
    ptrs_dev: torch.Tensor | None = None
    small: bool = False  # the whole cycle in one launch
    tiles: tuple | None = None  # (device copy-in table, tiles, device copy-out table, tiles)
    group: tuple = ()  # the buckets (this one included) whose cycles share every launch, or ()
    slot: int = 0  # position in the group: slot k uses fusion buffer set k; slot 0 runs the group


def _check_disjoint(tensors) -> None:
    """Raise ValueError when two of the tensors (any ranks) share memory.  The kernels
    read and write every rank's tensors in one launch (all of a group's buckets' in a
    grouped launch), so a tensor listed twice, or two views of one storage, would make the
    result depend on the order of blocks; the device pointers cannot be checked on the
    C side."""
    spans = sorted((x.data_ptr(), x.data_ptr() + x.numel() * x.element_size(), r, t)
                   for r, ts in enumerate(tensors) for t, x in enumerate(ts) if x.numel() > 0)
    for (a0, a1, ra, ta), (b0, b1, rb, tb) in zip(spans, spans[1:]):
        if b0 < a1:
            raise ValueError(f"tensors overlap in memory: rank {ra} tensor {ta} and rank {rb} tensor {tb}")


class FusedAllreduce:
    """In-place allreduce of N ranks' gradient lists (SUM or AVERAGE)."""

    def __init__(self, per_rank, op: str = "average", compress: bool = False,
                 threshold_bytes: int = L.DEFAULT_FUSION_THRESHOLD, align_bytes: int = L.DEFAULT_FUSION_ALIGN,
                 schedule: str = "ring", fuse_boundary: bool = True,
                 small_bucket_bytes: int = L.SMALL_BUCKET_BYTES, pair_buckets: bool = True, tiled: bool = True,
                 replace_in_tensors: bool = True, add_from_tensors: bool = True):
        """schedule "ring" runs the ring's 2(N-1) steps; "fold" computes the same bits
        with hvdx_fold_allreduce (no per-step messages: a one-GPU bound, not the ring).
        With fuse_boundary (ring schedule, N >= 3) a fusion buffer's copy-in runs with
        the ring's first adding step and its copy-out with the last replacing step
        (hvdx_fuse_allreduce); otherwise copy-in, ring and copy-out are separate calls.
        With the fused boundary, a bucket of at most small_bucket_bytes per rank (0:
        none) runs its whole cycle in one launch instead (compressed direct tensors
        excepted).  With pair_buckets (fused boundary) the fused buckets on the per-step
        path run in groups, every launch serving the group: up to TILED_MAX_BUCKETS (and
        TILED_MAX_BUFFERS // N) with both tensor flags, else two; if the last group is
        short, the first small fused bucket joins it instead of taking its one launch.
        With tiled (fused boundary, N >= 3) the fused copies of those buckets are driven by
        tile tables cut once here
        (hvdx_fuse_copy_tiles, hvdx_fuse_allreduce_tiled) instead of finding each stretch's
        tensors in the kernel.  With replace_in_tensors (tiled) their replacing steps
        deliver each chunk straight into the receiving rank's tensors and forward it from
        there, so no copy-out follows (HVDX_TILED_REPLACE_IN_TENSORS); with
        add_from_tensors as well, each adding step reads the receiver's own elements from
        its tensors, so no copy-in either (HVDX_TILED_ADD_FROM_TENSORS) and the fusion
        buffers hold only received partial sums.  Compressed buckets then work as the
        compressed ring of a direct tensor does: binary16 partial sums, binary32 values
        (binary16 results held exactly) in the replacing steps.  All give the same bits."""
        if schedule not in ("ring", "fold"):
            raise ValueError("schedule must be 'ring' or 'fold'")
        self.schedule = schedule
        self.fuse_boundary = fuse_boundary and schedule == "ring"
        if not per_rank or len(per_rank) > L.MAX_RANKS:
            raise ValueError(f"need 1..{L.MAX_RANKS} ranks")
        if op not in _OPS:
            raise ValueError(f"op must be one of {sorted(_OPS)}")
        self.nranks = n = len(per_rank)
        self.tensors = [list(ts) for ts in per_rank]
        t0 = self.tensors[0]
        ntensors = len(t0)
        for ts in self.tensors:
            if len(ts) != ntensors:
                raise ValueError("every rank needs the same number of tensors")
            for x, ref in zip(ts, t0):
                if x.shape != ref.shape or x.dtype != ref.dtype or x.device != ref.device:
                    raise ValueError("tensors must match across ranks in shape, dtype and device")
                if not x.is_contiguous() or x.device.type != "cuda":
                    raise ValueError("tensors must be contiguous GPU tensors")
        _check_disjoint(self.tensors)
        self.device = t0[0].device if ntensors else torch.device("cuda", torch.cuda.current_device())
        self.dtype = _HVDX_DTYPE[t0[0].dtype] if ntensors else L.FLOAT32
        if compress and self.dtype != L.FLOAT32:
            raise ValueError("fp16 compression applies to float32 gradients")
        self.op = _OPS[op]
        self.compress = L.COMPRESS_FP16 if compress else L.COMPRESS_NONE
        self.buf_dtype = L.FLOAT16 if compress else self.dtype
        self.numel = [x.numel() for x in t0]

        bucket_of, offset, counts, direct = L.hvdx_fuse_plan(self.numel, self.buf_dtype, threshold_bytes,
                                                             align_bytes)
        self.buckets = [Bucket([], [], c, bool(d)) for c, d in zip(counts, direct)]
        for t, (b, off) in enumerate(zip(bucket_of, offset)):
            self.buckets[b].tensors.append(t)
            self.buckets[b].offsets.append(off)
        for b in self.buckets:
            es = _TORCH_DTYPE[self.dtype if b.direct else self.buf_dtype].itemsize
            b.small = (self.fuse_boundary and b.count * es <= small_bucket_bytes
                       and not (b.direct and self.compress))

        self.tiled = tiled and self.fuse_boundary and n >= 3
        self.tiled_flags = L.TILED_BUFFERS
        if replace_in_tensors and self.tiled:
            self.tiled_flags = L.TILED_REPLACE_IN_TENSORS | (L.TILED_ADD_FROM_TENSORS if add_from_tensors else 0)
        self.groups = []
        if pair_buckets and self.fuse_boundary and n >= 3:
            # fused buckets on the per-step path, grouped in plan order: with the ring on the
            # tensors as many as one launch takes, else two (the two-buffer kernels); a group
            # runs at its first member's place, so a direct tensor or small bucket between its
            # members runs after them (the buckets share no data: the bits do not depend on
            # the order)
            size = 2
            if self.tiled_flags & L.TILED_ADD_FROM_TENSORS:
                size = max(2, min(L.TILED_MAX_BUCKETS, L.TILED_MAX_BUFFERS // n))
            ok = [i for i, x in enumerate(self.buckets) if not x.direct and not x.small and x.count > 0]
            small = [i for i, x in enumerate(self.buckets) if not x.direct and x.small and x.count > 0]
            if len(ok) % size and small:
                # a group left short takes the first small fused bucket along: its few elements
                # then ride in the others' 2N-2 launches instead of a launch of their own whose
                # threads walk all 2N-2 steps one after another
                self.buckets[small[0]].small = False
                ok = sorted(ok + small[:1])
            for g in range(0, len(ok), size):
                members = tuple(ok[g : g + size])
                if len(members) < 2:
                    continue
                self.groups.append(members)
                for slot, i in enumerate(members):
                    self.buckets[i].group, self.buckets[i].slot = members, slot

        dev = self.device
        # one fusion buffer per rank, allocated once and reused for every bucket; the other
        # members of a group run at the same time as the first and have buffers of their own
        nslots = max([len(g) for g in self.groups], default=1)
        caps = [max([b.count for b in self.buckets if not b.direct and b.slot == k], default=0) for k in range(nslots)]
        self.buf_sets = [[torch.empty(max(c, 1) if k == 0 else c, dtype=_TORCH_DTYPE[self.buf_dtype], device=dev)
                          for _ in range(n)] for k, c in enumerate(caps)]
        self.bufs = self.buf_sets[0]
        ws = max([L.hvdx_ring_workspace_bytes(n, b.count, self.dtype, self.compress)
                  for b in self.buckets if b.direct], default=0)
        self.workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
        self.workspace_bytes = ws
        for b in self.buckets:
            if b.direct:
                continue
            b.numel_dev = torch.tensor([self.numel[t] for t in b.tensors], dtype=torch.int64, device=dev)
            b.offset_dev = torch.tensor(b.offsets, dtype=torch.int64, device=dev)
            b.ptrs_dev = torch.tensor([self.tensors[r][t].data_ptr() for r in range(n) for t in b.tensors],
                                      dtype=torch.int64, device=dev)
        if self.tiled:
            for b in self.buckets:
                if b.direct or b.small or b.count == 0:
                    continue
                tabs = []
                for direction in (L.COPY_IN, L.COPY_OUT):
                    numel = [self.numel[t] for t in b.tensors]
                    arr, k = L.hvdx_fuse_copy_tiles(numel, b.offsets, b.count, self.dtype, self.buf_dtype, n, direction)
                    host = torch.frombuffer(bytearray(bytes(arr)), dtype=torch.uint8)
                    tabs += [host.to(dev), k]
                b.tiles = tuple(tabs)
        self._buf_ptrs = [[x.data_ptr() for x in bs] for bs in self.buf_sets]
        _timeline.start_from_env()

    # ---- the steps, exposed separately for tracing ------------------------------------
    def pack(self, b: Bucket, stream: int) -> None:
        L.hvdx_fuse_pack(b.ptrs_dev.data_ptr(), b.numel_dev.data_ptr(), b.offset_dev.data_ptr(), len(b.tensors),
                         self.dtype, self._buf_ptrs[0], b.count, self.buf_dtype, self.nranks, stream)

    def unpack(self, b: Bucket, stream: int) -> None:
        L.hvdx_fuse_unpack(self._buf_ptrs[0], b.count, self.buf_dtype, b.ptrs_dev.data_ptr(), b.numel_dev.data_ptr(),
                           b.offset_dev.data_ptr(), len(b.tensors), self.dtype, self.nranks, stream)

    def ring_args(self, b: Bucket):
        """(rank pointers, count, dtype, compress, workspace, workspace bytes) for a bucket's ring."""
        if b.direct:
            t = b.tensors[0]
            ptrs = [self.tensors[r][t].data_ptr() for r in range(self.nranks)]
            return ptrs, b.count, self.dtype, self.compress, self.workspace.data_ptr(), self.workspace_bytes
        return self._buf_ptrs[0], b.count, self.buf_dtype, L.COMPRESS_NONE, 0, 0

    def ring(self, b: Bucket, stream: int) -> None:
        ptrs, count, dtype, compress, ws, wsb = self.ring_args(b)
        if b.small:
            L.hvdx_ring_allreduce_small(ptrs, self.nranks, count, dtype, self.op, stream)
        elif self.schedule == "fold":
            L.hvdx_fold_allreduce(ptrs, self.nranks, count, dtype, self.op, compress, stream)
        else:
            L.hvdx_ring_allreduce(ptrs, self.nranks, count, dtype, self.op, compress, ws, wsb, stream)

    def ring_phase(self, b: Bucket, phase: int, stream: int) -> None:
        """All N-1 steps of one half of the ring (one C call)."""
        ptrs, count, dtype, compress, ws, wsb = self.ring_args(b)
        fn = L.hvdx_ring_reduce_scatter if phase == L.PHASE_REDUCE_SCATTER else L.hvdx_ring_allgather
        fn(ptrs, self.nranks, count, dtype, self.op, compress, ws, wsb, stream)

    def ring_step(self, b: Bucket, phase: int, step: int, stream: int) -> None:
        ptrs, count, dtype, compress, ws, wsb = self.ring_args(b)
        L.hvdx_ring_step(ptrs, self.nranks, count, dtype, self.op, compress, phase, step, ws, wsb, stream)

    def fused_cycle(self, b: Bucket, stream: int) -> None:
        """A fusion buffer's copy-in, ring and copy-out with the boundary steps fused
        (or, for a small bucket, all in one launch)."""
        if self.tiled and not b.small:
            L.hvdx_fuse_allreduce_tiled([self.tiled_desc(b)], self.dtype, self.buf_dtype, self.nranks, self.op,
                                        self.tiled_flags, stream)
            return
        fn = L.hvdx_fuse_allreduce_small if b.small else L.hvdx_fuse_allreduce
        fn(b.ptrs_dev.data_ptr(), b.numel_dev.data_ptr(), b.offset_dev.data_ptr(), len(b.tensors), self.dtype,
           self._buf_ptrs[0], b.count, self.buf_dtype, self.nranks, self.op, stream)

    def tiled_desc(self, x: Bucket):
        return (x.ptrs_dev.data_ptr(), x.numel_dev.data_ptr(), x.offset_dev.data_ptr(), len(x.tensors),
                self._buf_ptrs[x.slot], x.count, x.tiles[0].data_ptr(), x.tiles[1], x.tiles[2].data_ptr(), x.tiles[3])

    def fused_group(self, members, stream: int) -> None:
        """The cycles of a group of fusion buffers with every launch serving all of them."""
        bs = [self.buckets[i] for i in members]
        if self.tiled:
            L.hvdx_fuse_allreduce_tiled([self.tiled_desc(x) for x in bs], self.dtype, self.buf_dtype, self.nranks,
                                        self.op, self.tiled_flags, stream)
            return
        desc = [(x.ptrs_dev.data_ptr(), x.numel_dev.data_ptr(), x.offset_dev.data_ptr(), len(x.tensors),
                 self._buf_ptrs[x.slot], x.count) for x in bs]
        L.hvdx_fuse_allreduce_pair(desc[0], desc[1], self.dtype, self.buf_dtype, self.nranks, self.op, stream)

    def kernel_sequence(self):
        """The kernels one call launches, in order: (kind, bucket index, step) with
        kind "pack", "pack_rs" (copy-in with adding step 0), "rs", "rs_ag" (adding
        step N-2 fused with replacing step 0), "ag", "ag_unpack" (replacing step N-2
        with copy-out; with the replacing steps in the tensors, "rs_ag" and "ag" 1..N-2
        deliver into the tensors and no copy-out follows; with the adding steps from the
        tensors, "rs" 0..N-3 replace "pack_rs"), "unpack", "fold", "ring"
        (the one-rank compressed round trip),
        "cycle_small" or "ring_small" (a small bucket's whole cycle in one launch).
        A launch that serves a group of buckets names them all: (kind, (i, j, ...), step)."""
        out = []
        n = self.nranks
        for bi, b in enumerate(self.buckets):
            if b.count == 0 or b.slot > 0:
                continue
            if b.group:
                out += self._fused_sequence(b.group)
                continue
            if b.small:
                if not b.direct:
                    out.append(("cycle_small", bi, -1))
                elif n > 1:
                    out.append(("ring_small", bi, -1))
                continue
            if self.schedule == "fold":
                if not b.direct:
                    out.append(("pack", bi, -1))
                out.append(("fold", bi, -1))
                if not b.direct:
                    out.append(("unpack", bi, -1))
                continue
            if self.fuse_boundary and not b.direct and n >= 3:
                out += self._fused_sequence(bi)
                continue
            if not b.direct:
                out.append(("pack", bi, -1))
            if n == 1:
                if b.direct and self.compress:  # the only one-rank ring that launches a kernel
                    out.append(("ring", bi, -1))
            else:
                out += [("rs", bi, s) for s in range(n - 2)]
                out.append(("rs_ag", bi, n - 2))
                out += [("ag", bi, s) for s in range(1, n - 1)]
            if not b.direct:
                out.append(("unpack", bi, -1))
        return out

    def _fused_sequence(self, bi):
        n = self.nranks
        if self.tiled_flags & L.TILED_ADD_FROM_TENSORS:
            out = [("rs", bi, s) for s in range(n - 2)]
        else:
            out = [("pack_rs", bi, 0)] + [("rs", bi, s) for s in range(1, n - 2)]
        out.append(("rs_ag", bi, n - 2))
        if self.tiled_flags & L.TILED_REPLACE_IN_TENSORS:
            return out + [("ag", bi, s) for s in range(1, n - 1)]
        return out + [("ag", bi, s) for s in range(1, n - 2)] + [("ag_unpack", bi, n - 2)]

    def capture(self) -> "torch.cuda.CUDAGraph":
        """Record one call's launches (every bucket's copy-in, ring steps and copy-out)
        in a HIP graph and return it without running them.  ``graph.replay()`` then
        reduces the same tensors, in place, with one submission instead of one launch
        per kernel, which is what decides the time of small buckets.  The tensors,
        fusion buffers and descriptors the graph points at are this object's; the graph
        holds a reference to it.  Launches inside the capture get no
        timeline records."""
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream(self.device)  # default priority
        side.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.graph(graph, stream=side):
            self(side.cuda_stream)
        torch.cuda.current_stream(self.device).wait_stream(side)
        graph.owner = self  # the memory the graph points at lives as long as the graph
        return graph

    def __call__(self, stream: int | None = None) -> None:
        if stream is None:
            stream = torch.cuda.current_stream(self.device).cuda_stream
        for i, b in enumerate(self.buckets):
            if b.group and b.slot == 0:
                self.fused_group(b.group, stream)
            elif b.group:
                continue
            elif b.direct:
                self.ring(b, stream)
            elif self.fuse_boundary:
                self.fused_cycle(b, stream)
            else:
                self.pack(b, stream)
                self.ring(b, stream)
                self.unpack(b, stream)
