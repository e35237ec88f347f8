"""The five synthetic allreduce workloads.

Each workload is N simulated ranks, each holding the gradient tensors of one model in
the order backpropagation makes them ready, with values from `workloads.rng`:
rank r uses key ``seed + r`` and element index = position of the element in the
concatenation of that rank's tensors (in ready order).

The three models are the ones the paper's benchmark sections train (Inception V3,
ResNet, VGG-16); the values stand in for real gradients, which need the
benchmark suite and ImageNet.
"""
from __future__ import annotations

from dataclasses import dataclass

from . import models

__all__ = ["Workload", "WORKLOADS", "get"]

FUSION_THRESHOLD = 64 << 20  # bytes: the default fusion buffer size, read as 64 MiB
FUSION_ALIGN = 16  # bytes: every tensor starts on a 16-byte boundary of the buffer


@dataclass(frozen=True)
class Workload:
    name: str
    model: str
    nranks: int
    dist: str  # "uniform" (-1, 1) or "normal" (0, sigma)
    op: str  # "sum" or "average"
    compress: bool  # fp16 on the wire
    sigma: float = 0.01
    seed: int = 0

    def tensors(self):
        """(name, shape) list in ready (reverse definition) order."""
        return models.ready_order(models.MODELS[self.model]())

    def numel(self):
        return models.numel_list(self.tensors())

    def prefix(self):
        """Element index of each tensor's first element in the rank's concatenation."""
        out, acc = [], 0
        for n in self.numel():
            out.append(acc)
            acc += n
        return out

    def key(self, rank: int) -> int:
        return self.seed + rank

    @property
    def rank_bytes(self) -> int:
        """fp32 gradient bytes per rank."""
        return 4 * sum(self.numel())


WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny", "tiny", 4, "uniform", "average", False),
        Workload("resnet50", "resnet50", 8, "normal", "average", False),
        Workload("inceptionv3", "inceptionv3", 16, "normal", "average", False),
        Workload("vgg16", "vgg16", 32, "normal", "average", False),
        Workload("vgg16fp16", "vgg16", 64, "normal", "average", True),
    )
}


def get(name: str) -> Workload:
    return WORKLOADS[name]
