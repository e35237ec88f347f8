"""Workers for the exhaustive binary16 tests: the oracle on one block of inputs.  This
module imports numpy and the oracle only, so the worker processes never load the GPU
library."""
import numpy as np

from oracle import fusion, ring


def pairs(base: int, lo: int, hi: int) -> np.ndarray:
    """Elements [lo, hi) of a slice of pairs: rank 0 holds binary16 pattern
    base + k // 2^16 and rank 1 pattern k mod 2^16 at element k."""
    k = np.arange(lo, hi, dtype=np.uint32)
    a = (base + (k >> 16)).astype(np.uint16)
    b = (k & 0xFFFF).astype(np.uint16)
    return np.stack([a.view(np.float16), b.view(np.float16)])


def ring_sum_block(args) -> np.ndarray:
    """The oracle's ring (SUM, two ranks) on columns [lo, hi) of a `count`-element slice."""
    base, lo, hi, count = args
    x = pairs(base, lo, hi)
    with np.errstate(invalid="ignore"):  # inf + -inf is NaN by definition
        return ring.ring_allreduce(x, "sum", count=count, elems=np.arange(lo, hi))


def patterns32(lo: int, hi: int) -> np.ndarray:
    """The binary32 values whose bit patterns are lo .. hi-1."""
    return np.arange(lo, hi, dtype=np.uint32).view(np.float32)


def pack16_block(args) -> np.ndarray:
    """The oracle's copy-in of one binary32 tensor (patterns lo .. hi-1) into a
    binary16 buffer."""
    lo, hi = args
    bucket = fusion.Bucket(tensors=[0], offsets=[0], count=hi - lo)
    with np.errstate(invalid="ignore"):
        return fusion.pack([patterns32(lo, hi)], bucket, np.float16)
