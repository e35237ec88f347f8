"""CPU oracle for Horovod's data-parallel hot path (Tensor Fusion + ring-allreduce).

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything in this package.
The GPU library never calls it, and nothing here calls the GPU library: the two
share no code.  Inputs come from the separate ``workloads`` generator.

Plain, slow, written to be checked against the paper by eye:

* ``fusion``    -- Tensor Fusion, paper section 7 (the six-step list): the plan
                   that picks the tensors for each buffer, and the copies in and out.
* ``ring``      -- the ring-allreduce of paper section 3 (the paragraph after the
                   ring figure): N-1 adding iterations, N-1 replacing iterations,
                   simulated over N rank buffers, with per-rank traffic counters.
* ``allreduce`` -- the two composed: one averaging allreduce over every rank's
                   list of gradient tensors (paper section 5, the optimizer wrapper
                   that averages gradients).
* ``broadcast`` -- the root's variables copied to every rank (paper sections 4
                   and 5), as a pipelined chain along the ring.
* ``native``    -- the same allreduce as plain C (``csrc/oracle.c``, built by
                   ``build.py``), bit-identical to the numpy modules, fast enough to
                   run whole workloads on the host's cores.

Arithmetic is in the buffer's precision (binary32, or binary16 when compressed),
because the result of the method is defined by that arithmetic in ring order; an
fp64 sum is used only by the tests that bound the oracle's error.  Where the paper
is silent the readings are documented in ``ring`` and ``fusion``.  Every function
here is pinned by tests in ``tests/test_oracle_*.py``; none is "parity unpinned".
"""
from . import allreduce, broadcast, fusion, ring  # noqa: F401
