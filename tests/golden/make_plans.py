"""Write plans.txt: the oracle's Tensor Fusion plan for each of the five workloads.

Calls only the oracle and the workload shape lists.  Run from the repository root:
    python tests/golden/make_plans.py
"""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import fusion  # noqa: E402
from workloads import configs  # noqa: E402

lines = [
    "# <workload> <buffer elements> <tensors> <direct>   one row per fusion buffer, in order",
    "# written by tests/golden/make_plans.py (oracle.fusion.fuse_plan, 64 MiB, 16 B alignment)",
]
for name, w in configs.WORKLOADS.items():
    for b in fusion.fuse_plan(w.numel(), 2 if w.compress else 4):
        lines.append(f"{name} {b.count} {len(b.tensors)} {int(b.direct)}")
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "plans.txt"), "w") as f:
    f.write("\n".join(lines) + "\n")
