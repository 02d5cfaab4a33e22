"""Oracle for the memory balance of Memory Heuristic II (ParDNN, Sec. 3.2.2).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only ``tests/``, the smoke check
and the CPU-baseline leg of ``bench.py`` may use it. Plain numpy and Python
integers (exact rationals), no shared code with the HIP library.

The paper sorts operation-nodes into three kinds by how they hold memory
(Sec. 3.2.1): residual nodes keep their data for the whole training run,
reference nodes mutate a residual node's tensor and reserve nothing of their
own but must sit on the same device as it, and normal nodes hold their output
until their consumers ran. Heuristic II (Sec. 3.2.2) moves residual nodes
from the most to the least loaded partitions until Eq. 6 holds for every
partition: K / 2 times the sum of the partition's share of all residual
memory and its share of all normal memory is at least 1.

Readings (the paper leaves these open):

* node_type 0 = normal, 1 = residual, 2 = reference; a reference node adds no
  memory to any sum.
* When one kind has no memory at all, its share is taken as the fair share
  1 / K on every partition (neutral); with neither kind the predicate holds.
* A reference node whose target (``ref_target``, -1 for none) carries another
  label is "misplaced"; the count of those is reported per placement.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

NORMAL, RESIDUAL, REFERENCE = 0, 1, 2


def memory_balance(n_nodes, mem, node_type, ref_target, label, n_labels):
    """Per label: residual memory, normal memory and the Eq. 6 predicate; and
    the number of misplaced reference nodes. Raises ValueError on bad input."""
    mem = np.asarray(mem, dtype=np.int64)
    node_type = np.asarray(node_type, dtype=np.int64)
    ref_target = np.asarray(ref_target, dtype=np.int64)
    label = np.asarray(label, dtype=np.int64)
    K = int(n_labels)
    if K < 1:
        raise ValueError("n_labels must be >= 1")
    if not (mem.shape == node_type.shape == ref_target.shape == label.shape == (n_nodes,)):
        raise ValueError("array sizes")
    if n_nodes and ((label < 0).any() or (label >= K).any()):
        raise ValueError("label outside [0, n_labels)")
    if n_nodes and ((node_type < 0).any() or (node_type > 2).any()):
        raise ValueError("node_type outside {0, 1, 2}")
    if n_nodes and ((ref_target < -1).any() or (ref_target >= n_nodes).any()):
        raise ValueError("ref_target outside [-1, n_nodes)")
    if n_nodes and (mem < 0).any():
        raise ValueError("negative memory")

    # per-label sums (int64 is exact: the graph's total memory fits int64)
    res_np = np.zeros(K, np.int64)
    nor_np = np.zeros(K, np.int64)
    is_res, is_nor = node_type == RESIDUAL, node_type == NORMAL
    np.add.at(res_np, label[is_res], mem[is_res])
    np.add.at(nor_np, label[is_nor], mem[is_nor])
    res = [int(x) for x in res_np]
    nor = [int(x) for x in nor_np]
    RES, NOR = sum(res), sum(nor)

    # Eq. 6 for each partition (label)
    balanced = []
    for k in range(K):
        share_res = Fraction(res[k], RES) if RES > 0 else Fraction(1, K)
        share_nor = Fraction(nor[k], NOR) if NOR > 0 else Fraction(1, K)
        balanced.append(Fraction(K, 2) * (share_res + share_nor) >= 1)

    refs = np.nonzero((node_type == REFERENCE) & (ref_target >= 0))[0]
    misplaced = int((label[refs] != label[ref_target[refs]]).sum())

    return {"res_mem": np.array(res, dtype=np.int64), "nor_mem": np.array(nor, dtype=np.int64),
            "balanced": np.array(balanced, dtype=np.uint8), "ref_misplaced": misplaced}
