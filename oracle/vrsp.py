"""VRSP oracle (test infrastructure): Variance-Reduced Sequence Placement.

Pure Python integers, written from Sec. 4.2 of the paper (Algorithm 1,
Eq. 4) and the imbalance measure of Sec. 3.2:

* workload of a packed sequence: F_i = sum_j l_ij^2 over its raw samples;
* K = GBS / P pools of exactly P packed sequences each;
* packed sequences in order of decreasing F_i, then increasing i; each goes
  to the pool of least (load, index) among the pools that still hold fewer
  than P sequences (a min-heap of (load, k) from which full pools are
  dropped);
* the output is the pools concatenated in index order (GA-major, pool-minor),
  each pool's sequences in the order they were placed;
* residual imbalance R - 1 with R = max_k L_k / (P * mu), mu the mean F_i.

The production-order grouping the paper compares against takes pools of P
consecutive sequences in their original order.
"""
from __future__ import annotations

import heapq
from fractions import Fraction
from typing import List, Sequence, Tuple


def workload(lengths: Sequence[int]) -> int:
    """F = sum of squared raw-sample lengths of one packed sequence (Eq. 4)."""
    return sum(int(x) * int(x) for x in lengths)


def vrsp(F: Sequence[int], P: int) -> Tuple[List[int], List[List[int]], List[int]]:
    """Algorithm 1 on the workloads F of one GBS window.

    Returns (order, pools, loads): ``order`` lists the original indices in
    output order, ``pools[k]`` the indices placed in pool k in placement
    order, ``loads[k]`` the pool's summed workload.
    """
    D = len(F)
    if P < 1 or D % P:
        raise ValueError("pool size must divide the window")
    K = D // P
    pools: List[List[int]] = [[] for _ in range(K)]
    loads = [0] * K
    by_weight = sorted(range(D), key=lambda i: (-int(F[i]), i))
    heap = [(0, k) for k in range(K)]
    heapq.heapify(heap)
    for i in by_weight:
        load, k = heapq.heappop(heap)
        pools[k].append(i)
        loads[k] = load + int(F[i])
        if len(pools[k]) < P:
            heapq.heappush(heap, (loads[k], k))
    order = [i for pool in pools for i in pool]
    return order, pools, loads


def production_order(F: Sequence[int], P: int) -> List[int]:
    """Pool loads of the unbalanced grouping: pool k = sequences kP .. kP+P-1."""
    D = len(F)
    if P < 1 or D % P:
        raise ValueError("pool size must divide the window")
    return [sum(int(x) for x in F[k * P:(k + 1) * P]) for k in range(D // P)]


def imbalance(loads: Sequence[int], P: int) -> Fraction:
    """R - 1 with R = max_k L_k / (P * mu), mu = mean workload (Sec. 3.2), exact."""
    K = len(loads)
    total = sum(int(x) for x in loads)
    if total == 0:
        return Fraction(0)
    # P * mu = P * total / (K * P) = total / K
    return Fraction(max(int(x) for x in loads) * K, total) - 1
