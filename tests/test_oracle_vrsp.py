"""Pins of the VRSP oracle (Algorithm 1, Eq. 4, the R - 1 measure of Sec. 3.2).

* the hand-worked examples under tests/golden/ (weight order, least-loaded
  non-full pool, tie-breaks, the cardinality limit, the output order);
* closed forms: P = 1 (every pool one sequence: the output is the weight
  order), P = GBS (one pool, same), equal weights (round robin);
* invariants on random windows: a permutation, exactly P per pool, loads
  that sum to the window's workload;
* brute force on tiny windows: no partition into pools of P has a smaller
  maximum load than the optimum, and VRSP never beats it.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import vrsp as ov

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "vrsp_worked_examples.json")


def test_workload_is_sum_of_squares():
    assert ov.workload([3, 4]) == 25
    assert ov.workload([1] * 10) == 10
    assert ov.workload([40000]) == 1600000000


@pytest.mark.parametrize("ex", json.load(open(GOLDEN))["examples"], ids=lambda e: e["name"])
def test_worked_examples(ex):
    order, pools, loads = ov.vrsp(ex["F"], ex["P"])
    assert order == ex["order"]
    assert loads == ex["loads"]
    assert ov.imbalance(loads, ex["P"]) == Fraction(*ex["imbalance"])
    prod = ov.production_order(ex["F"], ex["P"])
    assert prod == ex["production_loads"]
    assert ov.imbalance(prod, ex["P"]) == Fraction(*ex["production_imbalance"])


@pytest.mark.parametrize("seed", range(10))
def test_single_sequence_pools_give_weight_order(seed):
    rng = np.random.default_rng(seed)
    F = [int(x) for x in rng.integers(0, 50, 20)]
    order, _, loads = ov.vrsp(F, 1)
    assert order == sorted(range(20), key=lambda i: (-F[i], i))
    assert loads == [F[i] for i in order]


@pytest.mark.parametrize("seed", range(10))
def test_one_pool_gives_weight_order(seed):
    rng = np.random.default_rng(100 + seed)
    F = [int(x) for x in rng.integers(0, 50, 12)]
    order, pools, loads = ov.vrsp(F, 12)
    assert order == sorted(range(12), key=lambda i: (-F[i], i))
    assert loads == [sum(F)]


@pytest.mark.parametrize("P,K", [(2, 3), (4, 4), (3, 5)])
def test_equal_weights_round_robin(P, K):
    order, pools, loads = ov.vrsp([9] * (P * K), P)
    assert pools == [[k + K * j for j in range(P)] for k in range(K)]
    assert loads == [9 * P] * K


@pytest.mark.parametrize("seed", range(30))
def test_random_windows_invariants(seed):
    rng = np.random.default_rng(200 + seed)
    P = int(rng.choice([1, 2, 4, 8]))
    K = int(rng.integers(1, 9))
    F = [int(x) for x in rng.integers(0, 10 ** 9, P * K)]
    order, pools, loads = ov.vrsp(F, P)
    assert sorted(order) == list(range(P * K))
    assert all(len(p) == P for p in pools)
    assert loads == [sum(F[i] for i in p) for p in pools]
    assert sum(loads) == sum(F)


def _opt_max_load(F, P):
    """Minimum over all partitions into pools of exactly P of the max pool load."""
    best = None
    idx = list(range(len(F)))

    def rec(rest, worst):
        nonlocal best
        if best is not None and worst >= best:
            return
        if not rest:
            best = worst
            return
        first = rest[0]
        for comb in itertools.combinations(rest[1:], P - 1):
            group = (first,) + comb
            left = [i for i in rest if i not in group]
            rec(left, max(worst, sum(F[i] for i in group)))

    rec(idx, 0)
    return best


@pytest.mark.parametrize("seed", range(25))
def test_brute_force_optimum_bounds_vrsp(seed):
    rng = np.random.default_rng(300 + seed)
    P, K = [(2, 2), (2, 3), (3, 2), (2, 4), (4, 2)][seed % 5]
    F = [int(x) ** 2 for x in rng.integers(1, 40, P * K)]
    _, _, loads = ov.vrsp(F, P)
    opt = _opt_max_load(F, P)
    assert opt <= max(loads)
    # and the optimum is never below the mean pool load
    assert opt * K >= sum(F)


def test_rejects_pool_size_not_dividing_window():
    with pytest.raises(ValueError):
        ov.vrsp([1, 2, 3], 2)
    with pytest.raises(ValueError):
        ov.vrsp([1, 2], 0)
