"""libra_vrsp (C ABI) against the VRSP oracle: bit-exact order, pool loads
and workloads on the hand-worked examples, random windows and synthetic
256K / 1M windows; error paths."""
import ctypes
import json
import os

import numpy as np
import pytest

import paper_2607_23250_amd as pl
from oracle import vrsp as ov
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "vrsp_worked_examples.json")

# packs whose squared lengths sum to the workloads of the worked examples
PACK_FOR = {50: [5, 5], 10: [3, 1], 40: [6, 2], 30: [5, 2, 1], 20: [4, 2], 5: [2, 1],
            35: [5, 3, 1], 7: [2, 1, 1, 1], 100: [10], 1: [1]}


def _same(packs, P):
    order, loads, work = pl.libra_vrsp(packs, P)
    F = [ov.workload(p) for p in packs]
    o_order, _, o_loads = ov.vrsp(F, P)
    assert work.tolist() == F
    assert order.tolist() == o_order
    assert loads.tolist() == o_loads
    return order, loads


@pytest.mark.parametrize("ex", json.load(open(GOLDEN))["examples"], ids=lambda e: e["name"])
def test_worked_examples(ex):
    packs = [PACK_FOR[f] for f in ex["F"]]
    order, loads = _same(packs, ex["P"])
    assert order.tolist() == ex["order"]
    assert loads.tolist() == ex["loads"]


@pytest.mark.parametrize("seed", range(200))
def test_random_windows(seed):
    rng = np.random.default_rng(seed)
    P = int(rng.choice([1, 2, 3, 4, 8]))
    K = int(rng.integers(1, 20))
    packs = []
    for _ in range(P * K):
        n = int(rng.integers(0, 6))
        # small values make equal workloads (ties) common
        packs.append([int(x) for x in rng.integers(1, 4 if seed % 2 else 3000, n)])
    _same(packs, P)


@pytest.mark.parametrize("kind", ["256K", "1M"])
@pytest.mark.parametrize("P", [1, 2, 4, 8, 16, 32, 64, 128])
def test_synthetic_windows(kind, P):
    packs = wl.vrsp_window(kind, 128, seed=P)
    order, loads = _same(packs, P)
    assert all(sum(p) == wl.VRSP_WINDOWS[kind][0] for p in packs)


def test_errors():
    with pytest.raises(pl.LibraError) as e:
        pl.libra_vrsp([[1], [2], [3]], 2)
    assert e.value.code == pl.LIBRA_EINVAL
    with pytest.raises(pl.LibraError):
        pl.libra_vrsp([[1], [2]], 0)
    with pytest.raises(pl.LibraError) as e:
        pl.libra_vrsp([[1, 0], [2]], 1)
    assert e.value.code == pl.LIBRA_EINVAL
    with pytest.raises(pl.LibraError) as e:
        pl.libra_vrsp([[2 ** 31 + 5, 2 ** 31 + 5]], 1)
    assert e.value.code == pl.LIBRA_EOVERFLOW
    # inconsistent offsets through the raw ABI
    L = pl.lib()
    lengths = np.array([1, 2, 3], dtype=np.int64)
    cu = np.array([0, 2, 1], dtype=np.int64)
    order = np.zeros(2, dtype=np.int64)
    rc = L.libra_vrsp(pl._ptr(lengths), 3, pl._ptr(cu), 2, 1, pl._ptr(order), None, None)
    assert rc == pl.LIBRA_EINVAL
