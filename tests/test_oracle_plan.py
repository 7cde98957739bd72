"""Pins of the plan oracle against what the paper and arithmetic fix.

* Eq. 6 costs against brute-force enumeration of causal same-sample pairs;
* total cost against the closed form h_q * sum_j l_j (l_j + 1) / 2 (Eq. 2 up to
  the causal constant), and a single-sample closed form per block;
* the Sec. 1 example (one 40K sample is about 10x ten 4K samples);
* Algorithm 2 on hand-worked examples (tests/golden: placement, loads and
  the bytes each worker receives), its load bound, full
  coverage, and a comparison with exhaustive search on tiny inputs.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import plan as op
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "plan_worked_examples.json")


def _cfg(w):
    return op.PlanCfg(B=w.B, H=w.H, P=w.P, CP=w.CP, h_q=w.h_q, h_kv=w.h_kv, d=w.d)


def _brute_block_pairs(lengths, lo, hi):
    """Count (q, k) with q in [lo, hi), same sample, k <= q, token by token."""
    sample_of = np.repeat(np.arange(len(lengths)), lengths)
    n = 0
    for qpos in range(lo, hi):
        for kpos in range(0, qpos + 1):
            if sample_of[kpos] == sample_of[qpos]:
                n += 1
    return n


@pytest.mark.parametrize("seed", range(40))
def test_costs_match_brute_force(seed):
    w = wl.tiny_random(seed, max_len=24)
    tiles = op.build_tiles(_cfg(w), w.lengths, w.pack_tokens)
    for t in tiles:
        pairs = _brute_block_pairs(w.lengths, t.q_begin, t.q_end)
        assert t.cost == (w.h_q // w.H) * pairs
        # every block lies inside its pack and is at most B tokens
        assert 0 < t.q_end - t.q_begin <= w.B


@pytest.mark.parametrize("name", wl.WORKLOADS)
def test_total_cost_closed_form(name):
    w = wl.workload(name)
    tiles = op.build_tiles(_cfg(w), w.lengths, w.pack_tokens)
    total = sum(t.cost for t in tiles)
    assert total == w.h_q * sum(n * (n + 1) // 2 for n in w.lengths)
    # blocks cover every token exactly once per shard
    assert sum(t.q_end - t.q_begin for t in tiles) == w.H * w.n_kv_rows


def test_single_sample_closed_form():
    B, nb, h_q, H = 64, 9, 8, 4
    L = B * nb
    cfg = op.PlanCfg(B=B, H=H, P=1, CP=1, h_q=h_q, h_kv=2, d=64)
    tiles = op.build_tiles(cfg, [L], [L])
    assert len(tiles) == nb * H
    for t in tiles:
        b = t.id // H
        assert t.cost == (h_q // H) * B * (2 * b * B + B + 1) // 2


def test_paper_ratio_40k_vs_ten_4k():
    cfg = op.PlanCfg(B=4096, H=1, P=1, CP=1, h_q=1, h_kv=1, d=64)
    one = sum(t.cost for t in op.build_tiles(cfg, [40000], [40000]))
    ten = sum(t.cost for t in op.build_tiles(cfg, [4000] * 10, [40000]))
    assert one / ten == pytest.approx(10.0, rel=1e-3)


def test_worked_examples():
    data = json.load(open(GOLDEN))
    for ex in data["examples"]:
        c = ex["cfg"]
        cfg = op.PlanCfg(**c)
        lengths = [n for p in ex["packs"] for n in p]
        packs = [sum(p) for p in ex["packs"]]
        tiles, loads = op.plan(cfg, lengths, packs)
        got = [{"id": t.id, "q_begin": t.q_begin, "q_end": t.q_end, "cost": t.cost,
                "home": t.home, "worker": t.worker} for t in tiles]
        assert got == ex["tiles"], ex["name"]
        assert loads == ex["loads"], ex["name"]
        assert op.worker_comm(tiles, cfg.V) == ex["received"], ex["name"]


def test_zigzag_home_layout():
    # CP=4, pack of 16: chunks of 2, ranks 0,1,2,3,3,2,1,0
    homes = [op.zigzag_home(x, 1, 16, 16, 4) for x in range(16, 32)]
    assert homes == [4 + r for r in (0, 0, 1, 1, 2, 2, 3, 3, 3, 3, 2, 2, 1, 1, 0, 0)]


@pytest.mark.parametrize("seed", range(60))
def test_placement_invariants(seed):
    w = wl.tiny_random(seed, max_len=64)
    cfg = _cfg(w)
    tiles, loads = op.plan(cfg, w.lengths, w.pack_tokens)
    S = sum(t.cost for t in tiles)
    assert sum(loads) == S
    V = cfg.V
    # every tile placed exactly once, on a valid worker; loads add up
    acc = [0] * V
    for t in tiles:
        assert 0 <= t.worker < V
        acc[t.worker] += t.cost
    assert acc == loads
    ids = [t.id for t in tiles]
    assert ids == sorted(ids) and len(set(ids)) == len(ids)
    # load bound: branch 1 keeps L <= C, branch 2 adds f to a load <= (S - f)/V
    fmax = max(t.cost for t in tiles)
    for L in loads:
        assert 100 * V * L <= 103 * S or V * L <= S + (V - 1) * fmax


def _opt_max_load(costs, V):
    best = None
    for assign in itertools.product(range(V), repeat=len(costs)):
        L = [0] * V
        for c, r in zip(costs, assign):
            L[r] += c
        m = max(L)
        best = m if best is None else min(best, m)
    return best


@pytest.mark.parametrize("seed", range(25))
def test_against_exhaustive_optimum(seed):
    """Alg. 2 is a heuristic: never below the optimum, never far above it."""
    rng = np.random.default_rng(seed)
    lengths = [int(x) for x in rng.integers(1, 12, size=int(rng.integers(2, 4)))]
    if sum(lengths) % 2:
        lengths[-1] += 1
    L = sum(lengths)
    cp = 2 if L % 4 == 0 and rng.random() < 0.5 else 1
    cfg = op.PlanCfg(B=int(rng.integers(2, 7)), H=1, P=1, CP=cp, h_q=1, h_kv=1,
                     d=1, elem_bytes=1)
    tiles, loads = op.plan(cfg, lengths, [L])
    if len(tiles) > 8:
        pytest.skip("too many tiles for exhaustive search")
    opt = _opt_max_load([t.cost for t in tiles], cfg.V)
    assert max(loads) >= opt
    fmax = max(t.cost for t in tiles)
    assert max(loads) <= max(1.03 * sum(loads) / cfg.V, opt) + fmax


def test_q_ranges_select_whole_blocks():
    w = wl.workload(wl.W_256K, scale=16)       # 16384-token pack, CP=16 share of rank 0
    cfg = _cfg(w)
    full = op.build_tiles(cfg, w.lengths, w.pack_tokens)
    share = op.build_tiles(cfg, w.lengths, w.pack_tokens, w.q_ranges)
    ids = {t.id for t in share}
    assert ids == {t.id for t in full
                   if any(b <= t.q_begin and t.q_end <= e for b, e in w.q_ranges)}
    rows = sorted((t.q_row, t.q_begin, t.q_end) for t in share if t.id % w.H == 0)
    nxt = 0
    for r, b, e in rows:
        assert r == nxt
        nxt += e - b
    assert nxt == w.n_q_rows
