"""GPU parity on the five workloads, in the launch configuration bench.py times.

bench.py runs the pool's eight virtual workers as separate launches that add
into fp32 dK / dV (accumulate mode) and the single-set workloads with bf16
dK / dV; every test below uses the same mode unless it says otherwise.

* reduced replicas of the pool, 256K-share and 1M-share workloads (same
  generator, every token count and the block size divided by a power of
  two): every output element against the float64 oracle, at the fixed
  bounds (max-abs 2e-2 beyond bf16 storage rounding, relative L2 1e-2); the
  1M replica also in accumulate mode;
* the four large workloads at full size: O, LSE and dQ of a few hundred
  deterministic rows (every tile's first and last row, rows either side of
  32-row item edges, sample starts, the longest sample's rows, random rows;
  all heads), which the oracle computes row by row; and dK / dV of every KV
  head from a second backward whose dO is zero except on a subset of those
  rows (then only those rows contribute, and the oracle computes the result
  exactly);
* the same four with K = 0: every row's O is the prefix mean of V,
  LSE = ln(q_loc + 1), dQ = 0, and dV and dK have closed forms (reverse
  prefix sums and suffix sums, tests/closed_forms.py), so every output
  element is checked at full size.
"""
import functools

import numpy as np
import pytest
import torch

import paper_2607_23250_amd as pl
from oracle import attention as oa
import workloads as wl
import closed_forms as cf
from gpu_util import DEV, LSE_TOL, check, cu_dev, plan, say, to_np

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=4)
def _tensors(name, scale=1):
    """Seeded inputs of a workload (cached: the largest take tens of seconds to draw)."""
    w = wl.workload(name, scale=scale)
    return wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)


def _launch_sets(w):
    """Tile sets as bench.py launches them."""
    full, _ = plan(w)
    if w.q_ranges is not None:
        return [plan(w, w.q_ranges)[0]]
    if w.per_worker:
        return [full[full["worker"] == r] for r in range(w.V) if (full["worker"] == r).any()]
    return [full]


def _run(w, sets, q, k, v, do, accumulate=None):
    """fwd + bwd of every tile set (accumulate: bench.py's choice when None);
    returns device tensors."""
    acc = len(sets) > 1 if accumulate is None else accumulate
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    cu = cu_dev(w)
    o = torch.empty_like(qd)
    lse = torch.empty((w.h_q, w.n_q_rows), dtype=torch.float32, device=DEV)
    dq = torch.empty_like(qd)
    kv_dtype = torch.float32 if acc else torch.bfloat16
    dk = torch.zeros(kd.shape, dtype=kv_dtype, device=DEV)
    dv = torch.zeros_like(dk)
    tds = [pl.tiles_to_device(s, DEV) for s in sets]
    for td in tds:
        pl.libra_attn_fwd(qd, kd, vd, cu, td, o=o, lse=lse)
    for td in tds:
        pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dq=dq, dk=dk, dv=dv, accumulate=acc)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv, acc


@pytest.mark.parametrize("name,scale,acc", [(wl.W_POOL, 16, None), (wl.W_256K, 16, None),
                                            (wl.W_1M, 64, None), (wl.W_1M, 64, True)])
def test_replica_full_parity(name, scale, acc):
    w = wl.workload(name, scale=scale)
    sets = _launch_sets(w)
    say(f"[replica {name}/{scale} accumulate={acc}] rows={w.n_q_rows} keys={w.n_kv_rows} "
        f"samples={len(w.lengths)} max={max(w.lengths)} launches={len(sets)}")
    q, kk, v, do = wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)
    o, lse, dq, dk, dv, acc = _run(w, sets, q, kk, v, do, accumulate=acc)
    pos = w.q_positions()
    O, LSE = oa.attention_fwd(q, kk, v, w.lengths, pos)
    check("O", to_np(o), O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))
    dQ, dK, dV = oa.attention_bwd(q, kk, v, do, w.lengths, pos)
    check("dQ", to_np(dq), dQ, bf16_out=True)
    check("dK" + (" fp32" if acc else ""), to_np(dk), dK, bf16_out=not acc)
    check("dV" + (" fp32" if acc else ""), to_np(dv), dV, bf16_out=not acc)


def _sample_rows(w, sets, n_random, seed):
    """Deterministic rows: the first and last row of every tile, rows on both
    sides of two 32-row item edges per tile, the first row of up to 64
    samples spread over the pool, the first / last / evenly spaced rows of
    the longest sample, plus random rows."""
    pos = w.q_positions()
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    rng = np.random.default_rng(seed)
    rows = set()
    for s in sets:
        for t in s:
            r0, r1 = int(t["q_row"]), int(t["q_row"] + t["q_end"] - t["q_begin"]) - 1
            rows.update((r0, r1))
            n_edges = (r1 - r0) // 32
            for e in rng.integers(1, n_edges + 1, 2) if n_edges >= 1 else ():
                rows.update((r0 + 32 * int(e) - 1, r0 + 32 * int(e)))
    j_long = int(np.argmax(w.lengths))
    present = np.nonzero((pos >= cu[j_long]) & (pos < cu[j_long + 1]))[0]
    if len(present):
        rows.update(int(x) for x in present[[0, -1, -2]])
        rows.update(int(x) for x in present[np.linspace(0, len(present) - 1, 8).astype(int)])
    starts = np.searchsorted(pos, cu[:-1])
    for j in np.unique(np.linspace(0, len(w.lengths) - 1, 64).astype(int)):
        if starts[j] < len(pos) and pos[starts[j]] == cu[j]:
            rows.add(int(starts[j]))
    rows.update(int(x) for x in rng.integers(0, len(pos), n_random))
    return np.array(sorted(r for r in rows if 0 <= r < len(pos)), dtype=np.int64)


def _probe_rows(w, rows, seed):
    """Rows of the sparse-dO probe: eight of the longest sample's sampled rows
    (the costly ones for the oracle) and 24 others."""
    pos = w.q_positions()
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    j_long = int(np.argmax(w.lengths))
    in_long = (pos[rows] >= cu[j_long]) & (pos[rows] < cu[j_long + 1])
    longs, others = rows[in_long], rows[~in_long]
    rng = np.random.default_rng(seed)
    pick = list(longs[np.linspace(0, len(longs) - 1, min(8, len(longs))).astype(int)]) \
        if len(longs) else []
    if len(others):
        pick += list(rng.choice(others, min(24, len(others)), replace=False))
    return np.array(sorted(set(int(x) for x in pick)), dtype=np.int64)


@pytest.mark.parametrize("name", wl.WORKLOADS[1:])
def test_full_size_sampled_rows(name):
    w = wl.workload(name)
    sets = _launch_sets(w)
    rows = _sample_rows(w, sets, 32, seed=w.seed)
    probe = _probe_rows(w, rows, seed=w.seed + 1)
    say(f"[full {name}] rows={w.n_q_rows} keys={w.n_kv_rows} launches={len(sets)} "
        f"sampled rows={len(rows)} probe rows={len(probe)}")
    q, kk, v, do = _tensors(name)
    o, lse, dq, _, _, acc = _run(w, sets, q, kk, v, do)
    pos = w.q_positions()
    say("  oracle forward rows ...")
    O, LSE = oa.attention_fwd(q, kk, v, w.lengths, pos, rows=rows)
    check("O rows", to_np(o[rows.tolist()]), O, bf16_out=True)
    check("LSE rows", to_np(lse[:, rows.tolist()]), LSE, (LSE_TOL, 1e-4))
    say("  oracle dQ rows ...")
    dQ, _, _ = oa.attention_bwd(q, kk, v, do, w.lengths, pos, rows=rows, dkdv=False)
    check("dQ rows", to_np(dq[rows.tolist()]), dQ, bf16_out=True)
    # sparse-dO probe: only the probe rows carry gradient, every KV head
    do_s = torch.zeros_like(do)
    do_s[probe] = do[probe]
    _, _, dq2, dk2, dv2, _ = _run(w, sets, q, kk, v, do_s)
    say("  oracle probe ...")
    dQ2, dK, dV = oa.attention_bwd(q, kk, v, do_s, w.lengths, pos, rows=probe)
    check("dQ probe rows", to_np(dq2[probe.tolist()]), dQ2, bf16_out=True)
    for g in range(w.h_kv):
        check(f"dK probe kv {g}" + (" fp32" if acc else ""), to_np(dk2[:, g]), dK[:, g],
              bf16_out=not acc)
        check(f"dV probe kv {g}" + (" fp32" if acc else ""), to_np(dv2[:, g]), dV[:, g],
              bf16_out=not acc)


@pytest.mark.parametrize("name", wl.WORKLOADS[1:])
def test_full_size_zero_k_closed_forms(name):
    w = wl.workload(name)
    say(f"[full {name} K=0] rows={w.n_q_rows} keys={w.n_kv_rows}")
    _check_zero_k(w, *_tensors(name))


def test_many_long_samples_zero_k():
    """More samples longer than 64 key blocks of 128 keys than the dK/dV item
    builder lists for whole-workgroup enumeration (256): its per-thread path
    then takes every sample; every output is checked against the K = 0 closed
    forms."""
    n_long, ell = 300, 8256                  # 65 key blocks each
    w = wl.Workload("long300", 7, [[ell] * n_long], 2, 1, 64, B=8192, H=1, CP=1)
    say(f"[many long samples K=0] samples={n_long} x {ell} rows={w.n_q_rows}")
    _check_zero_k(w, *wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d))


def _check_zero_k(w, q, kk, v, do):
    """fwd + bwd with K = 0 in bench.py's launch configuration, every output
    element against its closed form."""
    sets = _launch_sets(w)
    kk = torch.zeros_like(kk)
    o, lse, dq, dk, dv, acc = _run(w, sets, q, kk, v, do)
    pos = w.q_positions()
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    j_of = np.searchsorted(cu, pos, side="right") - 1
    qloc = pos - cu[j_of]
    G = w.h_q // w.h_kv
    # LSE = ln(q_loc + 1) for every head
    want_lse = np.broadcast_to(np.log(qloc + 1.0), (w.h_q, len(pos)))
    check("LSE", to_np(lse), want_lse, (LSE_TOL, 1e-4))
    assert torch.count_nonzero(dq).item() == 0, "dQ must be exactly zero when K = 0"
    o_np = to_np(o)
    tag = " fp32" if acc else ""
    for g in range(w.h_kv):
        v64 = v[:, g].double().numpy()
        hs = slice(g * G, (g + 1) * G)
        q64, do64 = q[:, hs].double().numpy(), do[:, hs].double().numpy()
        mean = cf.prefix_mean_v(v64, w.lengths, pos)
        for h in range(g * G, (g + 1) * G):
            check(f"O head {h}", o_np[:, h], mean, bf16_out=True)
        want_dv = cf.zero_k_dv(do64, w.lengths, pos, w.n_kv_rows)
        check(f"dV kv {g}{tag}", to_np(dv[:, g]), want_dv, bf16_out=not acc)
        want_dk = cf.zero_k_dk(q64, do64, v64, w.lengths, pos, w.n_kv_rows,
                               1.0 / np.sqrt(w.d))
        check(f"dK kv {g}{tag}", to_np(dk[:, g]), want_dk, bf16_out=not acc)
