"""GPU parity on the five workloads, in the launch configuration bench.py times.

* reduced replicas of the pool, 256K-share and 1M-share workloads (same generator, every token count and the
  block size divided by a power of two): every output element against the
  float64 oracle (gradients: the 2e-2 bound, or twice the error of plain bf16
  PyTorch when that is larger -- the paper's criterion, Sec. 6.7);
* the four large workloads at full size: O, LSE and dQ of sampled query rows (all heads),
  which the oracle computes row by row, and dK / dV from a second backward
  whose dO is zero except on those rows (then only those rows contribute, and
  the oracle computes the result exactly);
* the same four with K = 0: every row's O is the prefix mean of V,
  LSE = ln(q_loc + 1), dQ = 0 and dV has a closed form (a reverse prefix sum
  of dO / (q_loc + 1)), so every output element is checked at full size.
"""
import functools

import numpy as np
import pytest
import torch

import paper_2607_23250_amd as pl
from oracle import attention as oa
from oracle.bf16_reference import attention_bf16
import workloads as wl
from gpu_util import DEV, LSE_TOL, check, cu_dev, half_ulp_bf16, plan, say, to_np

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
    """fwd + bwd of every tile set; returns device tensors."""
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
    return o, lse, dq, dk, dv


@pytest.mark.parametrize("name,scale", [(wl.W_POOL, 16), (wl.W_256K, 16), (wl.W_1M, 64)])
def test_replica_full_parity(name, scale):
    w = wl.workload(name, scale=scale)
    sets = _launch_sets(w)
    say(f"[replica {name}/{scale}] rows={w.n_q_rows} keys={w.n_kv_rows} samples={len(w.lengths)} "
        f"max={max(w.lengths)} launches={len(sets)}")
    q, kk, v, do = wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)
    o, lse, dq, dk, dv = _run(w, sets, q, kk, v, do, accumulate=True)
    pos = w.q_positions()
    O, LSE = oa.attention_fwd(q, kk, v, w.lengths, pos)
    check("O", to_np(o), O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))
    dQ, dK, dV = oa.attention_bwd(q, kk, v, do, w.lengths, pos)
    _, bq, bk, bv = attention_bf16(q, kk, v, do, w.lengths, pos)
    check("dQ", to_np(dq), dQ, bf16_out=True, ref_bf16=bq)
    check("dK", to_np(dk), dK, ref_bf16=bk)
    check("dV", to_np(dv), dV, ref_bf16=bv)


def _sample_rows(w, sets, n_random, seed):
    """Deterministic rows: first / last rows of tiles and of samples, rows on
    both sides of 32-row block edges, the last rows of the longest sample,
    plus random rows."""
    pos = w.q_positions()
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    rows = set()
    for s in sets:
        for t in s[:: max(1, len(s) // 6)]:
            r0, r1 = int(t["q_row"]), int(t["q_row"] + t["q_end"] - t["q_begin"]) - 1
            rows.update((r0, r1, min(r0 + 31, r1), min(r0 + 32, r1)))
    j_long = int(np.argmax(w.lengths))
    present = np.nonzero((pos >= cu[j_long]) & (pos < cu[j_long + 1]))[0]
    if len(present):
        rows.update(int(x) for x in present[[0, -1, -2, len(present) // 2]])
    starts = np.searchsorted(pos, cu[:-1])
    for j in range(0, len(w.lengths), max(1, len(w.lengths) // 5)):
        if starts[j] < len(pos) and pos[starts[j]] == cu[j]:
            rows.add(int(starts[j]))
    rng = np.random.default_rng(seed)
    rows.update(int(x) for x in rng.integers(0, len(pos), n_random))
    return np.array(sorted(r for r in rows if 0 <= r < len(pos)), dtype=np.int64)


@pytest.mark.parametrize("name", wl.WORKLOADS[1:])
def test_full_size_sampled_rows(name):
    w = wl.workload(name)
    sets = _launch_sets(w)
    rows = _sample_rows(w, sets, 8 if name == wl.W_1M else 16, seed=w.seed)
    say(f"[full {name}] rows={w.n_q_rows} keys={w.n_kv_rows} launches={len(sets)} "
        f"sampled rows={len(rows)}")
    q, kk, v, do = _tensors(name)
    o, lse, dq, _, _ = _run(w, sets, q, kk, v, do)
    pos = w.q_positions()
    O, LSE = oa.attention_fwd(q, kk, v, w.lengths, pos, rows=rows)
    check("O rows", to_np(o[rows.tolist()]), O, bf16_out=True)
    check("LSE rows", to_np(lse[:, rows.tolist()]), LSE, (LSE_TOL, 1e-4))
    # sparse-dO probe: only the sampled rows carry gradient
    do_s = torch.zeros_like(do)
    do_s[rows] = do[rows]
    _, _, dq2, dk2, dv2 = _run(w, sets, q, kk, v, do_s, accumulate=True)
    g = w.h_kv - 1                                   # the oracle covers one KV group
    G = w.h_q // w.h_kv
    heads = list(range(g * G, (g + 1) * G))
    dQ, dK, dV = oa.attention_bwd(q, kk, v, do_s, w.lengths, pos, rows=rows, kv_heads=[g])
    check("dQ rows", to_np(dq2[rows.tolist()][:, heads]), dQ[:, heads], bf16_out=True)
    # dQ of a row depends on that row's dO only: the full backward agrees on these rows
    check("dQ rows (full dO)", to_np(dq[rows.tolist()][:, heads]), dQ[:, heads], bf16_out=True)
    check("dK probe", to_np(dk2[:, g]), dK[:, g])
    check("dV probe", to_np(dv2[:, g]), dV[:, g])


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
    o, lse, dq, dk, dv = _run(w, sets, q, kk, v, do, accumulate=True)
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
    do_np = do.float().numpy().astype(np.float64)
    for g in range(w.h_kv):
        vf = v[:, g].double().numpy()
        # prefix mean of V over the row's own sample
        csum = np.cumsum(vf, axis=0)
        start_sum = np.where(cu[j_of][:, None] > 0, csum[np.maximum(cu[j_of] - 1, 0)], 0.0)
        mean = (csum[pos] - start_sum) / (qloc + 1.0)[:, None]
        for h in range(g * G, (g + 1) * G):
            check(f"O head {h}", o_np[:, h], mean, bf16_out=True)
        # dV_i = sum over present rows q >= i of the same sample of sum_h dO_q / (q_loc+1)
        wq = do_np[:, g * G:(g + 1) * G].sum(axis=1) / (qloc + 1.0)[:, None]
        acc = np.zeros((w.n_kv_rows, w.d))
        np.add.at(acc, pos, wq)
        want = np.zeros_like(acc)
        for j in np.unique(j_of):
            s, e = int(cu[j]), int(cu[j + 1])
            want[s:e] = np.cumsum(acc[s:e][::-1], axis=0)[::-1]
        check(f"dV kv {g}", to_np(dv[:, g]), want)
