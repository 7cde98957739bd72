"""GPU parity of libra_attn_fwd / libra_attn_bwd against the float64 oracle.

Every case prints its name and sizes before touching the GPU.  Outputs are
compared element by element at fixed bounds: max-abs <= 2e-2 and relative
L2 <= 1e-2 for O, dQ, dK, dV; max-abs <= 1e-3 for the log-sum-exp.  bf16
outputs meet the max-abs bound beyond their own storage rounding (half a
bf16 ulp of the exact value, which reaches 3e-2 for |dV| >= 8 when many
heads and queries are summed); fp32 outputs (accumulate-mode dK / dV) get no
allowance."""
import numpy as np
import pytest
import torch

import paper_2607_23250_amd as pl
from oracle import attention as oa
import workloads as wl
from gpu_util import DEV, LSE_TOL, check, cu_dev, fwd, plan, say, to_np

pytestmark = pytest.mark.gpu


def _inputs(w, seed=None, n_q=None):
    seed = w.seed if seed is None else seed
    n_q = w.n_q_rows if n_q is None else n_q
    return wl.tensors(seed, n_q, w.n_kv_rows, w.h_q, w.h_kv, w.d)


def _dev(*ts):
    return [t.to(DEV) for t in ts]


@pytest.mark.parametrize("seed", range(16))
def test_fwd_small_random(seed):
    w = wl.small_random(seed)
    say(f"[fwd small {seed}] packs={w.pack_tokens} n={len(w.lengths)} heads=({w.h_q},{w.h_kv}) "
        f"d={w.d} B={w.B} H={w.H}")
    tiles, _ = plan(w)
    q, k, v, _ = _inputs(w)
    o, lse = fwd(w, tiles, *_dev(q, k, v), cu_dev(w))
    torch.cuda.synchronize()
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    check("O", to_np(o), O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))


def _span_tiles(spans):
    """Hand-made tiles over one sample: (q_begin, q_end, head_begin, head_end)
    each, Q rows in span order.  Returns the tiles and the rows' positions."""
    tiles = np.zeros(len(spans), dtype=pl.TILE_DTYPE)
    pos, row = [], 0
    for i, (b, e, hb, he) in enumerate(spans):
        tiles[i] = (b, e, row, 0, hb, he, 0, 0, 0, i)
        pos.extend(range(b, e))
        row += e - b
    return tiles, np.asarray(pos, dtype=np.int64)


@pytest.mark.parametrize("h_q,h_kv,d", [(4, 2, 128), (8, 1, 64), (6, 2, 64)])
def test_fwd_split_k_few_rows_long_sample(h_q, h_kv, d):
    """Few rows and heads against a 65,536-token sample: fewer work items than
    workgroups, so the forward cuts them into key ranges (split K) and merges
    the partial results.  O and LSE of the covered pairs against the oracle."""
    L = 65536
    spans = [(L - 256, L, 0, 2), (30000, 30128, 2, 4), (4100, 4200, 0, 1)]
    tiles, pos = _span_tiles(spans)
    n_q = len(pos)
    say(f"[fwd split K] sample {L} rows={n_q} heads=({h_q},{h_kv}) d={d}")
    q, k, v, _ = wl.tensors(7, n_q, L, h_q, h_kv, d, with_dout=False)
    cu = torch.tensor([0, L], dtype=torch.int64, device=DEV)
    o = torch.zeros((n_q, h_q, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.zeros((h_q, n_q), dtype=torch.float32, device=DEV)
    qd, kd, vd = _dev(q, k, v)
    td = pl.tiles_to_device(tiles, DEV)
    pl.libra_attn_fwd(qd, kd, vd, cu, td, o=o, lse=lse)
    o2, lse2 = torch.zeros_like(o), torch.zeros_like(lse)
    pl.libra_attn_fwd(qd, kd, vd, cu, td, o=o2, lse=lse2)
    torch.cuda.synchronize()
    # the parts are merged in key order: the result does not depend on which
    # workgroup ran which part
    assert torch.equal(o, o2) and torch.equal(lse, lse2), "split-K forward not deterministic"
    O, LSE = oa.attention_fwd(q, k, v, [L], pos, heads=range(4))
    cov = _coverage(tiles, n_q, h_q)
    check("O", to_np(o)[cov], O[cov], bf16_out=True)
    check("LSE", to_np(lse).T[cov], LSE.T[cov], (LSE_TOL, 1e-4))


@pytest.mark.parametrize("h_q,h_kv,d", [(4, 2, 128), (8, 1, 64), (6, 2, 64)])
def test_bwd_split_k_few_rows_long_sample(h_q, h_kv, d):
    """The split-K case of the forward test above through the backward: the
    dQ kernel's items split the same way, and its merge writes dQ and the
    -D records that the dK / dV kernel reads.  dQ of the covered pairs and
    dK / dV (bf16 and fp32) against the oracle, with dO zero outside them."""
    L = 65536
    spans = [(L - 256, L, 0, 2), (30000, 30128, 2, 4), (4100, 4200, 0, 1)]
    tiles, pos = _span_tiles(spans)
    n_q = len(pos)
    say(f"[bwd split K] sample {L} rows={n_q} heads=({h_q},{h_kv}) d={d}")
    q, k, v, do = wl.tensors(8, n_q, L, h_q, h_kv, d)
    cov = torch.from_numpy(_coverage(tiles, n_q, h_q))[:, :, None]
    do = torch.where(cov, do, torch.zeros_like(do))
    cu = torch.tensor([0, L], dtype=torch.int64, device=DEV)
    qd, kd, vd, dod = _dev(q, k, v, do)
    td = pl.tiles_to_device(tiles, DEV)
    o = torch.zeros((n_q, h_q, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.zeros((h_q, n_q), dtype=torch.float32, device=DEV)
    pl.libra_attn_fwd(qd, kd, vd, cu, td, o=o, lse=lse)
    dq = torch.zeros_like(qd)
    dq, dk, dv = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dq=dq)
    dq2 = torch.zeros_like(qd)
    dq2, dk2, dv2 = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dq=dq2)
    dk32 = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv32 = torch.zeros_like(dk32)
    pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dk=dk32, dv=dv32, accumulate=True)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq2) and torch.equal(dk, dk2) and torch.equal(dv, dv2), \
        "split-K backward not deterministic"
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, [L], pos)
    c = cov.expand_as(q).numpy()
    check("dQ covered", to_np(dq)[c], np.asarray(dQ)[c], bf16_out=True)
    check("dK", to_np(dk), dK, bf16_out=True)
    check("dV", to_np(dv), dV, bf16_out=True)
    check("dK fp32", to_np(dk32), dK)
    check("dV fp32", to_np(dv32), dV)


@pytest.mark.parametrize("h_q,h_kv,d", [(4, 2, 128), (4, 1, 64)])
def test_bwd_split_k_parts_sum_their_own_keys(h_q, h_kv, d):
    """Split K in the backward with the rows' attention held by every 32nd
    key block (blocks 28 mod 32: the fourth-last block of each 32-block key
    range), and dP taking different values on those blocks.  Each part of a
    split dQ item adds up dS over its key blocks for the D correction that
    the dK / dV kernel reads.  Here, counting the fourth-last block of every
    part but the last twice (a CPU emulation with these inputs) moves dK by
    0.16 (d = 128) and 0.24 (d = 64) in max-abs and by 0.24 in relative L2,
    far beyond the bounds.  Rows L - 256 .. L of a 65,536-token sample, query heads 0 and 1;
    small noise in every tensor."""
    L = 65536
    tiles, pos = _span_tiles([(L - 256, L, 0, 2)])
    n_q = len(pos)
    say(f"[bwd split K, concentrated attention] sample {L} rows={n_q} heads=({h_q},{h_kv}) d={d}")
    gen = torch.Generator().manual_seed(31)
    noise = lambda *shape: 0.1 * torch.randn(*shape, generator=gen)
    blk = torch.arange(L) // 64
    held = blk % 32 == 28
    sign = torch.where(blk // 32 >= 30, -15.0, 1.0)
    k = noise(L, h_kv, d)
    k[:, :, 0] = torch.where(held, 11.0, -11.0)[:, None]
    k[:, :, 2] = torch.where(held, sign, 0.0)[:, None]   # dQ of order 1
    v = noise(L, h_kv, d)
    v[:, :, 1] = torch.where(held, sign, 0.0)[:, None]
    q = noise(n_q, h_q, d)
    q[:, :, 0] = 8.0
    do = torch.zeros(n_q, h_q, d)
    do[:, :2] = noise(n_q, 2, d)
    do[:, :2, 1] = 1.0
    q, k, v, do = (t.to(torch.bfloat16) for t in (q, k, v, do))
    cu = torch.tensor([0, L], dtype=torch.int64, device=DEV)
    qd, kd, vd, dod = _dev(q, k, v, do)
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(qd, kd, vd, cu, td)
    dq, dk, dv = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td)
    dk32 = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv32 = torch.zeros_like(dk32)
    pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dk=dk32, dv=dv32, accumulate=True)
    torch.cuda.synchronize()
    O, LSE = oa.attention_fwd(q, k, v, [L], pos, heads=range(2))
    check("O", to_np(o)[:, :2], O[:, :2], bf16_out=True)
    check("LSE", to_np(lse)[:2], LSE[:2], (LSE_TOL, 1e-4))
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, [L], pos)
    check("dQ covered", to_np(dq)[:, :2], np.asarray(dQ)[:, :2], bf16_out=True)
    check("dK", to_np(dk), dK, bf16_out=True)
    check("dV", to_np(dv), dV, bf16_out=True)
    check("dK fp32", to_np(dk32), dK)
    check("dV fp32", to_np(dv32), dV)


@pytest.mark.parametrize("seed", range(16))
def test_bwd_small_random(seed):
    w = wl.small_random(seed)
    say(f"[bwd small {seed}] packs={w.pack_tokens} n={len(w.lengths)} heads=({w.h_q},{w.h_kv}) "
        f"d={w.d} B={w.B} H={w.H}")
    tiles, _ = plan(w)
    q, k, v, do = _inputs(w)
    qd, kd, vd, dod = _dev(q, k, v, do)
    cu = cu_dev(w)
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(qd, kd, vd, cu, td)
    dq, dk, dv = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td)
    torch.cuda.synchronize()
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    check("dQ", to_np(dq), dQ, bf16_out=True)
    check("dK", to_np(dk), dK, bf16_out=True)
    check("dV", to_np(dv), dV, bf16_out=True)
    # fp32 dK / dV of the same call in accumulate mode
    dk32 = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv32 = torch.zeros_like(dk32)
    pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dk=dk32, dv=dv32, accumulate=True)
    torch.cuda.synchronize()
    check("dK fp32", to_np(dk32), dK)
    check("dV fp32", to_np(dv32), dV)


# Inputs scaled by powers of two, with the score scale a * b = 1 so that S,
# P and LSE are unchanged: O scales by c, dV by e, dQ by e c b, dK by e c a.
# The rescaled outputs must match the oracle of the unscaled inputs.  These
# exercise the backward's fp16 operand scaling in both directions (tiny dO
# or V scaled up; large Q, K, V or dO scaled down).
MAGNITUDES = [(0, 0, 0, -14), (0, 0, 0, 13), (0, 0, 12, 0), (0, 0, -12, 0),
              (-6, 6, 0, 0), (5, -5, 0, 0), (4, -4, -8, 10)]


@pytest.mark.parametrize("exps", MAGNITUDES, ids=lambda e: "q%d_k%d_v%d_do%d" % tuple(e))
def test_bwd_input_magnitudes(exps):
    a, b, c, e = (2.0 ** x for x in exps)
    w = wl.small_random(3)
    say(f"[bwd magnitudes q*{a:g} k*{b:g} v*{c:g} dO*{e:g}] packs={w.pack_tokens} "
        f"heads=({w.h_q},{w.h_kv}) d={w.d}")
    tiles, _ = plan(w)
    q, k, v, do = _inputs(w)
    qd, kd, vd, dod = _dev(q * a, k * b, v * c, do * e)
    cu = cu_dev(w)
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(qd, kd, vd, cu, td)
    dq, dk, dv = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td)
    dk32 = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv32 = torch.zeros_like(dk32)
    pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dk=dk32, dv=dv32, accumulate=True)
    torch.cuda.synchronize()
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    check("O", to_np(o) / c, O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))
    check("dQ", to_np(dq) / (e * c * b), dQ, bf16_out=True)
    check("dK", to_np(dk) / (e * c * a), dK, bf16_out=True)
    check("dV", to_np(dv) / e, dV, bf16_out=True)
    check("dK fp32", to_np(dk32) / (e * c * a), dK)
    check("dV fp32", to_np(dv32) / e, dV)


def test_fwd_config1_full():
    w = wl.workload(wl.W_4K)
    say(f"[fwd 4K] {w.name} samples={len(w.lengths)}")
    tiles, _ = plan(w)
    q, k, v, _ = _inputs(w)
    o, lse = fwd(w, tiles, *_dev(q, k, v), cu_dev(w))
    torch.cuda.synchronize()
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    check("O", to_np(o), O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))


def test_fwd_bwd_config2_quarter_full():
    w = wl.workload(wl.W_32K, scale=4)
    say(f"[fwd+bwd 32K/4] {w.name} samples={len(w.lengths)}")
    tiles, _ = plan(w)
    q, k, v, do = _inputs(w)
    qd, kd, vd, dod = _dev(q, k, v, do)
    cu = cu_dev(w)
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(qd, kd, vd, cu, td)
    dq, dk, dv = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td)
    torch.cuda.synchronize()
    say("  oracle forward ...")
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    check("O", to_np(o), O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))
    say("  oracle backward ...")
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    check("dQ", to_np(dq), dQ, bf16_out=True)
    check("dK", to_np(dk), dK, bf16_out=True)
    check("dV", to_np(dv), dV, bf16_out=True)


def test_fwd_independent_of_plan_and_worker_split():
    """Rows and heads are computed independently of how tiles group them:
    every plan, and every split of a plan into per-worker launches, gives
    bit-identical O and LSE."""
    w = wl.workload(wl.W_32K, scale=4)
    say(f"[plan invariance] {w.name}/4")
    q, k, v, _ = _inputs(w)
    qd, kd, vd = _dev(q, k, v)
    cu = cu_dev(w)
    ref = None
    for B, H in ((512, 2), (128, 4), (1024, 1), (300, 8)):
        w.B, w.H = B, H
        tiles, _ = plan(w)
        o = torch.full_like(qd, float("nan"))
        lse = torch.full((w.h_q, w.n_q_rows), float("nan"), device=DEV)
        for r in range(w.V):
            mine = tiles[tiles["worker"] == r]
            if len(mine):
                pl.libra_attn_fwd(qd, kd, vd, cu, pl.tiles_to_device(mine, DEV), o=o, lse=lse)
        torch.cuda.synchronize()
        got = (o.cpu(), lse.cpu())
        assert not torch.isnan(got[1]).any()
        if ref is None:
            ref = got
        else:
            assert torch.equal(got[0], ref[0]) and torch.equal(got[1], ref[1]), (B, H)


def test_fwd_packed_equals_unpacked():
    w = wl.workload(wl.W_32K, scale=4)
    say(f"[packed == unpacked] {w.name}/4")
    tiles, _ = plan(w)
    q, k, v, _ = _inputs(w)
    o, lse = fwd(w, tiles, *_dev(q, k, v), cu_dev(w))
    o, lse = o.cpu(), lse.cpu()
    start = 0
    for j, n in enumerate(w.lengths):
        if j % 3 == 0 or n > 1000:
            one = wl.Workload("one", 0, [[n + (n % 2)]], w.h_q, w.h_kv, w.d, B=w.B, H=w.H, CP=1)
            ts, _ = plan(one)
            sl = slice(start, start + n)
            pad = lambda t: torch.cat([t[sl], t[sl][:1]]) if n % 2 else t[sl]   # noqa: E731
            o1, lse1 = fwd(one, ts, *_dev(pad(q), pad(k), pad(v)), cu_dev(one))
            torch.cuda.synchronize()
            assert torch.equal(o1.cpu()[:n], o[sl]), j
            assert torch.equal(lse1.cpu()[:, :n], lse[:, sl]), j
        start += n


def test_fwd_deterministic():
    w = wl.workload(wl.W_32K, scale=2)
    say(f"[determinism] {w.name}/2")
    tiles, _ = plan(w)
    q, k, v, _ = _dev(*_inputs(w))
    cu = cu_dev(w)
    a = fwd(w, tiles, q, k, v, cu)
    b = fwd(w, tiles, q, k, v, cu)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("seed", range(4))
def test_bwd_per_worker_accumulate(seed):
    """Each virtual worker's tile set runs as its own launch; dK/dV partials
    are summed in fp32 by the library's accumulate mode."""
    w = wl.small_random(100 + seed)
    w.CP = 2 if all(p % 4 == 0 for p in w.pack_tokens) else 1
    say(f"[bwd per worker {seed}] packs={w.pack_tokens} V={w.V} heads=({w.h_q},{w.h_kv}) d={w.d}")
    tiles, _ = plan(w)
    q, k, v, do = _inputs(w)
    qd, kd, vd, dod = _dev(q, k, v, do)
    cu = cu_dev(w)
    o = torch.empty_like(qd)
    lse = torch.empty((w.h_q, w.n_q_rows), device=DEV)
    dq = torch.empty_like(qd)
    dk = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv = torch.zeros_like(dk)
    for r in range(w.V):
        mine = tiles[tiles["worker"] == r]
        if not len(mine):
            continue
        td = pl.tiles_to_device(mine, DEV)
        pl.libra_attn_fwd(qd, kd, vd, cu, td, o=o, lse=lse)
        pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dq=dq, dk=dk, dv=dv, accumulate=True)
    torch.cuda.synchronize()
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    check("dQ", to_np(dq), dQ, bf16_out=True)
    check("dK", to_np(dk), dK)
    check("dV", to_np(dv), dV)


def _coverage(tiles, n_q, h_q):
    """(row, head) pairs that a tile list covers."""
    m = np.zeros((n_q, h_q), dtype=bool)
    for t in tiles:
        r0 = int(t["q_row"])
        m[r0:r0 + int(t["q_end"]) - int(t["q_begin"]), int(t["head_begin"]):int(t["head_end"])] = True
    return m


@pytest.mark.parametrize("seed", [200, 203, 207, 210, 211])
def test_bwd_ignores_uncovered_rows(seed):
    """One virtual worker's tile set, with NaN in every (row, head) of Q and
    dO that its tiles do not cover: dK / dV (bf16 and fp32) and the covered
    dQ match the oracle run with dO = 0 outside the covered pairs.  The
    dK / dV kernel stages whole 32-row blocks, so this checks that rows
    outside the tiles never reach its products."""
    w = wl.small_random(seed)
    w.CP = 2 if all(p % 4 == 0 for p in w.pack_tokens) else 1
    tiles, _ = plan(w)
    counts = np.bincount(tiles["worker"], minlength=w.V)
    mine = tiles[tiles["worker"] == int(np.argmax(counts))]
    say(f"[bwd uncovered NaN {seed}] packs={w.pack_tokens} V={w.V} tiles={len(mine)} "
        f"heads=({w.h_q},{w.h_kv}) d={w.d}")
    q, k, v, do = _inputs(w)
    cov = torch.from_numpy(_coverage(mine, w.n_q_rows, w.h_q))[:, :, None]
    nan = torch.tensor(float("nan"), dtype=q.dtype)
    qd, kd, vd, dod = _dev(torch.where(cov, q, nan), k, v, torch.where(cov, do, nan))
    cu = cu_dev(w)
    td = pl.tiles_to_device(mine, DEV)
    o = torch.zeros_like(qd)
    lse = torch.zeros((w.h_q, w.n_q_rows), device=DEV)
    pl.libra_attn_fwd(qd, kd, vd, cu, td, o=o, lse=lse)
    dq = torch.zeros_like(qd)
    dq, dk, dv = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dq=dq)
    dk32 = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv32 = torch.zeros_like(dk32)
    pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dk=dk32, dv=dv32, accumulate=True)
    torch.cuda.synchronize()
    dQ, dK, dV = oa.attention_bwd(q, k, v, torch.where(cov, do, torch.zeros_like(do)),
                                  w.lengths, w.q_positions())
    c = cov.expand_as(q).numpy()
    check("dQ covered", to_np(dq)[c], np.asarray(dQ)[c], bf16_out=True)
    check("dK", to_np(dk), dK, bf16_out=True)
    check("dV", to_np(dv), dV, bf16_out=True)
    check("dK fp32", to_np(dk32), dK)
    check("dV fp32", to_np(dv32), dV)


def test_empty_tile_list():
    """No tiles: the forward writes nothing, the backward writes nothing but
    the zero dK / dV of bf16 mode (and adds nothing in accumulate mode)."""
    w = wl.small_random(0)
    say(f"[empty tiles] heads=({w.h_q},{w.h_kv}) d={w.d}")
    q, k, v, do = _dev(*_inputs(w))
    cu = cu_dev(w)
    td = pl.tiles_to_device(np.zeros(0, dtype=pl.TILE_DTYPE), DEV)
    o = torch.full_like(q, 7.0)
    lse = torch.full((w.h_q, w.n_q_rows), 7.0, dtype=torch.float32, device=DEV)
    pl.libra_attn_fwd(q, k, v, cu, td, o=o, lse=lse)
    dq = torch.full_like(q, 7.0)
    dk, dv = torch.full_like(k, 7.0), torch.full_like(v, 7.0)
    pl.libra_attn_bwd(q, k, v, o, lse, do, cu, td, dq=dq, dk=dk, dv=dv)
    dk32 = torch.full(k.shape, 7.0, dtype=torch.float32, device=DEV)
    dv32 = torch.full_like(dk32, 7.0)
    pl.libra_attn_bwd(q, k, v, o, lse, do, cu, td, dq=dq, dk=dk32, dv=dv32, accumulate=True)
    torch.cuda.synchronize()
    assert bool((o == 7.0).all()) and bool((lse == 7.0).all()) and bool((dq == 7.0).all())
    assert torch.count_nonzero(dk).item() == 0 and torch.count_nonzero(dv).item() == 0
    assert bool((dk32 == 7.0).all()) and bool((dv32 == 7.0).all())


def test_out_of_range_tiles_are_skipped():
    """Tiles outside the buffers are skipped on the device and counted (read
    back with libra_attn_skipped_tiles, the int32 at LIBRA_WS_SKIPPED_OFFSET);
    the other tiles' results are bit-identical to a call without them."""
    w = wl.small_random(5)
    say(f"[out-of-range tiles] heads=({w.h_q},{w.h_kv}) d={w.d} rows={w.n_q_rows}")
    tiles, _ = plan(w)
    bad = np.zeros(3, dtype=pl.TILE_DTYPE)
    bad[0] = tiles[0]
    bad[0]["q_end"] = w.n_kv_rows + 64                  # keys past the buffer
    bad[1] = tiles[0]
    bad[1]["head_end"] = w.h_q + 1                      # heads past the buffer
    bad[2] = tiles[0]
    bad[2]["q_row"] = w.n_q_rows                        # rows past the buffer
    both = np.concatenate([tiles, bad])
    q, k, v, do = _dev(*_inputs(w))
    cu = cu_dev(w)
    outs = []
    for tl in (tiles, both):
        td = pl.tiles_to_device(tl, DEV)
        n = len(w.lengths)
        wsf = pl.alloc_workspace(pl.libra_attn_workspace_size(len(tl), n, w.n_q_rows, w.n_kv_rows,
                                                              w.h_q, w.h_kv, w.d, False), DEV)
        wsb = pl.alloc_workspace(pl.libra_attn_workspace_size(len(tl), n, w.n_q_rows, w.n_kv_rows,
                                                              w.h_q, w.h_kv, w.d, True), DEV)
        o, lse = pl.libra_attn_fwd(q, k, v, cu, td, workspace=wsf)
        dq, dk, dv = pl.libra_attn_bwd(q, k, v, o, lse, do, cu, td, workspace=wsb)
        torch.cuda.synchronize()
        skipped = (pl.libra_attn_skipped_tiles(wsf), pl.libra_attn_skipped_tiles(wsb))
        # the documented byte offset holds the same count
        assert skipped == (int(wsf[16:20].cpu().view(torch.int32).item()),
                           int(wsb[16:20].cpu().view(torch.int32).item()))
        outs.append(([to_np(x) for x in (o, lse, dq, dk, dv)], skipped))
    (ref, skip0), (got, skip1) = outs
    assert skip0 == (0, 0), skip0
    assert skip1 == (3, 3), skip1
    for name, a, b in zip(("O", "LSE", "dQ", "dK", "dV"), ref, got):
        assert np.array_equal(a, b), f"{name} changed when out-of-range tiles were added"


def _split_and_shuffle(tiles, seed):
    """The same (row, head) pairs as `tiles`, cut into pieces of very different
    lengths (single rows beside long remainders) and listed in shuffled order."""
    rng = np.random.default_rng(seed)
    out = []
    for t in tiles:
        n = int(t["q_end"] - t["q_begin"])
        cuts = sorted(set([0, n] + ([1, int(rng.integers(1, n))] if n > 2 else [])))
        for a, b in zip(cuts[:-1], cuts[1:]):
            p = t.copy()
            p["q_begin"], p["q_end"], p["q_row"] = t["q_begin"] + a, t["q_begin"] + b, t["q_row"] + a
            out.append(p)
    out = np.array(out, dtype=pl.TILE_DTYPE)
    return out[rng.permutation(len(out))]


@pytest.mark.parametrize("seed", range(4))
def test_fwd_bwd_ragged_shuffled_tiles(seed):
    """Work items are built by 32-row windows of the longest tile: tiles of one
    row next to long ones, in any list order, still cover every pair once."""
    w = wl.small_random(100 + seed)
    tiles = _split_and_shuffle(plan(w)[0], seed)
    say(f"[ragged tiles {seed}] packs={w.pack_tokens} n={len(w.lengths)} "
        f"heads=({w.h_q},{w.h_kv}) d={w.d} tiles={len(tiles)} "
        f"lengths {int((tiles['q_end'] - tiles['q_begin']).min())}.."
        f"{int((tiles['q_end'] - tiles['q_begin']).max())}")
    q, k, v, do = _inputs(w)
    qd, kd, vd, dod = _dev(q, k, v, do)
    cu = cu_dev(w)
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(qd, kd, vd, cu, td)
    dk32 = torch.zeros(kd.shape, dtype=torch.float32, device=DEV)
    dv32 = torch.zeros_like(dk32)
    dq, _, _ = pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cu, td, dk=dk32, dv=dv32,
                                 accumulate=True)
    torch.cuda.synchronize()
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    check("O", to_np(o), O, bf16_out=True)
    check("LSE", to_np(lse), LSE, (LSE_TOL, 1e-4))
    check("dQ", to_np(dq), dQ, bf16_out=True)
    check("dK fp32", to_np(dk32), dK)
    check("dV fp32", to_np(dv32), dV)
