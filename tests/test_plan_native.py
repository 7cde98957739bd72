"""libra_plan (C++) against the plan oracle: bit-exact tiles, costs,
placement, loads and received bytes on the five workloads and on random
small inputs; error paths forced from the host."""
import numpy as np
import pytest

import paper_2607_23250_amd as pl
from oracle import plan as op
import workloads as wl


def _native(w, q_ranges=None, **over):
    kw = dict(block_tokens=w.B, head_shards=w.H, cp=w.CP, num_q_heads=w.h_q,
              num_kv_heads=w.h_kv, head_dim=w.d)
    kw.update(over)
    return pl.libra_plan(w.lengths, w.pack_tokens, q_ranges=q_ranges, with_bytes=True, **kw)


def _oracle(w, q_ranges=None, elem_bytes=2, tau=(3, 100)):
    cfg = op.PlanCfg(B=w.B, H=w.H, P=w.P, CP=w.CP, h_q=w.h_q, h_kv=w.h_kv, d=w.d,
                     elem_bytes=elem_bytes, tau_num=tau[0], tau_den=tau[1])
    tiles, loads = op.plan(cfg, w.lengths, w.pack_tokens, q_ranges)
    return tiles, loads, op.worker_comm(tiles, cfg.V)


def _same(native, oracle):
    tiles, loads, recv = native
    otiles, oloads, orecv = oracle
    assert len(tiles) == len(otiles)
    for a, b in zip(tiles, otiles):
        got = (int(a["id"]), int(a["pack"]), int(a["q_begin"]), int(a["q_end"]), int(a["q_row"]),
               int(a["cost"]), int(a["head_begin"]), int(a["head_end"]), int(a["home"]),
               int(a["worker"]))
        want = (b.id, b.pack, b.q_begin, b.q_end, b.q_row, b.cost, b.head_begin, b.head_end,
                b.home, b.worker)
        assert got == want
    assert [int(x) for x in loads] == list(oloads)
    assert [int(x) for x in recv] == list(orecv)


@pytest.mark.parametrize("name", wl.WORKLOADS)
def test_workloads_bit_exact(name):
    w = wl.workload(name)
    _same(_native(w), _oracle(w))
    if w.q_ranges is not None:
        _same(_native(w, w.q_ranges), _oracle(w, w.q_ranges))


@pytest.mark.parametrize("name", wl.WORKLOADS)
def test_workloads_meet_load_target(name):
    w = wl.workload(name)
    tiles, loads, _ = _native(w)
    assert w.V * loads.max() / loads.sum() <= 1.05


@pytest.mark.parametrize("seed", range(1000))
def test_random_small_bit_exact(seed):
    w = wl.tiny_random(seed, max_packs=4, max_len=96)
    rng = np.random.default_rng(seed)
    tau = (int(rng.integers(0, 20)), int(rng.integers(1, 200)))
    eb = int(rng.choice([1, 2, 4]))
    _same(_native(w, elem_bytes=eb, tau=tau), _oracle(w, elem_bytes=eb, tau=tau))


@pytest.mark.parametrize("seed", range(200))
def test_random_q_ranges_bit_exact(seed):
    w = wl.tiny_random(seed + 1000, max_packs=3, max_len=96)
    rng = np.random.default_rng(seed)
    # whole blocks of each pack, chosen at random, merged into sorted ranges
    blocks = []
    off = 0
    for L in w.pack_tokens:
        for lo in range(off, off + L, w.B):
            blocks.append((lo, min(off + L, lo + w.B)))
        off += L
    keep = [b for b in blocks if rng.random() < 0.5] or blocks[:1]
    ranges = []
    for b, e in keep:
        if ranges and ranges[-1][1] == b:
            ranges[-1] = (ranges[-1][0], e)
        else:
            ranges.append((b, e))
    _same(_native(w, ranges), _oracle(w, ranges))


def test_size_query_and_enospc():
    w = wl.workload(wl.W_32K)
    tiles, _, _ = _native(w)
    import ctypes
    L = pl.lib()
    lengths = np.asarray(w.lengths, dtype=np.int64)
    cu = pl._offsets(lengths)
    pcu = pl._offsets(w.pack_tokens)
    cfg = pl._PlanCfg(w.B, w.H, w.P, w.CP, w.h_q, w.h_kv, w.d, 2, 3, 100)
    n = ctypes.c_int64(-1)
    out = np.zeros(3, dtype=pl.TILE_DTYPE)
    rc = L.libra_plan(ctypes.byref(cfg), pl._ptr(lengths), len(lengths), pl._ptr(cu), pl._ptr(pcu),
                      None, 0, pl._ptr(out), 3, ctypes.byref(n), None, None)
    assert rc == pl.LIBRA_ENOSPC and n.value == len(tiles)


def _expect(code, **kw):
    with pytest.raises(pl.LibraError) as e:
        pl.libra_plan(**kw)
    assert e.value.code == code


def test_error_paths():
    base = dict(lengths=[3, 5], pack_tokens=[8], block_tokens=4, head_shards=2, cp=1,
                num_q_heads=4, num_kv_heads=2, head_dim=64)
    pl.libra_plan(**base)
    _expect(pl.LIBRA_EINVAL, **{**base, "head_shards": 3})              # H does not divide h_q
    _expect(pl.LIBRA_EINVAL, **{**base, "num_kv_heads": 3})             # h_kv does not divide h_q
    _expect(pl.LIBRA_EINVAL, **{**base, "lengths": [3, 0, 5]})          # empty sample
    _expect(pl.LIBRA_EINVAL, **{**base, "pack_tokens": [4, 4]})         # pack cuts a sample
    _expect(pl.LIBRA_EINVAL, **{**base, "cp": 3})                       # 8 % 6 != 0
    _expect(pl.LIBRA_EINVAL, **{**base, "q_ranges": [(1, 4)]})          # not whole blocks
    _expect(pl.LIBRA_EINVAL, **{**base, "q_ranges": [(4, 8), (0, 4)]})  # unsorted
    _expect(pl.LIBRA_EINVAL, **{**base, "block_tokens": 0})
    _expect(pl.LIBRA_EINVAL, **{**base, "tau": (3, 0)})
    _expect(pl.LIBRA_EINVAL, **{**base, "head_shards": 4, "num_kv_heads": 3, "num_q_heads": 12})
    # costs beyond int64: one sample of 2^32 tokens with 2^31 heads per shard
    _expect(pl.LIBRA_EOVERFLOW, lengths=[1 << 32], pack_tokens=[1 << 32], block_tokens=1 << 30,
            head_shards=1, cp=1, num_q_heads=1 << 30, num_kv_heads=1, head_dim=64)


def _vrsp_pool(kind="256K", gbs=64, seed=1, P=8):
    """The heaviest Algorithm 1 pool of a synthetic window (the pool of the
    straggler emulation): its packs' sample lengths."""
    win = wl.vrsp_window(kind, gbs, seed)
    order, pool_load, _ = pl.libra_vrsp(win, P)
    k = int(np.argmax(pool_load))
    return [win[int(j)] for j in order[k * P:(k + 1) * P]]


def test_pool_of_eight_256k_packs_cp8_bit_exact():
    """64 workers (P = 8 packs of 262,144 tokens, CP = 8), B = 4096, H = 2:
    the largest placement the benchmarks run, bit-exact against the oracle."""
    packs = _vrsp_pool()
    L = 262144
    w = wl.Workload("pool8x256K-cp8", 0, packs, 32, 4, 128, B=4096, H=2, CP=8)
    assert w.pack_tokens == [L] * 8 and w.V == 64
    native, oracle = _native(w), _oracle(w)
    _same(native, oracle)
    assert w.V * native[1].max() / native[1].sum() <= 1.05


def test_pool_splits_partition_the_work():
    """The three splits of the pool straggler emulation: a head-parallel rank
    (h_q / CP heads, every row of its pack) times CP, the 2 CP zigzag shares
    of every pack, and Algorithm 2's workers each carry exactly the pool's
    h_q * sum l(l+1)/2 causal pairs, and each zigzag rank's rows are its head
    and tail chunks."""
    packs = _vrsp_pool()
    L, cp, h_q = 262144, 8, 32
    exact = h_q * sum(x * (x + 1) // 2 for p in packs for x in p)
    kw = dict(block_tokens=4096, num_q_heads=h_q, num_kv_heads=4, head_dim=128)
    uly = zig = 0
    for p in packs:
        t, _ = pl.libra_plan(p, [L], head_shards=cp, cp=1, **kw)
        first = t[t["head_begin"] == 0]
        assert (first["head_end"] == h_q // cp).all()
        assert first["q_begin"].min() == 0 and first["q_end"].max() == L
        uly += int(first["cost"].sum()) * cp
        c = L // (2 * cp)
        for r in range(cp):
            ranges = [(r * c, (r + 1) * c), ((2 * cp - 1 - r) * c, (2 * cp - r) * c)]
            tz, _ = pl.libra_plan(p, [L], head_shards=1, cp=cp, q_ranges=ranges, **kw)
            rows = np.concatenate([np.arange(a, b) for a, b in zip(tz["q_begin"], tz["q_end"])])
            want = np.concatenate([np.arange(a, b) for a, b in ranges])
            assert np.array_equal(np.sort(rows), want)
            zig += int(tz["cost"].sum())
    lengths = [x for p in packs for x in p]
    full, loads = pl.libra_plan(lengths, [L] * len(packs), head_shards=2, cp=cp, **kw)
    assert uly == exact and zig == exact
    assert int(full["cost"].sum()) == exact == int(loads.sum())
    assert sorted(set(full["worker"].tolist())) == list(range(len(packs) * cp))
