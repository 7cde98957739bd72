#!/usr/bin/env python3
"""Benchmark of the Libra hot path on one MI355X.

One step = the whole path over one batch of synthetic input: plan the
SH-Tiles (Eq. 6 costs + Algorithm 2, host C++), upload the tile list, run
the packed causal attention forward and backward kernels for every tile set.
The host plans step i+1 while the GPU runs step i, as the paper's
asynchronous planner does.

Default workload: one GPU's CP=16 head+tail share of a 1,048,576-token pack
(Qwen3-30B-A3B attention: 32 query heads, 4 KV heads, head_dim 128; 65,536
query rows against up to 1M causal keys, one ~900K-token sample), planned
over 16 virtual workers.  ``--workload NAME`` selects another of the five
seeded workloads.  Inputs are seeded synthetic tensors resident in HBM before the
timed region starts.

Prints ONE JSON line: useful causal-masked attention TFLOP/s of fwd+bwd
(4*d flops per causal same-sample (query, key) pair per query head forward,
10*d backward), its fraction of the bf16 dense MFMA peak, the planner's
max/mean worker load, the roofline entry of the dominant kernel (backward
main kernel, timed with HIP events on its own stream) and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA: 4096 flop/clk/CU x 256 CU x 2.4 GHz
METRIC = ("packed causal attention fwd+bwd useful TFLOP/s (and % bf16 MFMA peak); "
          "max/mean tile load")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="1M-cp16-share-qwen3-30b-a3b",
                    help="one of the seeded workloads: 4K-h2-kv1-d64, 32K-qwen3-8b, "
                         "pool8x64K-qwen3-30b-a3b, 256K-cp16-share-qwen3-235b-a22b, "
                         "1M-cp16-share-qwen3-30b-a3b")
    ap.add_argument("--cpu-rows", type=int, default=64,
                    help="query rows of the fixed subset the CPU oracle baseline runs on "
                         "(0 disables it)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="time budget of the oracle baseline of --vrsp")
    ap.add_argument("--vrsp", action="store_true",
                    help="only measure Variance-Reduced Sequence Placement (Algorithm 1) on the "
                         "host: time per GBS window and the inter-pool imbalance R - 1 against "
                         "production-order grouping, on synthetic 256K / 1M windows")
    ap.add_argument("--straggler", action="store_true",
                    help="one-GPU straggler emulation on the 1M-token pack: fwd+bwd time of each "
                         "of the 16 zigzag CP rank shares vs each of the 16 Libra worker tile "
                         "sets (Algorithm 2), plus throughput per call vs block length x heads")
    ap.add_argument("--straggler-pool", nargs="?", const="256K", choices=("256K", "1M"),
                    help="one-GPU straggler emulation on the heaviest VRSP pool of a synthetic "
                         "window: 256K = 8 packs of 262,144 tokens with CP=8, 1M = 4 packs of "
                         "1,048,576 tokens with CP=16 (64 workers either way); fwd+bwd time of "
                         "a head-parallel (Ulysses) rank of every pack, of all zigzag CP rank "
                         "shares, and of all Libra worker tile sets of the pool"),
    ap.add_argument("--simulate", action="store_true",
                    help="offline planner simulation (host only): the LLN estimate of Eq. 3 "
                         "against production-order grouping, and TAP's (B, H) grid on "
                         "VRSP-formed pools: load balance and exchanged bytes per worker")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain elementwise copy of a known size (1 GiB read, "
                         "1 GiB written, 3 launches): the reference the HBM byte counters "
                         "of the profiler are scaled by")
    return ap.parse_args()


def copy_calibration():
    import torch
    n = 1 << 28                                      # 2^28 fp32 = 1 GiB
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"kernel": "elementwise neg (copy)", "launches": 3,
                                           "read_bytes": 4 * n, "write_bytes": 4 * n}}),
          flush=True)


def vrsp_bench(seconds: float):
    """Algorithm 1 on synthetic optimizer-step windows (one host core)."""
    import ctypes
    import paper_2607_23250_amd as pl
    import workloads as wl
    from fractions import Fraction
    L = pl.lib()
    out_windows = []
    for kind, gbs in (("256K", 128), ("256K", 256), ("1M", 128), ("1M", 256)):
        packs = wl.vrsp_window(kind, gbs, seed=1)
        counts = [len(p) for p in packs]
        lengths = np.ascontiguousarray(np.concatenate([np.asarray(p, dtype=np.int64)
                                                       for p in packs]))
        cu = np.zeros(gbs + 1, dtype=np.int64)
        cu[1:] = np.cumsum(counts)
        order = np.zeros(gbs, dtype=np.int64)
        loads = np.zeros(gbs // 8, dtype=np.int64)
        args = (pl._ptr(lengths), len(lengths), pl._ptr(cu), gbs, 8, pl._ptr(order),
                pl._ptr(loads), None)
        assert L.libra_vrsp(*args) == 0
        n = 0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 0.5:
            for _ in range(50):
                L.libra_vrsp(*args)
            n += 50
        us = (time.perf_counter() - t0) * 1e6 / n
        rec = {"window": kind, "gbs": gbs, "pool_size": 8, "samples": int(len(lengths)),
               "us_per_window": round(us, 2)}
        if seconds > 0:
            from oracle import vrsp as ov
            m = 0
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < seconds / 4:
                ov.vrsp([ov.workload(p) for p in packs], 8)
                m += 1
            rec["oracle_us_per_window"] = round((time.perf_counter() - t0) * 1e6 / m, 1)
        out_windows.append(rec)

    def r_minus_1(loads_, P):
        return float(Fraction(int(max(loads_)) * len(loads_), int(sum(loads_))) - 1)

    sweep = {}
    for kind in ("256K", "1M"):
        rows = {}
        for P in (1, 2, 4, 8, 16, 32, 64):
            prod, bal = [], []
            for seed in range(8):
                packs = wl.vrsp_window(kind, 128, seed=100 + seed)
                _, loads, work = pl.libra_vrsp(packs, P)
                prod.append(r_minus_1(work.reshape(-1, P).sum(axis=1), P))
                bal.append(r_minus_1(loads, P))
            rows[str(P)] = {"production_order": round(float(np.mean(prod)), 4),
                            "vrsp": round(float(np.mean(bal)), 5)}
        sweep[kind] = rows
    main = next(r for r in out_windows if r["window"] == "1M" and r["gbs"] == 128)
    out = {"metric": "VRSP placement time per GBS window (host, one core)",
           "value": main["us_per_window"], "unit": "us", "higher_is_better": False,
           "data": "synthetic", "config": {"workload": "1M window, GBS 128, pool size 8"},
           "windows": out_windows,
           "imbalance_r_minus_1_gbs128_mean_of_8": sweep}
    if seconds > 0:
        out["cpu_baseline"] = {"value": main.get("oracle_us_per_window"), "unit": "us",
                               "cores": 1, "kind": "oracle",
                               "sample": "the same 1M window, GBS 128, pool size 8"}
    print(json.dumps(out), flush=True)


def straggler_bench():
    """Zigzag CP (every rank computes its head+tail share) against Libra's
    worker tile sets of the same 1,048,576-token pack, one set at a time on
    one GPU; the slowest set stands for the step's straggler.  Then the
    throughput of single calls of one tile (B rows x heads) from the middle
    of the 900K sample."""
    import torch
    import paper_2607_23250_amd as pl
    import workloads as wl
    dev = torch.device("cuda:0")
    w0 = wl.workload(wl.W_1M)
    cp = w0.CP
    g = torch.Generator(device=dev).manual_seed(11)

    def rnd(shape):
        return torch.randn(shape, device=dev, generator=g, dtype=torch.float32).to(torch.bfloat16)

    n_all = w0.n_kv_rows
    k = rnd((n_all, w0.h_kv, w0.d))
    v = rnd((n_all, w0.h_kv, w0.d))
    cu = np.zeros(len(w0.lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(w0.lengths)
    cud = torch.from_numpy(cu).to(dev)
    dk = torch.zeros((n_all, w0.h_kv, w0.d), dtype=torch.float32, device=dev)
    dv = torch.zeros_like(dk)

    def run_set(tiles, n_rows, q, do, o, lse, dq, reps=2):
        td = pl.tiles_to_device(tiles, dev)
        ws = pl.alloc_workspace(max(pl.libra_attn_workspace_size(len(tiles), len(w0.lengths),
                                                                   n_rows, n_all, w0.h_q,
                                                                   w0.h_kv, w0.d, b)
                                    for b in (False, True)), dev)
        times = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            pl.libra_attn_fwd(q, k, v, cud, td, o=o, lse=lse, workspace=ws)
            pl.libra_attn_bwd(q, k, v, o, lse, do, cud, td, dq=dq, dk=dk, dv=dv,
                              accumulate=True, workspace=ws)
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
        return min(times) * 1e3

    def flops(tiles):
        return 14.0 * w0.d * float(tiles["cost"].sum())

    # zigzag CP: rank r computes its head + tail chunk against every causal key
    share_rows = w0.n_q_rows
    q = rnd((share_rows, w0.h_q, w0.d))
    do = rnd((share_rows, w0.h_q, w0.d))
    o = torch.empty_like(q)
    dq = torch.empty_like(q)
    lse = torch.empty((w0.h_q, share_rows), dtype=torch.float32, device=dev)
    zig = []
    for r in range(cp):
        wr = wl.workload(wl.W_1M, rank=r)
        tiles = plan(pl, wr, wr.q_ranges)[0]
        ms = run_set(tiles, share_rows, q, do, o, lse, dq)
        zig.append({"rank": r, "ms": round(ms, 2), "tflop": round(flops(tiles) / 1e12, 2)})
        print(json.dumps({"zigzag_rank": zig[-1]}), file=sys.stderr, flush=True)
    del q, do, o, dq, lse
    # Libra: the whole pack planned over the same 16 workers
    full, loads = plan(pl, w0)
    q = rnd((n_all, w0.h_q, w0.d))
    do = rnd((n_all, w0.h_q, w0.d))
    o = torch.empty_like(q)
    dq = torch.empty_like(q)
    lse = torch.empty((w0.h_q, n_all), dtype=torch.float32, device=dev)
    lib = []
    for r in range(cp):
        tiles = full[full["worker"] == r]
        ms = run_set(tiles, n_all, q, do, o, lse, dq)
        lib.append({"worker": r, "ms": round(ms, 2), "tflop": round(flops(tiles) / 1e12, 2)})
        print(json.dumps({"libra_worker": lib[-1]}), file=sys.stderr, flush=True)
    # throughput per call: one tile of B rows x heads ending at row 450K of the
    # 900K sample (the pack's last sample)
    j = len(w0.lengths) - 1
    heat = {}
    for B in (1024, 2048, 4096, 8192, 16384):
        for heads in (2, 4, 8, 16, 32):
            end = int(cu[j]) + 450000
            t = np.zeros(1, dtype=pl.TILE_DTYPE)
            t["q_begin"], t["q_end"], t["q_row"] = end - B, end, end - B
            loc = np.arange(end - B, end) - cu[j]
            t["cost"] = heads * int((loc + 1).sum())
            t["head_begin"], t["head_end"] = 0, heads
            ms = run_set(t, n_all, q, do, o, lse, dq, reps=3)
            heat[f"B{B}_h{heads}"] = round(flops(t) / (ms * 1e-3) / 1e12, 1)
    zmax = max(x["ms"] for x in zig)
    lmax = max(x["ms"] for x in lib)
    out = {"metric": "one-GPU straggler emulation, 1M-token pack, 16 workers (fwd+bwd)",
           "value": round(zmax / lmax, 3), "unit": "x (zigzag max / Libra max)",
           "higher_is_better": True, "data": "synthetic",
           "config": {"workload": "1M-token pack (packs of the 1M workload), CP=16, B=8192, H=2"},
           "zigzag": {"max_ms": zmax, "mean_ms": round(float(np.mean([x["ms"] for x in zig])), 2),
                      "max_over_mean": round(zmax / float(np.mean([x["ms"] for x in zig])), 4),
                      "ranks": zig},
           "libra": {"max_ms": lmax, "mean_ms": round(float(np.mean([x["ms"] for x in lib])), 2),
                     "max_over_mean": round(lmax / float(np.mean([x["ms"] for x in lib])), 4),
                     "plan_load_max_over_mean": round(float(cp * loads.max() / loads.sum()), 4),
                     "workers": lib},
           "tflops_per_call_tile_B_x_heads": heat}
    print(json.dumps(out), flush=True)


def straggler_pool_bench(kind: str = "256K", pool_packs: int = 8, cp: int = 8, seed: int = 1,
                         gbs: int = 64, B: int = 4096, reps: int = 2):
    """The paper's core-attention straggler comparison (Sec. 6.3) on one GPU.

    A window of `gbs` packed sequences (the long-tailed 256K or 1M stand-in)
    is grouped into pools of `pool_packs` by Algorithm 1; the pool with the
    largest load (the one that sets the step) is run three ways, each worker's
    share fwd+bwd alone on the GPU, best of `reps`:
      * head-parallel CP (Ulysses) per pack: a rank computes every row of its
        pack for h_q / cp query heads, so the cp ranks of a pack are equal and
        one is timed per pack;
      * zigzag CP per pack: rank r computes its head and tail chunks, all heads;
      * Libra: the whole pool planned by Algorithm 2 (block B, H = 2) over
        pool_packs * cp workers.
    Every tile list comes from libra_plan; attention shapes are Qwen3-30B-A3B's
    (32 query heads, 4 KV heads, d = 128)."""
    import torch
    import paper_2607_23250_amd as pl
    import workloads as wl
    dev = torch.device("cuda:0")
    h_q, h_kv, d = 32, 4, 128
    L = wl.VRSP_WINDOWS[kind][0]
    win = wl.vrsp_window(kind, gbs, seed)
    order, pool_load, _ = pl.libra_vrsp(win, pool_packs)
    k_top = int(np.argmax(pool_load))
    packs = [win[int(j)] for j in order[k_top * pool_packs:(k_top + 1) * pool_packs]]
    lengths = [x for p in packs for x in p]
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(lengths)
    n_all = len(packs) * L
    g = torch.Generator(device=dev).manual_seed(12)

    def rnd(shape, chunk=1 << 20):
        """bf16 N(0, 1), drawn in fp32 a million rows at a time (bounded temporaries)."""
        out = torch.empty(shape, dtype=torch.bfloat16, device=dev)
        for i in range(0, shape[0], chunk):
            rows = min(chunk, shape[0] - i)
            out[i:i + rows] = torch.randn((rows,) + tuple(shape[1:]), device=dev, generator=g,
                                          dtype=torch.float32).to(torch.bfloat16)
        return out

    q, k, v, do = rnd((n_all, h_q, d)), rnd((n_all, h_kv, d)), rnd((n_all, h_kv, d)), \
        rnd((n_all, h_q, d))
    o, dq = torch.empty_like(q), torch.empty_like(q)
    lse = torch.empty((h_q, n_all), dtype=torch.float32, device=dev)
    dk = torch.zeros((n_all, h_kv, d), dtype=torch.float32, device=dev)
    dv = torch.zeros_like(dk)
    cud = torch.from_numpy(cu).to(dev)
    max_tiles = 4096
    ws = pl.alloc_workspace(pl.libra_attn_workspace_size(max_tiles, len(lengths), n_all, n_all,
                                                         h_q, h_kv, d, True), dev)

    def plan_tiles(pack_lengths_, cp_, H, q_ranges=None, offset=0):
        """Tiles of one pack, moved to its place in the pool; the buffers hold
        every row of the pool, so a tile's row is its pool position."""
        t, _ = pl.libra_plan(pack_lengths_, [L], block_tokens=B, head_shards=H, cp=cp_,
                             num_q_heads=h_q, num_kv_heads=h_kv, head_dim=d, q_ranges=q_ranges)
        t["q_begin"] += offset
        t["q_end"] += offset
        t["q_row"] = t["q_begin"]
        return t

    def run_set(tiles):
        assert 0 < len(tiles) <= max_tiles
        td = pl.tiles_to_device(tiles, dev)
        best = None
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            pl.libra_attn_fwd(q, k, v, cud, td, o=o, lse=lse, workspace=ws)
            pl.libra_attn_bwd(q, k, v, o, lse, do, cud, td, dq=dq, dk=dk, dv=dv,
                              accumulate=True, workspace=ws)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3
            best = ms if best is None else min(best, ms)
        return best, 14.0 * d * float(tiles["cost"].sum()) / 1e12

    def summary(items):
        ms = [x["ms"] for x in items]
        return {"max_ms": round(max(ms), 2), "mean_ms": round(float(np.mean(ms)), 2),
                "max_over_mean": round(max(ms) / float(np.mean(ms)), 4)}

    uly, zig = [], []
    for p, pk in enumerate(packs):
        off = p * L
        t = plan_tiles(pk, 1, cp, offset=off)           # head shards of width h_q / cp
        ms, tf = run_set(t[t["head_begin"] == 0])
        uly.append({"pack": p, "ms": round(ms, 2), "tflop": round(tf, 2)})
        print(json.dumps({"ulysses_rank_of_pack": uly[-1]}), file=sys.stderr, flush=True)
        for r in range(cp):
            c = L // (2 * cp)
            ranges = [(r * c, (r + 1) * c), ((2 * cp - 1 - r) * c, (2 * cp - r) * c)]
            ms, tf = run_set(plan_tiles(pk, cp, 1, q_ranges=ranges, offset=off))
            zig.append({"pack": p, "rank": r, "ms": round(ms, 2), "tflop": round(tf, 2)})
        print(json.dumps({"zigzag_pack_done": p, "max_ms": max(x["ms"] for x in zig[-cp:])}),
              file=sys.stderr, flush=True)
    full, loads = pl.libra_plan(lengths, [L] * len(packs), block_tokens=B, head_shards=2, cp=cp,
                                num_q_heads=h_q, num_kv_heads=h_kv, head_dim=d)
    lib = []
    for r in range(len(packs) * cp):
        ms, tf = run_set(full[full["worker"] == r])
        lib.append({"worker": r, "ms": round(ms, 2), "tflop": round(tf, 2)})
    print(json.dumps({"libra_workers_done": len(lib)}), file=sys.stderr, flush=True)
    su, sz, sl = summary(uly), summary(zig), summary(lib)
    pack_work = [sum(x * x for x in pk) for pk in packs]
    out = {"metric": f"one-GPU straggler emulation, VRSP pool of {len(packs)} packs of {L:,} "
                     f"tokens, CP={cp}, {len(packs) * cp} workers (fwd+bwd)",
           "value": round(su["max_ms"] / sl["max_ms"], 3),
           "unit": "x (head-parallel CP straggler / Libra straggler)",
           "higher_is_better": True, "data": "synthetic",
           "config": {"window": f"{gbs} packs of {L} tokens ({kind} stand-in law), seed {seed}",
                      "pool": f"the heaviest of {len(pool_load)} Algorithm 1 pools of "
                              f"{pool_packs}", "h_q": h_q, "h_kv": h_kv, "head_dim": d,
                      "cp": cp, "block_tokens": B, "head_shards": 2, "best_of": reps},
           "pack_sum_l2_max_over_mean": round(max(pack_work) / float(np.mean(pack_work)), 4),
           "zigzag_straggler_over_libra": round(sz["max_ms"] / sl["max_ms"], 3),
           "ulysses": dict(su, ranks_timed=uly),
           "zigzag": dict(sz, ranks=zig),
           "libra": dict(sl, plan_load_max_over_mean=round(float(len(loads) * loads.max()
                                                                 / loads.sum()), 4),
                         workers=lib)}
    print(json.dumps(out), flush=True)


def simulate():
    """Planner-only simulation on synthetic optimizer-step windows."""
    import math
    import paper_2607_23250_amd as pl
    import workloads as wl
    out = {"metric": "offline (P, H, B) simulation of the planner (host only)",
           "data": "synthetic", "lln": {}, "grid": {}}
    # (1) Eq. 3: E[R] ~ 1 + CV / sqrt(P) * sqrt(2 ln(D / P)) for random grouping
    for kind in ("256K", "1M"):
        rows = {}
        wins = [wl.vrsp_window(kind, 128, seed=200 + s) for s in range(8)]
        for P in (1, 2, 4, 8, 16, 32, 64):
            meas, pred = [], []
            for packs in wins:
                _, _, F = pl.libra_vrsp(packs, P)
                Ff = F.astype(np.float64)
                loads = Ff.reshape(-1, P).sum(axis=1)
                meas.append(loads.max() / (P * Ff.mean()))
                cv = Ff.std() / Ff.mean()
                pred.append(1 + cv / math.sqrt(P) * math.sqrt(2 * math.log(len(F) / P)))
            rows[str(P)] = {"measured_R": round(float(np.mean(meas)), 3),
                            "eq3_R": round(float(np.mean(pred)), 3)}
        out["lln"][kind] = rows
    # (2) TAP grid on VRSP pools (Sec. 6.6 settings)
    grids = {"256K": dict(cp=8, P=8, gbs=128, h_q=32, h_kv=16, Bs=(2048, 4096, 8192, 16384)),
             "1M": dict(cp=16, P=4, gbs=32, h_q=32, h_kv=4, Bs=(4096, 8192, 16384, 32768))}
    for kind, g in grids.items():
        packs = wl.vrsp_window(kind, g["gbs"], seed=300)
        order, _, _ = pl.libra_vrsp(packs, g["P"])
        pools = [[packs[i] for i in order[k * g["P"]:(k + 1) * g["P"]]]
                 for k in range(g["gbs"] // g["P"])]
        res = {}
        for B in g["Bs"]:
            for H in (1, 2, 4, 8):
                mm, recv_max, recv_tot, ms = [], [], [], []
                for pool in pools:
                    lengths = [x for pk in pool for x in pk]
                    t0 = time.perf_counter()
                    tiles, loads, recv = pl.libra_plan(
                        lengths, [sum(pk) for pk in pool], block_tokens=B, head_shards=H,
                        cp=g["cp"], num_q_heads=g["h_q"], num_kv_heads=g["h_kv"], head_dim=128,
                        with_bytes=True)
                    ms.append((time.perf_counter() - t0) * 1e3)
                    mm.append(len(loads) * loads.max() / loads.sum())
                    recv_max.append(recv.max())
                    recv_tot.append(recv.sum())
                res[f"B{B}_H{H}"] = {
                    "tiles_per_pack": int(len(tiles) // g["P"]),
                    "max_over_mean_load": round(float(np.mean(mm)), 4),
                    "max_worker_recv_GB": round(float(np.mean(recv_max)) / 1e9, 3),
                    "pool_recv_GB": round(float(np.mean(recv_tot)) / 1e9, 2),
                    "plan_ms": round(float(np.mean(ms)), 2)}
        out["grid"][kind] = {"setting": {k: v for k, v in g.items() if k != "Bs"}, "cells": res}
    print(json.dumps(out), flush=True)


def plan(pl, w, q_ranges=None):
    return pl.libra_plan(w.lengths, w.pack_tokens, block_tokens=w.B, head_shards=w.H, cp=w.CP,
                         num_q_heads=w.h_q, num_kv_heads=w.h_kv, head_dim=w.d, q_ranges=q_ranges)


def launch_sets(w, full_tiles, share_tiles):
    """Tile sets run as separate launches: one worker each for a pool (per-worker
    execution), else the whole (share) tile list."""
    if w.q_ranges is not None:
        return [share_tiles]
    if w.per_worker:
        return [full_tiles[full_tiles["worker"] == r] for r in range(w.V)
                if (full_tiles["worker"] == r).any()]
    return [full_tiles]


def traffic_entry(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 PMC summary of this
    kernel on this workload, or None when missing or taken on a different
    kernel source (sha256 over the listed source files, in order)."""
    path = os.path.join(ROOT, "profiles", f"{kernel}__{workload}__traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    srcs = rec.get("source", [])
    srcs = [srcs] if isinstance(srcs, str) else srcs
    h = hashlib.sha256()
    for name in srcs:
        src = os.path.join(ROOT, "paper_2607_23250_amd", "csrc", name)
        if not os.path.exists(src):
            return None
        h.update(open(src, "rb").read())
    if not srcs or h.hexdigest() != rec.get("source_sha256"):
        return None
    return rec.get("bytes_per_launch")


def mfma_loop_peak(pl, torch, dev):
    """Matrix-core throughput the device sustains under load: the library's
    reference loop of independent bf16 32x32x16 products, at one and two waves
    per SIMD, timed with events on the stream it runs on; best of 3 launches
    of about 20 ms each.  The shader clock comes from the loop's own cycle and
    wall-clock counters."""
    res = {}
    stream = torch.cuda.current_stream(dev)
    for wps in (1, 2):
        words, prods = pl.libra_mfma_loop_size(wps)
        rec = torch.zeros(words, dtype=torch.int64, device=dev)
        iters = 200000 // wps
        pl.libra_mfma_loop(wps, 1000, rec)                     # warm-up
        best = None
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            pl.libra_mfma_loop(wps, iters, rec)
            e1.record(stream)
            e1.synchronize()
            ms = e0.elapsed_time(e1)
            r = rec.view(-1, 3).cpu().numpy()
            ghz = float(r[:, 0].sum() / r[:, 1].sum() * 0.1)
            tf = 32768.0 * iters * prods / (ms * 1e-3) / 1e12
            if best is None or tf > best[0]:
                best = (tf, ghz, ms)
        res[wps] = best
    top = max(res, key=lambda x: res[x][0])
    return {"value": round(res[top][0], 1), "unit": "TFLOP/s", "waves_per_simd": top,
            "clock_ghz": round(res[top][1], 3),
            "one_wave_per_simd": {"value": round(res[1][0], 1), "clock_ghz": round(res[1][1], 3)},
            "frac_of_published": round(res[top][0] / PEAK_BF16_TFLOPS, 4),
            "kind": "independent v_mfma_f32_32x32x16_bf16 products, no other work"}


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_rows(w, n_rows: int) -> np.ndarray:
    """The fixed CPU-baseline row subset: 1/8 of the rows evenly spaced over
    the present rows of the longest sample (the straggler rows, each attending
    up to the whole sample), the rest evenly spaced over all other rows."""
    pos = w.q_positions()
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    j_long = int(np.argmax(w.lengths))
    in_long = (pos >= cu[j_long]) & (pos < cu[j_long + 1])
    longs, others = np.nonzero(in_long)[0], np.nonzero(~in_long)[0]
    n_long = min(len(longs), max(1, n_rows // 8))
    n_other = min(len(others), n_rows - n_long)
    pick = [longs[np.linspace(0, len(longs) - 1, n_long).round().astype(np.int64)]] if n_long else []
    if n_other:
        pick.append(others[np.linspace(0, len(others) - 1, n_other).round().astype(np.int64)])
    return np.unique(np.concatenate(pick))


def cpu_baseline(w, q, k, v, do, n_rows):
    """The oracle, as it stands, on a fixed subset of query rows of the same
    workload (all heads, forward + backward, one call each: the oracle groups
    the rows by sample itself)."""
    import torch
    from oracle import attention as oa
    pos = w.q_positions()
    rows = cpu_rows(w, n_rows)
    t0 = time.perf_counter()
    oa.attention_fwd(q, k, v, w.lengths, pos, rows=rows)
    oa.attention_bwd(q, k, v, do, w.lengths, pos, rows=rows)
    dt = time.perf_counter() - t0
    pairs = oa.useful_pairs(w.lengths, pos[rows])
    flops = 14.0 * w.d * w.h_q * pairs
    rate = flops / dt / 1e12
    full_pairs = oa.useful_pairs(w.lengths, pos)
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    j_long = int(np.argmax(w.lengths))
    n_long = int(((pos[rows] >= cu[j_long]) & (pos[rows] < cu[j_long + 1])).sum())
    return {"value": rate, "unit": "TFLOP/s",
            "cores": len(os.sched_getaffinity(0)),
            "blas_threads": torch.get_num_threads(),
            "cpu_model": _cpu_model(),
            "kind": "oracle",
            "sample": (f"fixed subset of {len(rows)} of {len(pos)} query rows x {w.h_q} heads "
                       f"({n_long} rows of the longest sample, {len(rows) - n_long} spread over "
                       f"the others), fwd+bwd in float64: {pairs} causal pairs per head in "
                       f"{dt:.1f} s"),
            "seconds": round(dt, 2),
            # the whole step's useful work at the sampled rate (extrapolated, not timed)
            "extrapolated_step_s": round(14.0 * w.d * w.h_q * full_pairs / 1e12 / rate, 1)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU; --gpus {args.gpus} is not supported (the "
              "multi-GPU tile exchange of the paper is not implemented)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.vrsp:
        vrsp_bench(args.cpu_seconds)
        return
    if args.straggler:
        straggler_bench()
        return
    if args.straggler_pool:
        if args.straggler_pool == "1M":
            straggler_pool_bench("1M", pool_packs=4, cp=16, gbs=32, B=8192, reps=1)
        else:
            straggler_pool_bench()
        return
    if args.simulate:
        simulate()
        return
    import torch
    import paper_2607_23250_amd as pl
    import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    w = wl.workload(args.workload)
    full_tiles, loads = plan(pl, w)
    share_tiles = plan(pl, w, w.q_ranges)[0] if w.q_ranges is not None else None
    sets = launch_sets(w, full_tiles, share_tiles)
    cost = sum(int(s["cost"].sum()) for s in sets)            # = h_q * causal pairs
    fwd_flops = 4.0 * w.d * cost
    bwd_flops = 10.0 * w.d * cost
    max_over_mean = float(w.V * loads.max() / loads.sum())

    # inputs resident in HBM
    q, k, v, do = wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)
    qd, kd, vd, dod = (t.to(dev) for t in (q, k, v, do))
    cu = np.zeros(len(w.lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(w.lengths)
    cud = torch.from_numpy(cu).to(dev)
    o = torch.empty_like(qd)
    lse = torch.empty((w.h_q, w.n_q_rows), dtype=torch.float32, device=dev)
    dq = torch.empty_like(qd)
    acc = len(sets) > 1
    kv_dtype = torch.float32 if acc else torch.bfloat16
    dk = torch.zeros(kd.shape, dtype=kv_dtype, device=dev)
    dv = torch.zeros(kd.shape, dtype=kv_dtype, device=dev)
    n = len(w.lengths)
    ws_bytes = max(max(pl.libra_attn_workspace_size(len(s), n, w.n_q_rows, w.n_kv_rows, w.h_q,
                                                    w.h_kv, w.d, b) for b in (False, True))
                   for s in sets)
    ws = pl.alloc_workspace(ws_bytes, dev)
    tile_bytes = [len(s) * pl.TILE_DTYPE.itemsize for s in sets]
    dev_tiles = [torch.empty(b, dtype=torch.uint8, device=dev) for b in tile_bytes]
    host_tiles = [[torch.empty(b, dtype=torch.uint8, pin_memory=True) for b in tile_bytes]
                  for _ in range(2)]
    copied = [None, None]
    stream = torch.cuda.current_stream(dev)
    plan_ms = []

    def make_plan(buf):
        """Plan on the host into pinned buffer `buf` (the tile sets of the step)."""
        if copied[buf] is not None:
            copied[buf].synchronize()
        t0 = time.perf_counter()
        ft, _ = plan(pl, w)
        st = plan(pl, w, w.q_ranges)[0] if w.q_ranges is not None else None
        plan_ms.append((time.perf_counter() - t0) * 1e3)
        for h, s in zip(host_tiles[buf], launch_sets(w, ft, st)):
            h.numpy()[:] = np.ascontiguousarray(s).view(np.uint8)

    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    # per launch set (virtual worker): events around its forward and its backward
    ev_w = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in sets]
    split_ms = []

    def step(i, record):
        buf = i % 2
        for d_t, h_t in zip(dev_tiles, host_tiles[buf]):
            d_t.copy_(h_t, non_blocking=True)
        copied[buf] = torch.cuda.Event()
        copied[buf].record(stream)
        if acc:
            dk.zero_()
            dv.zero_()
        if record:
            ev[0].record(stream)
        for j, td in enumerate(dev_tiles):
            if record:
                ev_w[j][0].record(stream)
            pl.libra_attn_fwd(qd, kd, vd, cud, td, o=o, lse=lse, workspace=ws)
            if record:
                ev_w[j][1].record(stream)
        if record:
            ev[1].record(stream)
        for j, td in enumerate(dev_tiles):
            if record:
                ev_w[j][2].record(stream)
            pl.libra_attn_bwd(qd, kd, vd, o, lse, dod, cud, td, dq=dq, dk=dk, dv=dv,
                              accumulate=acc, workspace=ws)
            if record:
                ev_w[j][3].record(stream)
        if record:
            ev[2].record(stream)
        make_plan((i + 1) % 2)          # host plans the next step while the GPU runs

    make_plan(0)
    for i in range(args.warmup):
        step(i, False)
    torch.cuda.synchronize()
    # one step with fwd / bwd split events (not part of the timed region)
    step(args.warmup, True)
    torch.cuda.synchronize()
    split_ms = (ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2]))
    # fwd + bwd time of each launch set: for a pool run per virtual worker,
    # the one-GPU stand-in for each worker's share of the step
    worker_ms = [e[0].elapsed_time(e[1]) + e[2].elapsed_time(e[3]) for e in ev_w]

    pl.libra_timing_enable(True)
    plan_ms.clear()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + 1 + i, False)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    fwd_main_ms, n_fwd = pl.libra_timing_read(0)
    kv_ms, n_kv = pl.libra_timing_read(1)
    dq_ms, n_dq = pl.libra_timing_read(2)
    pl.libra_timing_enable(False)

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = (fwd_flops + bwd_flops) / (ms_per_step * 1e-3) / 1e12
    # dominant kernel: the backward dK/dV kernel; its algorithmic work is the
    # S, dP, dV and dK contractions, 8*d flops per causal pair per query head
    kv_launch_ms = kv_ms / max(n_kv, 1)
    kv_launch_flops = 8.0 * w.d * cost / len(sets)
    achieved = kv_launch_flops / (kv_launch_ms * 1e-3) / 1e12
    dq_launch_ms = dq_ms / max(n_dq, 1)
    fwd_achieved = (fwd_flops / len(sets)) / (fwd_main_ms / max(n_fwd, 1) * 1e-3) / 1e12
    traffic = traffic_entry("attn_bwd_dkdv_kernel", w.name)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "pack_tokens": w.pack_tokens if w.P <= 2 else [w.pack_tokens[0]] * w.P,
            "query_rows": w.n_q_rows, "kv_rows": w.n_kv_rows, "samples": len(w.lengths),
            "max_sample": max(w.lengths), "h_q": w.h_q, "h_kv": w.h_kv, "head_dim": w.d,
            "block_tokens": w.B, "head_shards": w.H, "cp": w.CP, "virtual_workers": w.V,
            "launches_per_step": len(sets), "tiles_executed": int(sum(len(s) for s in sets)),
            "assumptions": w.notes,
        },
        "pct_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "max_over_mean_load": round(max_over_mean, 4),
        "useful_tflop_per_step": round((fwd_flops + bwd_flops) / 1e12, 3),
        "fwd_ms": round(split_ms[0], 3),
        "bwd_ms": round(split_ms[1], 3),
        "fwd_tflops": round(fwd_flops / (split_ms[0] * 1e-3) / 1e12, 1),
        "bwd_tflops": round(bwd_flops / (split_ms[1] * 1e-3) / 1e12, 1),
        "fwd_main_kernel_tflops": round(fwd_achieved, 1),
        "bwd_dkdv_kernel_ms": round(kv_launch_ms, 3),
        "bwd_dq_kernel_ms": round(dq_launch_ms, 3),
        "bwd_dq_kernel_useful_tflops": round(2.0 * w.d * cost / len(sets) / (dq_launch_ms * 1e-3)
                                             / 1e12, 1),
        "plan_ms": round(float(np.mean(plan_ms)), 3) if plan_ms else None,
        "launch_set_ms": [round(x, 3) for x in worker_ms],
        "launch_set_time_max_over_mean": round(max(worker_ms) / float(np.mean(worker_ms)), 4),
        "roofline": {
            "kernel": f"attn_bwd_dkdv_kernel<{w.d}>",
            "bound": "mfma",
            "achieved": round(achieved, 1),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "launch_ms": round(kv_launch_ms, 3),
            "flops_per_launch": kv_launch_flops,
        },
    }
    loop = mfma_loop_peak(pl, torch, dev)
    out["mfma_loop_peak"] = loop
    out["roofline"]["frac_of_mfma_loop_peak"] = round(achieved / loop["value"], 4)
    if args.cpu_rows > 0:
        out["cpu_baseline"] = cpu_baseline(w, q, k, v, do, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
