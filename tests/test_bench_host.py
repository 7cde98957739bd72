"""Host-side logic of bench.py (no GPU): the command-line contract for more
than one GPU, the fixed CPU-baseline row subset, the launch sets of the
per-worker pool and of a CP share, and the rule that ties the reported HBM
traffic to the kernel sources it was measured on."""
import hashlib
import json
import os
import subprocess
import sys

import numpy as np

import bench
import paper_2607_23250_amd as pl
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_cpu_rows_fixed_subset():
    w = wl.workload(wl.W_1M)
    rows = bench.cpu_rows(w, 64)
    assert len(rows) == 64 and np.all(np.diff(rows) > 0)
    assert np.array_equal(rows, bench.cpu_rows(w, 64)), "subset must be deterministic"
    pos = w.q_positions()
    cu = np.concatenate([[0], np.cumsum(w.lengths)])
    j = int(np.argmax(w.lengths))
    in_long = (pos[rows] >= cu[j]) & (pos[rows] < cu[j + 1])
    # 1/8 of the rows from the longest sample, the rest from the other samples
    assert in_long.sum() == 8
    assert (~in_long).sum() == 56
    # the subset spans both ends of the present rows
    assert rows[0] == 0 or in_long[0]
    assert rows[-1] >= len(pos) - len(pos) // 56


def test_launch_sets():
    w = wl.workload(wl.W_POOL)
    tiles, _ = bench.plan(pl, w)
    sets = bench.launch_sets(w, tiles, None)
    workers = sorted({int(s["worker"][0]) for s in sets})
    assert len(sets) == len(workers) == len(set(tiles["worker"].tolist()))
    assert sum(len(s) for s in sets) == len(tiles)
    for s in sets:
        assert len(set(s["worker"].tolist())) == 1
    w = wl.workload(wl.W_1M)
    full, _ = bench.plan(pl, w)
    share, _ = bench.plan(pl, w, q_ranges=w.q_ranges)
    sets = bench.launch_sets(w, full, share)
    assert len(sets) == 1 and sets[0] is share


def _sha(srcs):
    h = hashlib.sha256()
    for name in srcs:
        h.update(open(os.path.join(ROOT, "paper_2607_23250_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def test_traffic_entry_follows_the_sources(tmp_path, monkeypatch):
    name = "attn_bwd_dkdv_kernel__1M-cp16-share-qwen3-30b-a3b__traffic.json"
    rec = json.load(open(os.path.join(ROOT, "profiles", name)))
    got = bench.traffic_entry("attn_bwd_dkdv_kernel", "1M-cp16-share-qwen3-30b-a3b")
    # reported exactly when the record was taken on the current sources
    if _sha(rec["source"]) == rec["source_sha256"]:
        assert got == rec["bytes_per_launch"]
    else:
        assert got is None
    assert bench.traffic_entry("attn_bwd_dkdv_kernel", "no-such-workload") is None
    # a record whose hash does not match the sources is ignored
    prof = tmp_path / "profiles"
    prof.mkdir()
    stale = dict(rec, source_sha256="0" * 64)
    (prof / name).write_text(json.dumps(stale))
    csrc = tmp_path / "paper_2607_23250_amd" / "csrc"
    csrc.mkdir(parents=True)
    for src in rec["source"]:
        (csrc / src).write_bytes(open(os.path.join(ROOT, "paper_2607_23250_amd", "csrc", src),
                                      "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_entry("attn_bwd_dkdv_kernel", "1M-cp16-share-qwen3-30b-a3b") is None
    (prof / name).write_text(json.dumps(dict(rec, source_sha256=_sha(rec["source"]))))
    assert bench.traffic_entry("attn_bwd_dkdv_kernel",
                               "1M-cp16-share-qwen3-30b-a3b") == rec["bytes_per_launch"]
