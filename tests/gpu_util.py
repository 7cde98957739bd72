"""Helpers shared by the GPU parity tests (not collected by pytest)."""
import json
import os
import sys

import numpy as np
import torch

import paper_2607_23250_amd as pl

DEV = "cuda:0"
O_TOL = (2e-2, 1e-2)      # max-abs, relative L2 against float64
LSE_TOL = 1e-3


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def plan(w, q_ranges=None):
    tiles, loads = pl.libra_plan(w.lengths, w.pack_tokens, block_tokens=w.B, head_shards=w.H,
                                 cp=w.CP, num_q_heads=w.h_q, num_kv_heads=w.h_kv, head_dim=w.d,
                                 q_ranges=q_ranges)
    return tiles, loads


def cu_dev(w):
    cu = np.zeros(len(w.lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(w.lengths)
    return torch.from_numpy(cu).to(DEV)


def errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = got - ref
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    denom = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(diff)) / denom if denom > 0 else float(np.linalg.norm(diff))
    return max_abs, rel


def half_ulp_bf16(ref):
    """Half a bf16 ulp at |ref|: the error of storing the exact value in bf16."""
    a = np.abs(np.asarray(ref, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return np.where(a > 0, 2.0 ** (e - 8), 0.0)


def _log(record):
    """Append one parity record (JSON) to the file named by LIBRA_PARITY_LOG, if set."""
    path = os.environ.get("LIBRA_PARITY_LOG")
    if not path:
        return
    record["test"] = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    with open(path, "a") as f:
        f.write(json.dumps(record) + "\n")


def check(name, got, ref, tol=O_TOL, bf16_out=False):
    """max-abs and relative-L2 error against float64, at the fixed bounds
    (max-abs <= 2e-2, relative L2 <= 1e-2 for O, dQ, dK, dV).

    bf16 outputs: the max-abs bound applies to the error beyond the output's
    own rounding (half a bf16 ulp of the exact value), which no bf16 result
    can avoid.  fp32 outputs (accumulate-mode dK / dV) get no allowance.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ma, rl = errors(got, ref)
    excess = ma
    if bf16_out and got.size:
        excess = float((np.abs(got - ref) - half_ulp_bf16(ref)).max())
    t_ma, t_rl = tol
    finite = bool(np.isfinite(got).all())
    ok = finite and excess <= t_ma and rl <= t_rl
    ref_max = float(np.abs(ref).max()) if ref.size else 0.0
    _log(dict(name=name, elements=int(got.size), bf16_out=bool(bf16_out), max_abs=ma,
              excess=excess, rel_l2=rl, ref_max_abs=ref_max, bound=[t_ma, t_rl], ok=ok))
    say(f"  {name}: max_abs={ma:.3e} (beyond bf16 rounding {excess:.3e}) rel_l2={rl:.3e} "
        f"|ref|max={ref_max:.3e}")
    assert finite, f"{name}: non-finite"
    assert excess <= t_ma and rl <= t_rl, \
        f"{name}: max_abs {ma:.3e} (excess {excess:.3e}) rel_l2 {rl:.3e} over {(t_ma, t_rl)}"


def fwd(w, tiles, q, k, v, cu):
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(q, k, v, cu, td)
    return o, lse


def to_np(t):
    return t.detach().float().cpu().numpy()
