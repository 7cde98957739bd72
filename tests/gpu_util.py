"""Helpers shared by the GPU parity tests (not collected by pytest)."""
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


def check(name, got, ref, tol=O_TOL, bf16_out=False, ref_bf16=None):
    """max-abs and relative-L2 error against float64.

    * bf16 outputs: the max-abs bound is applied on top of the output's own
      rounding (half a bf16 ulp of the exact value), which no bf16 result
      can avoid;
    * ``ref_bf16`` (the same attention in plain bf16 PyTorch): the paper's
      fidelity criterion (Sec. 6.7) -- errors within twice that reference's
      -- relaxes each bound when the reference itself exceeds half of it.
    """
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    ma, rl = errors(got, ref)
    excess = ma
    if bf16_out and got.size:
        excess = float((np.abs(got - ref) - half_ulp_bf16(ref)).max())
    t_ma, t_rl = tol
    extra = ""
    if ref_bf16 is not None:
        b_ma, b_rl = errors(ref_bf16, ref)
        t_ma, t_rl = max(t_ma, 2 * b_ma), max(t_rl, 2 * b_rl)
        extra = f" [bf16 torch: max_abs={b_ma:.3e} rel_l2={b_rl:.3e}]"
    say(f"  {name}: max_abs={ma:.3e} (beyond bf16 rounding {excess:.3e}) rel_l2={rl:.3e}{extra}")
    assert np.isfinite(got).all(), f"{name}: non-finite"
    assert excess <= t_ma and rl <= t_rl, \
        f"{name}: max_abs {ma:.3e} (excess {excess:.3e}) rel_l2 {rl:.3e} over {(t_ma, t_rl)}"


def fwd(w, tiles, q, k, v, cu):
    td = pl.tiles_to_device(tiles, DEV)
    o, lse = pl.libra_attn_fwd(q, k, v, cu, td)
    return o, lse


def to_np(t):
    return t.detach().float().cpu().numpy()
