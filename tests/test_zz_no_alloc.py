"""libra_attn_fwd_noalloc (the forward without a workspace argument, for
callers that cannot allocate) against libra_attn_fwd, through the C ABI:
two calls in a row, the second with a smaller input, each bit-identical to
the workspace entry point (same kernels); oversized inputs are rejected."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2607_23250_amd as pl
import workloads as wl
from gpu_util import DEV, cu_dev, plan, say

pytestmark = pytest.mark.gpu


def _noalloc(q, k, v, cu, td, o, lse):
    n_q, h_q, d = q.shape
    n_kv, h_kv, _ = k.shape
    n = cu.numel() - 1
    T = td.numel() // pl.TILE_DTYPE.itemsize
    stream = ctypes.c_void_p(torch.cuda.current_stream(q.device).cuda_stream)
    return pl.lib().libra_attn_fwd_noalloc(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), cu.data_ptr(), n, td.data_ptr(), T, n_q, n_kv,
        h_q, h_kv, d, ctypes.c_float(0.0), o.data_ptr(), lse.data_ptr(), stream)


def _case(w):
    tiles, _ = plan(w)
    q, k, v, _ = (t.to(DEV) for t in wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv,
                                                  w.d))
    cu = cu_dev(w)
    td = pl.tiles_to_device(tiles, DEV)
    o_ref, lse_ref = pl.libra_attn_fwd(q, k, v, cu, td)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.h_q, w.n_q_rows), float("nan"), dtype=torch.float32, device=DEV)
    rc = _noalloc(q, k, v, cu, td, o, lse)
    assert rc == pl.LIBRA_OK, pl.lib().libra_last_error().decode()
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref)
    return len(tiles)


def test_noalloc_forward_matches_workspace_forward_twice():
    big = wl.workload(wl.W_32K, scale=2)          # 16384-token pack, 32 / 8 heads, d = 128
    small = wl.small_random(6)
    say(f"[no-alloc fwd] first {big.name}/2 rows={big.n_q_rows}, then {small.name} "
        f"rows={small.n_q_rows} heads=({small.h_q},{small.h_kv}) d={small.d}")
    t1 = _case(big)
    t2 = _case(small)
    assert t2 < t1


def test_noalloc_forward_rejects_sizes_beyond_its_scratch():
    w = wl.small_random(6)
    q, k, v, _ = (t.to(DEV) for t in wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv,
                                                  w.d))
    cu = cu_dev(w)
    # a tile count whose work-item list needs more than the built-in scratch
    T = pl.LIBRA_FWD_NOALLOC_MAX_WORKSPACE // 32
    assert pl.libra_attn_workspace_size(T, len(w.lengths), w.n_q_rows, w.n_kv_rows, w.h_q,
                                        w.h_kv, w.d, False) > pl.LIBRA_FWD_NOALLOC_MAX_WORKSPACE
    td = torch.zeros(T * pl.TILE_DTYPE.itemsize, dtype=torch.uint8, device=DEV)
    o = torch.empty_like(q)
    lse = torch.empty((w.h_q, w.n_q_rows), dtype=torch.float32, device=DEV)
    assert _noalloc(q, k, v, cu, td, o, lse) == pl.LIBRA_ENOSPC
