"""Python binding of ``liblibra.so`` (argument marshalling only).

Every entry point of ``include/libra.h`` is exposed under the same name.  The
planner works on NumPy arrays; the attention calls take torch tensors for
device memory and enqueue on torch's current HIP stream.  All computation
happens in the library: nothing here falls back to another implementation,
and a missing library raises immediately.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblibra.so")

LIBRA_OK = 0
LIBRA_EINVAL = -1
LIBRA_ENOSPC = -2
LIBRA_EUNSUPPORTED = -3
LIBRA_EOVERFLOW = -4
LIBRA_EHIP = -5
LIBRA_BWD_ACCUMULATE_DKV = 1

# libra_tile_t (56 bytes)
TILE_DTYPE = np.dtype([("q_begin", "<i8"), ("q_end", "<i8"), ("q_row", "<i8"), ("cost", "<i8"),
                       ("head_begin", "<i4"), ("head_end", "<i4"), ("pack", "<i4"),
                       ("home", "<i4"), ("worker", "<i4"), ("id", "<i4")])
assert TILE_DTYPE.itemsize == 56

EXPORTED = ("libra_strerror", "libra_last_error", "libra_plan", "libra_vrsp",
            "libra_attn_workspace_size", "libra_attn_fwd", "libra_attn_bwd",
            "libra_timing_enable", "libra_timing_read", "libra_mfma_loop_size",
            "libra_mfma_loop", "libra_attn_skipped_tiles", "libra_attn_fwd_noalloc")
LIBRA_WS_SKIPPED_OFFSET = 16
LIBRA_FWD_NOALLOC_MAX_WORKSPACE = 16 << 20


class LibraError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {code} ({detail})")
        self.code = code


class _PlanCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "block_tokens", "head_shards", "num_packs", "cp", "num_q_heads", "num_kv_heads",
        "head_dim", "elem_bytes", "tau_num", "tau_den")]


_lib = None


def lib() -> ctypes.CDLL:
    """Load ``liblibra.so`` (built in-tree by ``paper_2607_23250_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with "
                          "`python -m paper_2607_23250_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    L.libra_strerror.restype = ctypes.c_char_p
    L.libra_strerror.argtypes = [ctypes.c_int]
    L.libra_last_error.restype = ctypes.c_char_p
    L.libra_last_error.argtypes = []
    L.libra_plan.restype = ctypes.c_int
    L.libra_plan.argtypes = [ctypes.POINTER(_PlanCfg), P, I64, P, P, P, I32, P, I64, P, P, P]
    L.libra_vrsp.restype = ctypes.c_int
    L.libra_vrsp.argtypes = [P, I64, P, I64, I32, P, P, P]
    L.libra_attn_workspace_size.restype = SZ
    L.libra_attn_workspace_size.argtypes = [I64, I64, I64, I64, I32, I32, I32, I32]
    L.libra_attn_fwd.restype = ctypes.c_int
    L.libra_attn_fwd.argtypes = [P, P, P, P, I64, P, I64, I64, I64, I32, I32, I32,
                                 ctypes.c_float, P, P, P, SZ, P]
    L.libra_attn_bwd.restype = ctypes.c_int
    L.libra_attn_bwd.argtypes = [P, P, P, P, P, P, P, I64, P, I64, I64, I64, I32, I32, I32,
                                 ctypes.c_float, P, P, P, ctypes.c_uint32, P, SZ, P]
    L.libra_timing_enable.restype = ctypes.c_int
    L.libra_timing_enable.argtypes = [ctypes.c_int]
    L.libra_timing_read.restype = ctypes.c_int
    L.libra_timing_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int64)]
    L.libra_mfma_loop_size.restype = ctypes.c_int
    L.libra_mfma_loop_size.argtypes = [I32, ctypes.POINTER(ctypes.c_int64),
                                       ctypes.POINTER(ctypes.c_int64)]
    L.libra_mfma_loop.restype = ctypes.c_int
    L.libra_mfma_loop.argtypes = [I32, I32, P, I64, P]
    L.libra_attn_fwd_noalloc.restype = ctypes.c_int
    L.libra_attn_fwd_noalloc.argtypes = [P, P, P, P, I64, P, I64, I64, I64, I32, I32, I32,
                                         ctypes.c_float, P, P, P]
    L.libra_attn_skipped_tiles.restype = ctypes.c_int
    L.libra_attn_skipped_tiles.argtypes = [P, ctypes.POINTER(ctypes.c_int32), P]
    _lib = L
    return L


def _check(rc: int, where: str):
    if rc != LIBRA_OK:
        L = lib()
        raise LibraError(rc, where, f"{L.libra_strerror(rc).decode()}: "
                                    f"{L.libra_last_error().decode()}")


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _offsets(counts) -> np.ndarray:
    out = np.zeros(len(counts) + 1, dtype=np.int64)
    out[1:] = np.cumsum(np.asarray(counts, dtype=np.int64))
    return out


def libra_plan(lengths: Sequence[int], pack_tokens: Sequence[int], *, block_tokens: int,
               head_shards: int, cp: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
               elem_bytes: int = 2, tau: Tuple[int, int] = (3, 100),
               q_ranges: Optional[Sequence[Tuple[int, int]]] = None, with_bytes: bool = False
               ):
    """SH-Tiles with Eq. 6 costs and the Algorithm 2 placement.

    Returns ``(tiles, loads)``: a ``TILE_DTYPE`` array in tile-ID order and the
    int64 load of each of the ``len(pack_tokens) * cp`` workers; with
    ``with_bytes``, also the bytes each worker receives under the plan.
    """
    L = lib()
    lengths = np.ascontiguousarray(lengths, dtype=np.int64)
    cu = _offsets(lengths)
    pack_cu = _offsets(pack_tokens)
    cfg = _PlanCfg(block_tokens, head_shards, len(pack_tokens), cp, num_q_heads, num_kv_heads,
                   head_dim, elem_bytes, tau[0], tau[1])
    qr = None
    nqr = 0
    if q_ranges is not None:
        qr = np.ascontiguousarray(np.asarray(q_ranges, dtype=np.int64).reshape(-1))
        nqr = len(qr) // 2
    n_tiles = ctypes.c_int64(0)
    args = (ctypes.byref(cfg), _ptr(lengths), len(lengths), _ptr(cu), _ptr(pack_cu), _ptr(qr), nqr)
    _check(L.libra_plan(*args, None, 0, ctypes.byref(n_tiles), None, None), "libra_plan")
    tiles = np.zeros(n_tiles.value, dtype=TILE_DTYPE)
    loads = np.zeros(len(pack_tokens) * cp, dtype=np.int64)
    recv = np.zeros(len(pack_tokens) * cp, dtype=np.int64) if with_bytes else None
    _check(L.libra_plan(*args, _ptr(tiles), len(tiles), ctypes.byref(n_tiles), _ptr(loads),
                        _ptr(recv)), "libra_plan")
    return (tiles, loads, recv) if with_bytes else (tiles, loads)


def libra_vrsp(packs: Sequence[Sequence[int]], pool_size: int
               ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Algorithm 1 over one window of packed sequences (each a list of raw
    sample lengths).  Returns ``(order, pool_load, seq_work)``: original
    sequence indices in output order, the load of each of the
    ``len(packs) // pool_size`` pools and every sequence's workload F_i."""
    L = lib()
    counts = [len(p) for p in packs]
    lengths = np.ascontiguousarray(np.concatenate([np.asarray(p, dtype=np.int64) for p in packs])
                                   if packs else np.zeros(0, dtype=np.int64))
    seq_cu = _offsets(counts)
    D = len(packs)
    order = np.zeros(D, dtype=np.int64)
    loads = np.zeros(D // pool_size if pool_size > 0 else 0, dtype=np.int64)
    work = np.zeros(D, dtype=np.int64)
    _check(L.libra_vrsp(_ptr(lengths), len(lengths), _ptr(seq_cu), D, pool_size, _ptr(order),
                        _ptr(loads), _ptr(work)), "libra_vrsp")
    return order, loads, work


def libra_attn_workspace_size(num_tiles: int, num_samples: int, n_q_rows: int, n_kv_rows: int,
                              h_q: int, h_kv: int, head_dim: int, backward: bool) -> int:
    return int(lib().libra_attn_workspace_size(num_tiles, num_samples, n_q_rows, n_kv_rows, h_q,
                                               h_kv, head_dim, int(bool(backward))))


def libra_timing_enable(enable: bool = True) -> None:
    _check(lib().libra_timing_enable(int(bool(enable))), "libra_timing_enable")


def libra_timing_read(which: int) -> Tuple[float, int]:
    """(summed milliseconds, launches) of the forward kernel (0), the backward
    dK/dV kernel (1) or the backward dQ kernel (2)."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().libra_timing_read(which, ctypes.byref(ms), ctypes.byref(n)), "libra_timing_read")
    return ms.value, n.value


def libra_mfma_loop_size(waves_per_simd: int) -> Tuple[int, int]:
    """(uint64 words of the record, MFMA products per round over the launch)."""
    words = ctypes.c_int64(0)
    prods = ctypes.c_int64(0)
    _check(lib().libra_mfma_loop_size(waves_per_simd, ctypes.byref(words), ctypes.byref(prods)),
           "libra_mfma_loop_size")
    return words.value, prods.value


# ---------------------------------------------------------------------------
# torch-facing helpers (device memory and streams only)

def _torch():
    import torch
    return torch


def tiles_to_device(tiles: np.ndarray, device):
    """Device copy of a tile array (raw bytes in a uint8 tensor)."""
    torch = _torch()
    raw = np.ascontiguousarray(tiles).view(np.uint8)
    return torch.from_numpy(raw.copy()).to(device)


def _dptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t, dtype, shape, name):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() \
            or not t.is_cuda:
        raise ValueError(f"{name}: need a contiguous {dtype} device tensor of shape {shape}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def alloc_workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def libra_attn_fwd(q, k, v, cu_seqlens, tiles, *, softmax_scale: float = 0.0, o=None, lse=None,
                   workspace=None):
    """O (bf16) and LSE (fp32 [h_q][n_q]) for the rows / heads of ``tiles``.

    ``tiles`` is a device uint8 tensor from ``tiles_to_device``; ``cu_seqlens``
    a device int64 tensor of ``num_samples + 1`` offsets.
    """
    torch = _torch()
    n_q, h_q, d = q.shape
    n_kv, h_kv, _ = k.shape
    n = cu_seqlens.numel() - 1
    T = tiles.numel() // TILE_DTYPE.itemsize
    _need(q, torch.bfloat16, (n_q, h_q, d), "q")
    _need(k, torch.bfloat16, (n_kv, h_kv, d), "k")
    _need(v, torch.bfloat16, (n_kv, h_kv, d), "v")
    _need(cu_seqlens, torch.int64, (n + 1,), "cu_seqlens")
    if o is None:
        o = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((h_q, n_q), dtype=torch.float32, device=q.device)
    _need(o, torch.bfloat16, (n_q, h_q, d), "o")
    _need(lse, torch.float32, (h_q, n_q), "lse")
    need = libra_attn_workspace_size(T, n, n_q, n_kv, h_q, h_kv, d, False)
    if workspace is None:
        workspace = alloc_workspace(need, q.device)
    _check(lib().libra_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cu_seqlens.data_ptr(), n,
                                tiles.data_ptr(), T, n_q, n_kv, h_q, h_kv, d, softmax_scale,
                                o.data_ptr(), lse.data_ptr(), workspace.data_ptr(),
                                workspace.numel(), _stream(q.device)), "libra_attn_fwd")
    return o, lse


def libra_attn_skipped_tiles(workspace) -> int:
    """Tiles skipped as out of range by the last fwd / bwd call that used
    ``workspace`` (synchronizes the current stream)."""
    n = ctypes.c_int32(0)
    _check(lib().libra_attn_skipped_tiles(workspace.data_ptr(), ctypes.byref(n),
                                          _stream(workspace.device)), "libra_attn_skipped_tiles")
    return int(n.value)


def libra_mfma_loop(waves_per_simd: int, iters: int, record) -> None:
    """Enqueue the matrix-core reference loop on the current stream; ``record``
    is a device int64 tensor of at least ``libra_mfma_loop_size(...)[0]``
    words (per workgroup: shader cycles, 100 MHz ticks, unused)."""
    torch = _torch()
    if record.dtype != torch.int64 or not record.is_cuda or not record.is_contiguous():
        raise ValueError("record: need a contiguous int64 device tensor")
    _check(lib().libra_mfma_loop(waves_per_simd, iters, record.data_ptr(), record.numel(),
                                 _stream(record.device)), "libra_mfma_loop")


def libra_attn_bwd(q, k, v, o, lse, dout, cu_seqlens, tiles, *, softmax_scale: float = 0.0,
                   dq=None, dk=None, dv=None, accumulate: bool = False, workspace=None):
    """dQ (bf16), dK / dV (bf16, or fp32 summed into when ``accumulate``)."""
    torch = _torch()
    n_q, h_q, d = q.shape
    n_kv, h_kv, _ = k.shape
    n = cu_seqlens.numel() - 1
    T = tiles.numel() // TILE_DTYPE.itemsize
    for t, name in ((q, "q"), (o, "o"), (dout, "dout")):
        _need(t, torch.bfloat16, (n_q, h_q, d), name)
    for t, name in ((k, "k"), (v, "v")):
        _need(t, torch.bfloat16, (n_kv, h_kv, d), name)
    _need(lse, torch.float32, (h_q, n_q), "lse")
    _need(cu_seqlens, torch.int64, (n + 1,), "cu_seqlens")
    kv_dtype = torch.float32 if accumulate else torch.bfloat16
    if dq is None:
        dq = torch.empty_like(q)
    if dk is None:
        dk = (torch.zeros if accumulate else torch.empty)((n_kv, h_kv, d), dtype=kv_dtype,
                                                          device=q.device)
    if dv is None:
        dv = (torch.zeros if accumulate else torch.empty)((n_kv, h_kv, d), dtype=kv_dtype,
                                                          device=q.device)
    _need(dq, torch.bfloat16, (n_q, h_q, d), "dq")
    _need(dk, kv_dtype, (n_kv, h_kv, d), "dk")
    _need(dv, kv_dtype, (n_kv, h_kv, d), "dv")
    need = libra_attn_workspace_size(T, n, n_q, n_kv, h_q, h_kv, d, True)
    if workspace is None:
        workspace = alloc_workspace(need, q.device)
    _check(lib().libra_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                lse.data_ptr(), dout.data_ptr(), cu_seqlens.data_ptr(), n,
                                tiles.data_ptr(), T, n_q, n_kv, h_q, h_kv, d, softmax_scale,
                                dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                LIBRA_BWD_ACCUMULATE_DKV if accumulate else 0,
                                workspace.data_ptr(), workspace.numel(), _stream(q.device)),
           "libra_attn_bwd")
    return dq, dk, dv
