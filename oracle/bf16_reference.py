"""bf16 PyTorch reference of the paper's fidelity criterion (test infrastructure).

Sec. 6.7 of the paper accepts forward and gradient errors (against a
high-precision reference) up to twice those of the same attention computed
with plain bf16 PyTorch operations.  This module is that bf16 computation:
per sample and per KV group, scores, softmax, output and autograd gradients
in torch bfloat16 on the CPU.  It is used only to derive the error allowance
of that criterion; the float64 oracle stays the reference the errors are
measured against.
"""
from __future__ import annotations

import math
from typing import Sequence

import numpy as np
import torch


def attention_bf16(q, k, v, dout, lengths: Sequence[int], q_pos=None):
    """(O, dQ, dK, dV) as float64 NumPy arrays, computed in bf16.

    ``q_pos[r]`` is the pool position of Q row r (default: row r is position
    r).  Only present rows contribute to dK / dV.
    """
    n_q, h_q, d = q.shape
    n_k, h_kv, _ = k.shape
    G = h_q // h_kv
    pos = np.arange(n_q) if q_pos is None else np.asarray(q_pos, dtype=np.int64)
    cu = np.concatenate([[0], np.cumsum(np.asarray(lengths, dtype=np.int64))])
    j_of = np.searchsorted(cu, pos, side="right") - 1
    O = np.zeros((n_q, h_q, d))
    dQ = np.zeros((n_q, h_q, d))
    dK = np.zeros((n_k, h_kv, d))
    dV = np.zeros((n_k, h_kv, d))
    for j in np.unique(j_of):
        rows = np.nonzero(j_of == j)[0]
        s = int(cu[j])
        loc = torch.as_tensor(pos[rows] - s)
        n_keys = int(loc.max()) + 1
        mask = torch.arange(n_keys)[None, :] <= loc[:, None]
        for g in range(h_kv):
            hs = slice(g * G, (g + 1) * G)
            qt = q[rows][:, hs].to(torch.bfloat16).transpose(0, 1).contiguous().requires_grad_(True)
            kt = k[s:s + n_keys, g].to(torch.bfloat16).contiguous().requires_grad_(True)
            vt = v[s:s + n_keys, g].to(torch.bfloat16).contiguous().requires_grad_(True)
            sc = (qt @ kt.t().contiguous()) * (1.0 / math.sqrt(d))       # [G, rows, keys]
            sc = sc.masked_fill(~mask, float("-inf"))
            o = torch.softmax(sc, dim=-1) @ vt
            o.backward(dout[rows][:, hs].to(torch.bfloat16).transpose(0, 1))
            O[rows, hs] = o.detach().transpose(0, 1).double().numpy()
            dQ[rows, hs] = qt.grad.transpose(0, 1).double().numpy()
            dK[s:s + n_keys, g] += kt.grad.double().numpy()
            dV[s:s + n_keys, g] += vt.grad.double().numpy()
    return O, dQ, dK, dV
