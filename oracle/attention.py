"""Attention oracle (test infrastructure): packed causal attention in float64.

What is computed (Sec. 2.2, Eq. 1, under the block-diagonal causal mask of
fixed-token packing, Sec. 2.3): for every present query row of sample j and
every query head, softmax(q K_j^T / sqrt(d_h)) V_j over the keys of the same
sample at sample-local positions 0..q_loc (keys of other samples and later
keys are masked).  The backward pass is the textbook gradient of the same
expression; the paper's backward reuses the forward assignment (Sec. 4.3.3),
so it computes exactly these gradients.

Readings (listed in the design notes): grouped-query heads map contiguously,
kv_head = q_head // (h_q / h_kv); the log-sum-exp is natural-log,
LSE = m + ln(sum exp(s - m)) of the *scaled* scores, one fp32 value per
(q_head, row) in a [h_q][rows] array; the default scale is 1/sqrt(d).

Every sample and head is handled on its own with plain float64 arithmetic
(torch CPU tensor ops, which use every host core; rows are processed in
chunks only to bound memory, each row sees its whole causal key range at
once).  Inputs may be torch tensors (bf16 values are upcast exactly) or NumPy
arrays; results are NumPy float64 arrays.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence

import numpy as np
import torch

_MAX_ENTRIES = 1 << 25      # scores held at once per chunk (256 MiB in fp64)


def _f64(x) -> torch.Tensor:
    """Exact float64 CPU copy of a (bf16/fp32) torch tensor or array slice."""
    if isinstance(x, torch.Tensor):
        return x.detach().to("cpu", torch.float64)
    return torch.as_tensor(np.asarray(x, dtype=np.float64))


def _offsets(lengths: Sequence[int]) -> np.ndarray:
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    return cu


def _chunks(n_keys: int, rows: np.ndarray) -> Iterable[np.ndarray]:
    step = max(1, _MAX_ENTRIES // max(1, n_keys))
    for i in range(0, len(rows), step):
        yield rows[i:i + step]


class _Plan:
    """Which present rows fall in which sample (query rows sorted per sample),
    and where each requested row goes in the output (``out[row]``)."""

    def __init__(self, lengths, q_pos, rows):
        self.cu = _offsets(lengths)
        q_pos = np.asarray(q_pos, dtype=np.int64)
        rows = np.arange(len(q_pos)) if rows is None else np.asarray(rows, dtype=np.int64)
        self.n_out = len(rows)
        self.out = np.full(len(q_pos), -1, dtype=np.int64)
        self.out[rows] = np.arange(len(rows))
        pos = q_pos[rows]
        j_of = np.searchsorted(self.cu, pos, side="right") - 1
        self.groups = []
        for j in np.unique(j_of):
            sel = rows[j_of == j]
            loc = q_pos[sel] - self.cu[j]
            order = np.argsort(loc, kind="stable")
            self.groups.append((int(j), sel[order], loc[order]))


def attention_fwd(q, k, v, lengths: Sequence[int], q_pos, scale: Optional[float] = None,
                  rows=None, heads=None):
    """Forward oracle.

    ``q`` [N_q, h_q, d], ``k``/``v`` [N_k, h_kv, d]; ``q_pos[r]`` is the pool
    position of Q row r.  Returns ``(O, LSE)`` in float64: O [R, h_q, d] and
    LSE [h_q, R] for the R requested ``rows`` in the order given (every row
    when ``rows`` is None); entries of heads not requested are NaN.
    """
    n_q, h_q, d = q.shape
    h_kv = k.shape[1]
    G = h_q // h_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    heads = range(h_q) if heads is None else heads
    pl = _Plan(lengths, q_pos, rows)
    O = np.full((pl.n_out, h_q, d), np.nan)
    LSE = np.full((h_q, pl.n_out), np.nan)
    for j, sel, loc in pl.groups:
        s = int(pl.cu[j])
        n_need = int(loc[-1]) + 1
        for g in sorted({hq // G for hq in heads}):
            Kg = _f64(k[s:s + n_need, g, :])
            Vg = _f64(v[s:s + n_need, g, :])
            for hq in [h for h in heads if h // G == g]:
                for c in _chunks(n_need, np.arange(len(sel))):
                    rc, lc = sel[c], loc[c]
                    n_keys = int(lc.max()) + 1
                    Kj, Vj = Kg[:n_keys], Vg[:n_keys]
                    Qc = _f64(q[rc, hq, :])
                    S = (Qc @ Kj.T) * scale
                    S.masked_fill_(torch.arange(n_keys)[None, :] > torch.as_tensor(lc)[:, None],
                                   -math.inf)
                    m = S.max(dim=1).values
                    E = torch.exp(S - m[:, None])
                    l = E.sum(dim=1)
                    oc = pl.out[rc]
                    O[oc, hq, :] = ((E @ Vj) / l[:, None]).numpy()
                    LSE[hq, oc] = (m + torch.log(l)).numpy()
    return O, LSE


def attention_bwd(q, k, v, dout, lengths: Sequence[int], q_pos,
                  scale: Optional[float] = None, rows=None, kv_heads=None, dkdv: bool = True):
    """Backward oracle: gradients of sum(dO * O) with respect to Q, K, V.

    Only the requested ``rows`` contribute (for a ``dout`` that is zero on
    every other row this is the full gradient).  ``kv_heads`` restricts the
    computation to the query heads of those KV heads.  Returns
    ``(dQ, dK, dV)`` in float64: dQ [R, h_q, d] for the R requested rows in
    the order given (every row when ``rows`` is None; NaN for heads not
    computed), dK / dV [N_k, h_kv, d] (views of per-KV-head arrays).  With
    ``dkdv=False`` the dK / dV sums are skipped (they stay zero); dQ is the
    same.
    """
    n_q, h_q, d = q.shape
    n_k, h_kv, _ = k.shape
    G = h_q // h_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    kv_heads = range(h_kv) if kv_heads is None else kv_heads
    pl = _Plan(lengths, q_pos, rows)
    dQ = np.full((pl.n_out, h_q, d), np.nan)
    dK = np.zeros((h_kv, n_k, d))
    dV = np.zeros((h_kv, n_k, d))
    for j, sel, loc in pl.groups:
        s = int(pl.cu[j])
        n_need = int(loc[-1]) + 1
        for g in kv_heads:
            Kg = _f64(k[s:s + n_need, g, :])
            Vg = _f64(v[s:s + n_need, g, :])
            for hq in range(g * G, (g + 1) * G):
                for c in _chunks(n_need, np.arange(len(sel))):
                    rc, lc = sel[c], loc[c]
                    n_keys = int(lc.max()) + 1
                    Kj, Vj = Kg[:n_keys], Vg[:n_keys]
                    Qc = _f64(q[rc, hq, :])
                    dOc = _f64(dout[rc, hq, :])
                    S = (Qc @ Kj.T) * scale
                    S.masked_fill_(torch.arange(n_keys)[None, :] > torch.as_tensor(lc)[:, None],
                                   -math.inf)
                    m = S.max(dim=1).values
                    lse = m + torch.log(torch.exp(S - m[:, None]).sum(dim=1))
                    Pm = torch.exp(S - lse[:, None])            # softmax rows
                    Oc = Pm @ Vj
                    D = (dOc * Oc).sum(dim=1)
                    if dkdv:
                        dV[g, s:s + n_keys, :] += (Pm.T @ dOc).numpy()
                    dP = dOc @ Vj.T
                    dS = Pm * (dP - D[:, None])
                    dQ[pl.out[rc], hq, :] = ((dS @ Kj) * scale).numpy()
                    if dkdv:
                        dK[g, s:s + n_keys, :] += ((dS.T @ Qc) * scale).numpy()
    return dQ, np.moveaxis(dK, 0, 1), np.moveaxis(dV, 0, 1)


def useful_pairs(lengths: Sequence[int], q_pos) -> int:
    """Causal same-sample (query, key) pairs of the present query rows."""
    cu = _offsets(lengths)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    j = np.searchsorted(cu, q_pos, side="right") - 1
    return int((q_pos - cu[j] + 1).sum())
