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

Every sample and head is handled on its own with plain NumPy float64 arrays
(rows are processed in chunks only to bound memory; each row sees its whole
causal key range at once).  Inputs may be torch tensors (bf16 values are
upcast exactly) or NumPy arrays.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional, Sequence

import numpy as np

_MAX_ENTRIES = 1 << 25      # scores held at once per chunk (256 MiB in fp64)


def _f64(x) -> np.ndarray:
    """Exact float64 copy of a (bf16/fp32) torch tensor or array slice."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.float64).numpy()
    except ImportError:                                     # pragma: no cover
        pass
    return np.asarray(x, dtype=np.float64)


def _offsets(lengths: Sequence[int]) -> np.ndarray:
    cu = np.zeros(len(lengths) + 1, dtype=np.int64)
    cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    return cu


def _chunks(n_keys: int, rows: np.ndarray) -> Iterable[np.ndarray]:
    step = max(1, _MAX_ENTRIES // max(1, n_keys))
    for i in range(0, len(rows), step):
        yield rows[i:i + step]


class _Plan:
    """Which present rows fall in which sample (query rows sorted per sample)."""

    def __init__(self, lengths, q_pos, rows):
        self.cu = _offsets(lengths)
        q_pos = np.asarray(q_pos, dtype=np.int64)
        rows = np.arange(len(q_pos)) if rows is None else np.asarray(rows, dtype=np.int64)
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
    position of Q row r.  Returns ``(O, LSE)``: O float64 [N_q, h_q, d] and LSE
    float64 [h_q, N_q]; entries of rows / heads not requested are NaN.
    """
    n_q, h_q, d = q.shape
    h_kv = k.shape[1]
    G = h_q // h_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    heads = range(h_q) if heads is None else heads
    O = np.full((n_q, h_q, d), np.nan)
    LSE = np.full((h_q, n_q), np.nan)
    pl = _Plan(lengths, q_pos, rows)
    for j, sel, loc in pl.groups:
        s = int(pl.cu[j])
        for hq in heads:
            g = hq // G
            for c in _chunks(int(loc[-1]) + 1, np.arange(len(sel))):
                rc, lc = sel[c], loc[c]
                n_keys = int(lc.max()) + 1
                Kj = _f64(k[s:s + n_keys, g, :])
                Vj = _f64(v[s:s + n_keys, g, :])
                Qc = _f64(q[rc, hq, :])
                S = (Qc @ Kj.T) * scale
                S[np.arange(n_keys)[None, :] > lc[:, None]] = -np.inf
                m = S.max(axis=1)
                E = np.exp(S - m[:, None])
                l = E.sum(axis=1)
                O[rc, hq, :] = (E @ Vj) / l[:, None]
                LSE[hq, rc] = m + np.log(l)
    return O, LSE


def attention_bwd(q, k, v, dout, lengths: Sequence[int], q_pos,
                  scale: Optional[float] = None, rows=None, kv_heads=None):
    """Backward oracle: gradients of sum(dO * O) with respect to Q, K, V.

    Only the requested ``rows`` contribute (for a ``dout`` that is zero on
    every other row this is the full gradient).  ``kv_heads`` restricts the
    computation to the query heads of those KV heads.  Returns
    ``(dQ, dK, dV)`` in float64: dQ [N_q, h_q, d] (NaN where not computed),
    dK / dV [N_k, h_kv, d].
    """
    n_q, h_q, d = q.shape
    n_k, h_kv, _ = k.shape
    G = h_q // h_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    kv_heads = range(h_kv) if kv_heads is None else kv_heads
    dQ = np.full((n_q, h_q, d), np.nan)
    dK = np.zeros((n_k, h_kv, d))
    dV = np.zeros((n_k, h_kv, d))
    pl = _Plan(lengths, q_pos, rows)
    for j, sel, loc in pl.groups:
        s = int(pl.cu[j])
        for g in kv_heads:
            for hq in range(g * G, (g + 1) * G):
                for c in _chunks(int(loc[-1]) + 1, np.arange(len(sel))):
                    rc, lc = sel[c], loc[c]
                    n_keys = int(lc.max()) + 1
                    Kj = _f64(k[s:s + n_keys, g, :])
                    Vj = _f64(v[s:s + n_keys, g, :])
                    Qc = _f64(q[rc, hq, :])
                    dOc = _f64(dout[rc, hq, :])
                    S = (Qc @ Kj.T) * scale
                    S[np.arange(n_keys)[None, :] > lc[:, None]] = -np.inf
                    m = S.max(axis=1)
                    lse = m + np.log(np.exp(S - m[:, None]).sum(axis=1))
                    Pm = np.exp(S - lse[:, None])               # softmax rows
                    Oc = Pm @ Vj
                    D = (dOc * Oc).sum(axis=1)
                    dV[s:s + n_keys, g, :] += Pm.T @ dOc
                    dP = dOc @ Vj.T
                    dS = Pm * (dP - D[:, None])
                    dQ[rc, hq, :] = (dS @ Kj) * scale
                    dK[s:s + n_keys, g, :] += (dS.T @ Qc) * scale
    return dQ, dK, dV


def useful_pairs(lengths: Sequence[int], q_pos) -> int:
    """Causal same-sample (query, key) pairs of the present query rows."""
    cu = _offsets(lengths)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    j = np.searchsorted(cu, q_pos, side="right") - 1
    return int((q_pos - cu[j] + 1).sum())
