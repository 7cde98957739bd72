"""Closed forms of the attention outputs when every key is zero (K = 0).

Then every score is 0, so a row at sample-local position t weighs the t + 1
keys of its sample up to itself equally: P = 1 / (t + 1) (Eq. 1 with a
constant score).  From the textbook gradients:

* O_q     = mean of V_i over i <= q (same sample);  LSE_q = ln(t + 1);
* dQ      = 0 (dQ = scale * dS K and K = 0);
* dV_i    = sum over rows q >= i of the sample of sum_h dO_qh / (t_q + 1);
* dK_i    = scale * sum_{q >= i} sum_h (dO_qh . V_i - D_qh) Q_qh / (t_q + 1),
  with D_qh = dO_qh . O_q.

Suffix sums over the present rows make these O(rows * d^2 + keys * d^2) per
KV head: dK_i = scale * (A(i) V_i - c(i)) where A(i) sums the d x d matrices
Q_qh dO_qh^T / (t_q + 1) and c(i) the vectors D_qh Q_qh / (t_q + 1) over the
present rows q >= i of i's sample.  Everything is float64 NumPy.  These are
mathematical identities, independent of the oracle and of the library; a CPU
test checks them against the oracle on small inputs.
"""
from __future__ import annotations

import numpy as np


def _layout(lengths, pos):
    cu = np.concatenate([[0], np.cumsum(np.asarray(lengths, dtype=np.int64))])
    pos = np.asarray(pos, dtype=np.int64)
    j_of = np.searchsorted(cu, pos, side="right") - 1
    return cu, pos, j_of, pos - cu[j_of]


def prefix_mean_v(v64, lengths, pos):
    """O for one KV head's V (float64 [n_kv, d]): [rows, d]."""
    cu, pos, j_of, qloc = _layout(lengths, pos)
    csum = np.cumsum(v64, axis=0)
    start = cu[j_of]
    before = np.where(start[:, None] > 0, csum[np.maximum(start - 1, 0)], 0.0)
    return (csum[pos] - before) / (qloc + 1.0)[:, None]


def zero_k_dv(do64, lengths, pos, n_kv):
    """dV of one KV head from its query heads' dO (float64 [rows, G, d]): [n_kv, d]."""
    cu, pos, j_of, qloc = _layout(lengths, pos)
    wq = do64.sum(axis=1) / (qloc + 1.0)[:, None]
    acc = np.zeros((n_kv, do64.shape[2]))
    np.add.at(acc, pos, wq)
    out = np.zeros_like(acc)
    for j in np.unique(j_of):
        s, e = int(cu[j]), int(cu[j + 1])
        out[s:e] = np.cumsum(acc[s:e][::-1], axis=0)[::-1]
    return out


def zero_k_dk(q64, do64, v64, lengths, pos, n_kv, scale, chunk=128):
    """dK of one KV head: q64 / do64 float64 [rows, G, d] (its query heads),
    v64 float64 [n_kv, d]; rows in position order.  Returns [n_kv, d].

    Per sample, the present rows are taken in chunks from the last one back;
    A (d x d) and c (d) carry the sums over all later chunks.  Keys at or
    before a chunk's first row see every row of the chunk and of the later
    chunks; keys inside the chunk's span see the later chunks fully and the
    chunk's own rows q >= key (an explicit mask)."""
    cu, pos, j_of, qloc = _layout(lengths, pos)
    assert np.all(np.diff(pos) > 0), "rows must be in position order"
    G, d = q64.shape[1], v64.shape[1]
    w = 1.0 / (qloc + 1.0)
    o = prefix_mean_v(v64, lengths, pos)
    D = (do64 * o[:, None, :]).sum(axis=2)                    # D_qh = dO_qh . O_q
    out = np.zeros((n_kv, d))
    js = np.unique(j_of)
    r_start = np.searchsorted(j_of, js, side="left")
    r_end = np.searchsorted(j_of, js, side="right")
    for j, ra0, rb0 in zip(js, r_start, r_end):
        s = int(cu[j])
        A = np.zeros((d, d))
        c = np.zeros(d)
        for rb in range(int(rb0), int(ra0), -chunk):
            ra = max(int(ra0), rb - chunk)
            P = pos[ra:rb]
            Qf = q64[ra:rb].reshape(-1, d)                    # (rows x heads, d)
            dOf = do64[ra:rb].reshape(-1, d)
            wf = np.repeat(w[ra:rb], G)
            Df = D[ra:rb].reshape(-1)
            Pf = np.repeat(P, G)
            Qw = Qf * wf[:, None]
            A_new = A + Qw.T @ dOf
            c_new = c + (Qw * Df[:, None]).sum(axis=0)
            lo_full = s if ra == ra0 else int(pos[ra - 1]) + 1
            if lo_full <= P[0]:
                ks = slice(lo_full, int(P[0]) + 1)
                out[ks] = v64[ks] @ A_new.T - c_new
            for k0 in range(int(P[0]) + 1, int(P[-1]) + 1, chunk):
                k1 = min(int(P[-1]) + 1, k0 + chunk)
                Vk = v64[k0:k1]
                M = (dOf @ Vk.T - Df[:, None]) * wf[:, None]  # (rows x heads, keys)
                M *= Pf[:, None] >= np.arange(k0, k1)[None, :]
                out[k0:k1] = M.T @ Qf + Vk @ A.T - c
            A, c = A_new, c_new
    return out * scale
