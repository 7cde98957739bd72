"""Pins of the attention oracle against independent formulations.

* the explicit whole-pack softmax under a block-diagonal causal mask (Sec. 2.3);
* PyTorch's float64 scaled_dot_product_attention with a boolean mask, and its
  autograd gradients;
* central finite differences of <dO, O>;
* closed forms: K = 0 gives the prefix mean of V and LSE = ln(q_loc + 1);
  a length-1 sample returns its own V row; dQ = 0 when K = 0;
* exact identities: per sample and KV head, sum_i dK_i = 0 and
  sum_i dV_i = sum over the group's query heads of sum_q dO_q.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import plan as op
import workloads as wl


def _inputs(w, seed, zero_k=False):
    q, k, v, do = wl.tensors(seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d, zero_k=zero_k)
    return q, k, v, do


def _sample_ids(lengths):
    return np.repeat(np.arange(len(lengths)), lengths)


def _dense_pack(q, k, v, lengths, scale):
    """Whole-pool softmax with the block-diagonal causal mask written out as an L x L matrix."""
    qf, kf, vf = (x.double().numpy() for x in (q, k, v))
    n, h_q, d = qf.shape
    G = h_q // kf.shape[1]
    sid = _sample_ids(lengths)
    pos = np.arange(n)
    allowed = (sid[:, None] == sid[None, :]) & (pos[None, :] <= pos[:, None])
    O = np.zeros_like(qf)
    LSE = np.zeros((h_q, n))
    for h in range(h_q):
        S = qf[:, h, :] @ kf[:, h // G, :].T * scale
        S = np.where(allowed, S, -np.inf)
        m = S.max(1)
        E = np.exp(S - m[:, None])
        O[:, h, :] = E @ vf[:, h // G, :] / E.sum(1)[:, None]
        LSE[h] = m + np.log(E.sum(1))
    return O, LSE


@pytest.mark.parametrize("seed", range(12))
def test_fwd_equals_dense_pack_softmax(seed):
    w = wl.tiny_random(seed, max_len=48, d_choices=(8, 16))
    q, k, v, _ = _inputs(w, seed)
    scale = 1.0 / math.sqrt(w.d)
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions(), scale)
    O2, LSE2 = _dense_pack(q, k, v, w.lengths, scale)
    np.testing.assert_allclose(O, O2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(LSE, LSE2, rtol=0, atol=1e-12)


def _torch_reference(q, k, v, do, lengths):
    """float64 SDPA over the whole pool with a boolean block-diagonal causal mask."""
    n, h_q, d = q.shape
    G = h_q // k.shape[1]
    sid = torch.as_tensor(_sample_ids(lengths))
    pos = torch.arange(n)
    mask = (sid[:, None] == sid[None, :]) & (pos[None, :] <= pos[:, None])
    qt = q.double().transpose(0, 1).contiguous().requires_grad_(True)     # [h, n, d]
    kt = k.double().transpose(0, 1).contiguous().requires_grad_(True)
    vt = v.double().transpose(0, 1).contiguous().requires_grad_(True)
    kx = kt.repeat_interleave(G, dim=0)
    vx = vt.repeat_interleave(G, dim=0)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kx, vx, attn_mask=mask)
    o.backward(do.double().transpose(0, 1))
    return (o.detach().transpose(0, 1).numpy(), qt.grad.transpose(0, 1).numpy(),
            kt.grad.transpose(0, 1).numpy(), vt.grad.transpose(0, 1).numpy())


@pytest.mark.parametrize("seed", range(12))
def test_fwd_bwd_equal_torch_sdpa_autograd(seed):
    w = wl.tiny_random(seed, max_len=48, d_choices=(8, 16))
    q, k, v, do = _inputs(w, seed)
    o_ref, dq_ref, dk_ref, dv_ref = _torch_reference(q, k, v, do, w.lengths)
    O, _ = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    np.testing.assert_allclose(O, o_ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dQ, dq_ref, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dK, dk_ref, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dV, dv_ref, rtol=0, atol=1e-11)


def test_bwd_central_differences():
    w = wl.Workload("fd", 7, [[5, 3, 8]], h_q=4, h_kv=2, d=6, B=4, H=1, CP=1)
    q, k, v, do = (x.double() for x in _inputs(w, 7))
    pos = w.q_positions()

    def loss(qq, kk, vv):
        O, _ = oa.attention_fwd(qq, kk, vv, w.lengths, pos)
        return float((O * do.numpy()).sum())

    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, pos)
    rng = np.random.default_rng(0)
    eps = 1e-6
    for name, X, G in (("q", q, dQ), ("k", k, dK), ("v", v, dV)):
        for _ in range(12):
            idx = tuple(int(rng.integers(0, s)) for s in X.shape)
            Xp, Xm = X.clone(), X.clone()
            Xp[idx] += eps
            Xm[idx] -= eps
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = Xp, Xm
            num = (loss(args_p["q"], args_p["k"], args_p["v"])
                   - loss(args_m["q"], args_m["k"], args_m["v"])) / (2 * eps)
            assert num == pytest.approx(G[idx], abs=1e-7), (name, idx)


def test_zero_k_closed_forms():
    w = wl.tiny_random(3, max_len=64, d_choices=(16,))
    q, k, v, do = _inputs(w, 3, zero_k=True)
    pos = w.q_positions()
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, pos)
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, pos)
    G = w.h_q // w.h_kv
    vf, dof = v.double().numpy(), do.double().numpy()
    start = 0
    for n in w.lengths:
        for i in range(n):
            r = start + i
            for h in range(w.h_q):
                # uniform weights over the i+1 causal keys
                np.testing.assert_allclose(O[r, h], vf[start:r + 1, h // G].mean(0), atol=1e-13)
                assert LSE[h, r] == pytest.approx(math.log(i + 1), abs=1e-13)
            for g in range(w.h_kv):
                want = sum(dof[start + qq, g * G:(g + 1) * G].sum(0) / (qq + 1)
                           for qq in range(i, n))
                np.testing.assert_allclose(dV[r, g], want, atol=1e-12)
        start += n
    np.testing.assert_allclose(dQ, 0.0, atol=0)


def test_length_one_sample():
    w = wl.Workload("one", 5, [[1, 4, 1, 2]], h_q=2, h_kv=1, d=8, B=8, H=1, CP=1)
    q, k, v, _ = _inputs(w, 5)
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, w.q_positions())
    for r in (0, 5):
        for h in range(2):
            np.testing.assert_array_equal(O[r, h], v[r, 0].double().numpy())
            want = float(q[r, h].double() @ k[r, 0].double()) / math.sqrt(8)
            assert LSE[h, r] == pytest.approx(want, abs=1e-14)


@pytest.mark.parametrize("seed", range(6))
def test_gradient_column_sums(seed):
    w = wl.tiny_random(seed, max_len=64, d_choices=(16,))
    q, k, v, do = _inputs(w, seed)
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions())
    G = w.h_q // w.h_kv
    dof = do.double().numpy()
    start = 0
    for n in w.lengths:
        sl = slice(start, start + n)
        for g in range(w.h_kv):
            np.testing.assert_allclose(dK[sl, g].sum(0), 0.0, atol=1e-11)
            np.testing.assert_allclose(dV[sl, g].sum(0), dof[sl, g * G:(g + 1) * G].sum((0, 1)),
                                       atol=1e-11)
        start += n


def test_row_subsets_and_sparse_dout():
    """Rows computed alone equal the same rows of a full run; a dO that is zero
    off the chosen rows gives the same dK/dV as restricting to those rows."""
    w = wl.workload(wl.W_256K, scale=64)          # 4096-token pack, CP=16 share of rank 0
    q_all, k, v, do_all = wl.tensors(4, w.n_kv_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)
    pos_share = w.q_positions()
    q, do = q_all[pos_share], do_all[pos_share]
    rows = np.array([0, 1, 77, 127, 128, 200, 255])
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, pos_share, rows=rows, heads=[0, 17, 63])
    O_full, LSE_full = oa.attention_fwd(q_all, k, v, w.lengths, np.arange(w.n_kv_rows),
                                        rows=pos_share[rows], heads=[0, 17, 63])
    for h in (0, 17, 63):
        np.testing.assert_array_equal(O[:, h], O_full[:, h])
        np.testing.assert_array_equal(LSE[h], LSE_full[h])
    O_all, _ = oa.attention_fwd(q, k, v, w.lengths, pos_share, heads=[17])
    np.testing.assert_array_equal(O[:, 17], O_all[rows, 17])
    do_sparse = torch.zeros_like(do)
    do_sparse[rows] = do[rows]
    _, dK1, dV1 = oa.attention_bwd(q, k, v, do_sparse, w.lengths, pos_share, kv_heads=[1])
    _, dK2, dV2 = oa.attention_bwd(q, k, v, do_sparse, w.lengths, pos_share, rows=rows,
                                   kv_heads=[1])
    np.testing.assert_allclose(dK1, dK2, atol=1e-12)
    np.testing.assert_allclose(dV1, dV2, atol=1e-12)


@pytest.mark.parametrize("name", [wl.W_4K, wl.W_32K, wl.W_256K])
def test_useful_pairs_equal_plan_cost(name):
    w = wl.workload(name)
    cfg = op.PlanCfg(B=w.B, H=w.H, P=w.P, CP=w.CP, h_q=w.h_q, h_kv=w.h_kv, d=w.d)
    tiles = op.build_tiles(cfg, w.lengths, w.pack_tokens, w.q_ranges)
    assert sum(t.cost for t in tiles) == w.h_q * oa.useful_pairs(w.lengths, w.q_positions())


def test_dq_only_mode_matches_full_backward():
    """dkdv=False only skips the dK / dV sums: dQ is bit-identical."""
    w = wl.small_random(4)
    q, k, v, do = wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)
    rows = np.arange(0, w.n_q_rows, 7)
    dQ1, _, _ = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions(), rows=rows)
    dQ2, dK2, dV2 = oa.attention_bwd(q, k, v, do, w.lengths, w.q_positions(), rows=rows,
                                     dkdv=False)
    np.testing.assert_array_equal(dQ1, dQ2)
    assert not dK2.any() and not dV2.any()


@pytest.mark.parametrize("name,scale", [(wl.W_256K, 64), (wl.W_1M, 256), (wl.W_32K, 16)])
def test_zero_k_closed_forms_match_the_oracle(name, scale):
    """The K = 0 closed forms used at full size on the GPU (prefix means,
    reverse prefix sums of dO, suffix sums for dK) equal the oracle with K = 0,
    on replicas with a CP share (rows missing between the head and tail
    chunks) and on a whole pack."""
    import closed_forms as cf
    w = wl.workload(name, scale=scale)
    q, k, v, do = wl.tensors(w.seed, w.n_q_rows, w.n_kv_rows, w.h_q, w.h_kv, w.d)
    k = torch.zeros_like(k)
    pos = w.q_positions()
    O, LSE = oa.attention_fwd(q, k, v, w.lengths, pos)
    dQ, dK, dV = oa.attention_bwd(q, k, v, do, w.lengths, pos)
    G = w.h_q // w.h_kv
    scale_sm = 1.0 / np.sqrt(w.d)
    np.testing.assert_allclose(LSE, np.broadcast_to(
        np.log(pos - np.concatenate([[0], np.cumsum(w.lengths)])[
            np.searchsorted(np.cumsum(w.lengths), pos, side="right")] + 1.0), LSE.shape),
        atol=1e-12)
    np.testing.assert_allclose(dQ, 0.0, atol=1e-12)
    q64, do64, v64 = (t.double().numpy() for t in (q, do, v))
    for g in range(w.h_kv):
        hs = slice(g * G, (g + 1) * G)
        mean = cf.prefix_mean_v(v64[:, g], w.lengths, pos)
        np.testing.assert_allclose(O[:, g * G], mean, atol=1e-12)
        np.testing.assert_allclose(dV[:, g], cf.zero_k_dv(do64[:, hs], w.lengths, pos,
                                                          w.n_kv_rows), atol=1e-10)
        np.testing.assert_allclose(dK[:, g], cf.zero_k_dk(q64[:, hs], do64[:, hs], v64[:, g],
                                                          w.lengths, pos, w.n_kv_rows, scale_sm,
                                                          chunk=13), atol=1e-10)
