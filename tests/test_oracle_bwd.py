"""Pins of the oracle's backward with the straight-through estimator
(Sec. 3.1, Eq. (6)): the gradient of a query / key coordinate is the
gradient of its code value on the support, zero elsewhere.

The oracle writes the chain rule out by hand; it is pinned against things
that do not share that derivation:
  * central finite differences of a scalar loss in the code values and V
    (the attention is smooth in the stored values, so these are the exact
    gradients up to O(h^2));
  * torch autograd (float64) through the dense formulation, with Top-k as
    a fixed mask, read at the supports -- Eq. (6) directly;
  * k = d: every coordinate is on the support, so the result is the
    gradient of plain softmax attention (torch SDPA, float64);
  * identities: sum_j dV_j = sum_i dO_i (each row of P sums to one), and
    the first query under the causal mask (its only key is key 0, weight 1
    whatever the score) has dq = 0;
  * the sampled row / column forms agree with the full backward;
  * O in its stored (bf16) form: unchanged results when every O_i is exact
    in bf16, and otherwise shifts of dq and dk that the forward oracle and
    the D-free dV part give independently.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _case(rng, B, Hq, Hkv, n, d, k, dv=None):
    dv = dv or d
    q = rng.standard_normal((B, Hq, n, d)).astype(np.float32)
    kk = rng.standard_normal((B, Hkv, n, d)).astype(np.float32)
    qi, qv = oracle.topk_encode(q, k)
    ki, kv = oracle.topk_encode(kk, k)
    v = rng.standard_normal((B, Hkv, n, dv)).astype(np.float32)
    do = rng.standard_normal((B, Hq, n, dv)).astype(np.float32)
    return qi, qv, ki, kv, v, do


def _loss(qi, qv, ki, kv, v, do, d, scale, causal):
    O, _ = oracle.attn_fwd(qi, qv.astype(np.float64), ki, kv.astype(np.float64),
                           v.astype(np.float64), d, scale, causal)
    return float((O * oracle.widen(do)).sum())


@pytest.mark.parametrize("causal", [True, False])
def test_finite_differences(causal):
    rng = np.random.default_rng(3)
    d, k, n = 16, 4, 9
    qi, qv, ki, kv, v, do = _case(rng, 1, 2, 1, n, d, k)
    scale = 1 / math.sqrt(d)
    dq, dk, dvv = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, scale, causal)
    h = 1e-6
    qv64, kv64, v64 = qv.astype(np.float64), kv.astype(np.float64), v.astype(np.float64)
    for arr, grad, name in ((qv64, dq, "q"), (kv64, dk, "k"), (v64, dvv, "v")):
        flat = arr.reshape(-1)
        for pos in rng.choice(flat.size, size=12, replace=False):
            old = flat[pos]
            flat[pos] = old + h
            lp = _loss(qi, qv64, ki, kv64, v64, do, d, scale, causal)
            flat[pos] = old - h
            lm = _loss(qi, qv64, ki, kv64, v64, do, d, scale, causal)
            flat[pos] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad.reshape(-1)[pos]) < 1e-6 * max(1.0, abs(fd)), (name, pos)


def test_autograd_through_dense_mask():
    """Eq. (6) read literally: Q~ = Q * M with M the (constant) Top-k mask, so
    dL/dQ = M * dL/dQ~; compare its values at the supports with the oracle."""
    rng = np.random.default_rng(5)
    B, Hq, Hkv, n, d, k = 2, 4, 2, 21, 32, 6
    q = rng.standard_normal((B, Hq, n, d))
    kk = rng.standard_normal((B, Hkv, n, d))
    v = rng.standard_normal((B, Hkv, n, 20))
    do = rng.standard_normal((B, Hq, n, 20))
    qi, qv = oracle.topk_encode(q.astype(np.float32), k)
    ki, kv = oracle.topk_encode(kk.astype(np.float32), k)
    qf, kf = q.astype(np.float32).astype(np.float64), kk.astype(np.float32).astype(np.float64)
    mq = np.zeros_like(qf); np.put_along_axis(mq, qi.astype(np.int64), 1.0, -1)
    mk = np.zeros_like(kf); np.put_along_axis(mk, ki.astype(np.int64), 1.0, -1)
    scale = 0.3
    G = Hq // Hkv
    for causal in (True, False):
        Q = torch.tensor(qf, requires_grad=True)
        K = torch.tensor(kf, requires_grad=True)
        V = torch.tensor(v, requires_grad=True)
        Qs = Q * torch.from_numpy(mq)
        Ks = (K * torch.from_numpy(mk)).repeat_interleave(G, dim=1)
        S = scale * torch.matmul(Qs, Ks.transpose(-1, -2))
        if causal:
            S = S.masked_fill(~torch.ones(n, n, dtype=torch.bool).tril(), float("-inf"))
        O = torch.matmul(torch.softmax(S, dim=-1), V.repeat_interleave(G, dim=1))
        (O * torch.from_numpy(do)).sum().backward()
        dq, dk, dvv = oracle.attn_bwd(qi, qv, ki, kv, v.astype(np.float64), do, d, scale, causal)
        gq = np.take_along_axis(Q.grad.numpy(), qi.astype(np.int64), -1)
        gk = np.take_along_axis(K.grad.numpy(), ki.astype(np.int64), -1)
        assert np.abs(gq - dq).max() < 1e-12
        assert np.abs(gk - dk).max() < 1e-12
        assert np.abs(V.grad.numpy() - dvv).max() < 1e-12
        # off-support coordinates carry no gradient (the mask's zeros)
        assert np.abs(Q.grad.numpy() * (1 - mq)).max() == 0.0


def test_k_equals_d_is_sdpa_backward():
    rng = np.random.default_rng(7)
    B, H, n, d = 1, 2, 17, 8
    qi, qv, ki, kv, v, do = _case(rng, B, H, H, n, d, d)
    for causal in (True, False):
        qd = torch.tensor(oracle.densify(qi, qv, d), requires_grad=True)
        kd = torch.tensor(oracle.densify(ki, kv, d), requires_grad=True)
        vt = torch.tensor(v.astype(np.float64), requires_grad=True)
        out = F.scaled_dot_product_attention(qd, kd, vt, is_causal=causal, scale=0.5)
        out.backward(torch.from_numpy(do.astype(np.float64)))
        dq, dk, dvv = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, 0.5, causal)
        assert np.abs(np.take_along_axis(qd.grad.numpy(), qi.astype(np.int64), -1) - dq).max() < 1e-11
        assert np.abs(np.take_along_axis(kd.grad.numpy(), ki.astype(np.int64), -1) - dk).max() < 1e-11
        assert np.abs(vt.grad.numpy() - dvv).max() < 1e-11


def test_dv_column_sum_and_first_row():
    rng = np.random.default_rng(11)
    B, Hq, Hkv, n, d, k = 1, 4, 2, 30, 32, 8
    qi, qv, ki, kv, v, do = _case(rng, B, Hq, Hkv, n, d, k)
    dq, dk, dvv = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, 0.2, True)
    G = Hq // Hkv
    for g in range(Hkv):
        # sum over keys of dV = sum over the group's queries of dO (rows of P sum to 1)
        want = oracle.widen(do)[0, g * G:(g + 1) * G].sum(axis=(0, 1))
        assert np.abs(dvv[0, g].sum(axis=0) - want).max() < 1e-10
    # row 0 attends only to key 0: its softmax weight is 1 whatever the score,
    # so its query gradient is exactly zero
    assert np.abs(dq[:, :, 0]).max() == 0.0


def test_rows_and_cols_match_the_full_backward():
    rng = np.random.default_rng(13)
    B, Hq, Hkv, n, d, k = 1, 4, 2, 40, 32, 8
    qi, qv, ki, kv, v, do = _case(rng, B, Hq, Hkv, n, d, k, dv=24)
    for causal in (True, False):
        dq, dk, dvv = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, 0.25, causal)
        rows = [0, 1, 17, 39]
        for h in range(Hq):
            g = h // (Hq // Hkv)
            got = oracle.attn_bwd_rows(qi[0, h], qv[0, h], ki[0, g], kv[0, g], v[0, g], do[0, h],
                                       d, 0.25, causal, rows)
            assert np.abs(got - dq[0, h, rows]).max() < 1e-12
        cols = [0, 5, 38, 39]
        for g in range(Hkv):
            hs = slice(g * 2, g * 2 + 2)
            gk, gv = oracle.attn_bwd_cols(qi[0, hs], qv[0, hs], ki[0, g], kv[0, g], v[0, g],
                                          do[0, hs], d, 0.25, causal, cols, row_chunk=7)
            assert np.abs(gk - dk[0, g, cols]).max() < 1e-12
            assert np.abs(gv - dvv[0, g, cols]).max() < 1e-12
            if causal:
                # rows below the first selected key add nothing under the causal mask
                late = [20, 38, 39]
                gk2, gv2 = oracle.attn_bwd_cols(qi[0, hs], qv[0, hs], ki[0, g], kv[0, g], v[0, g],
                                                do[0, hs], d, 0.25, causal, late, row_chunk=7,
                                                row_from=17)
                assert np.abs(gk2 - dk[0, g, late]).max() < 1e-12
                assert np.abs(gv2 - dvv[0, g, late]).max() < 1e-12


def test_stored_output_exact_in_bf16_changes_nothing():
    """V rows all equal to one bf16-exact vector: every O_i is that vector
    (the weights sum to one), its bf16 form is exact, and D_i, hence every
    gradient, is the same as with the exact output."""
    rng = np.random.default_rng(21)
    B, Hq, Hkv, n, d, k = 1, 4, 2, 24, 16, 4
    qi, qv, ki, kv, _, do = _case(rng, B, Hq, Hkv, n, d, k)
    row = rng.integers(-8, 9, size=d).astype(np.float32)
    v = np.broadcast_to(row, (B, Hkv, n, d)).copy()
    for causal in (True, False):
        a = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, 0.3, causal)
        b = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, 0.3, causal, o_store="bf16")
        for x, y in zip(a, b):
            assert np.abs(x - y).max() < 1e-12


def test_stored_output_shifts_dq_dk_as_the_forward_predicts():
    """With O rounded to bf16, D_i moves by dD_i = dO_i . (bf16(O_i) - O_i),
    so dS_ij moves by -P_ij dD_i:
      dq~_i moves by -scale dD_i sum_j P_ij k~_j, the forward's output with
        V replaced by the dense key codes;
      dk~_j moves by -scale sum_i P_ij dD_i q~_i, the backward's dV (which
        has no D term) with dO_i replaced by dD_i q~_i;
      dV does not move."""
    rng = np.random.default_rng(23)
    B, Hq, Hkv, n, d, k = 1, 4, 2, 28, 16, 4
    G = Hq // Hkv
    scale = 0.35
    qi, qv, ki, kv, v, do = _case(rng, B, Hq, Hkv, n, d, k)
    for causal in (True, False):
        dq0, dk0, dv0 = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, scale, causal)
        dq1, dk1, dv1 = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, scale, causal, o_store="bf16")
        assert np.abs(dv1 - dv0).max() < 1e-12
        O, _ = oracle.attn_fwd(qi, qv, ki, kv, v, d, scale, causal)
        dD = (do.astype(np.float64) * (oracle.stored_output(O, "bf16") - O)).sum(axis=-1)
        assert np.abs(dD).max() > 0  # the rounding does move D here
        kd = np.stack([oracle.densify(ki[0, g], kv[0, g], d) for g in range(Hkv)])[None]
        OK, _ = oracle.attn_fwd(qi, qv, ki, kv, kd, d, scale, causal)      # sum_j P_ij k~_j
        shift_q = -scale * dD[..., None] * OK
        want_q = dq0 + np.take_along_axis(shift_q, qi.astype(np.int64), -1)
        assert np.abs(dq1 - want_q).max() < 1e-12
        qd = np.stack([oracle.densify(qi[0, h], qv[0, h], d) for h in range(Hq)])[None]
        _, _, pq = oracle.attn_bwd(qi, qv, ki, kv, np.zeros((B, Hkv, n, d)), dD[..., None] * qd,
                                   d, scale, causal)                        # sum_i P_ij dD_i q~_i
        shift_k = -scale * pq
        want_k = dk0 + np.take_along_axis(shift_k, ki.astype(np.int64), -1)
        assert np.abs(dk1 - want_k).max() < 1e-12
        # the sampled forms take the same stored output
        rows = [0, 9, 27]
        for h in range(Hq):
            g = h // G
            got = oracle.attn_bwd_rows(qi[0, h], qv[0, h], ki[0, g], kv[0, g], v[0, g], do[0, h],
                                       d, scale, causal, rows, o_store="bf16")
            assert np.abs(got - dq1[0, h, rows]).max() < 1e-12
        cols = [0, 13, 27]
        for g in range(Hkv):
            hs = slice(g * G, g * G + G)
            gk, gv = oracle.attn_bwd_cols(qi[0, hs], qv[0, hs], ki[0, g], kv[0, g], v[0, g],
                                          do[0, hs], d, scale, causal, cols, o_store="bf16")
            assert np.abs(gk - dk1[0, g, cols]).max() < 1e-12
            assert np.abs(gv - dv1[0, g, cols]).max() < 1e-12
