"""Pins of the oracle's token-sparsity composition (App. E: SFA combined with
Longformer-style token patterns): the causal mask and'ed with a sliding
window |i - j| < w and n_global leading global tokens.

  * closed form: with disjoint supports every allowed score is 0, so O_i is
    the mean of the allowed values and LSE_i = ln(count_i), where count_i is
    written out from the pattern's geometry;
  * torch SDPA (float64) with a band mask built from tril / triu and global
    rows / columns set by slicing equals the oracle;
  * a window at least n long (no global tokens) is plain causal attention; a
    window of 1 leaves each query alone with its own key;
  * decode at position L-1 with a window equals attention over just the keys
    it may see, gathered by hand, with no mask, and equals the last row of the
    windowed forward.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _codes(rng, H, n, d, k, lo=0):
    """Codes whose supports lie in [lo, lo + k): disjoint for different lo."""
    idx = np.broadcast_to(np.arange(lo, lo + k), (1, H, n, k)).copy()
    val = rng.standard_normal((1, H, n, k)).astype(np.float32)
    return idx, val


@pytest.mark.parametrize("causal,w,g", [(True, 5, 0), (True, 5, 3), (True, 1, 0), (False, 4, 2),
                                        (True, 40, 0), (False, 7, 0)])
def test_disjoint_supports_closed_form(causal, w, g):
    rng = np.random.default_rng(w + 10 * g)
    n, d, k = 30, 16, 4
    qi, qv = _codes(rng, 1, n, d, k, 0)
    ki, kv = _codes(rng, 1, n, d, k, k)
    v = rng.standard_normal((1, 1, n, 8))
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.7, causal, window=w, n_global=g)
    for i in range(n):
        if causal:
            if i < g:
                keys = list(range(i + 1))
            else:
                keys = sorted(set(range(max(0, i - w + 1), i + 1)) | set(range(min(g, i + 1))))
        else:
            if i < g:
                keys = list(range(n))
            else:
                keys = sorted(set(range(max(0, i - w + 1), min(n, i + w))) | set(range(g)))
        assert abs(L[0, 0, i] - math.log(len(keys))) < 1e-12
        assert np.abs(O[0, 0, i] - v[0, 0, keys].mean(axis=0)).max() < 1e-12


@pytest.mark.parametrize("causal,w,g", [(True, 6, 0), (True, 6, 2), (False, 5, 3), (True, 3, 9)])
def test_sdpa_with_band_mask(causal, w, g):
    rng = np.random.default_rng(7)
    n, d, k = 25, 16, 5
    q = rng.standard_normal((1, 2, n, d)).astype(np.float32)
    kk = rng.standard_normal((1, 2, n, d)).astype(np.float32)
    v = rng.standard_normal((1, 2, n, 12))
    qi, qv = oracle.topk_encode(q, k)
    ki, kv = oracle.topk_encode(kk, k)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.3, causal, window=w, n_global=g)
    ones = torch.ones(n, n, dtype=torch.bool)
    band = torch.tril(ones, w - 1) & torch.triu(ones, -(w - 1))
    band[:g, :] = True
    band[:, :g] = True
    mask = band & torch.tril(ones) if causal else band
    qd = torch.from_numpy(oracle.densify(qi, qv, d))
    kd = torch.from_numpy(oracle.densify(ki, kv, d))
    ref = F.scaled_dot_product_attention(qd, kd, torch.from_numpy(v), attn_mask=mask, scale=0.3)
    assert np.abs(O - ref.numpy()).max() < 1e-12


def test_limits_of_the_window():
    rng = np.random.default_rng(8)
    n, d, k = 20, 16, 4
    q = rng.standard_normal((1, 1, n, d)).astype(np.float32)
    kk = rng.standard_normal((1, 1, n, d)).astype(np.float32)
    v = rng.standard_normal((1, 1, n, 6))
    qi, qv = oracle.topk_encode(q, k)
    ki, kv = oracle.topk_encode(kk, k)
    O0, L0 = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.5, True)
    O1, L1 = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.5, True, window=n)
    assert np.array_equal(O0, O1) and np.array_equal(L0, L1)
    O2, L2 = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.5, True, window=1)
    s = 0.5 * (oracle.densify(qi, qv, d) * oracle.densify(ki, kv, d)).sum(-1)
    assert np.abs(O2 - v).max() < 1e-12 and np.abs(L2 - s).max() < 1e-12


@pytest.mark.parametrize("w,g", [(16, 0), (16, 4), (1, 0), (100, 2)])
def test_decode_window(w, g):
    rng = np.random.default_rng(9)
    B, Hq, Hkv, Lmax, d, k = 2, 4, 2, 60, 16, 4
    kk = rng.standard_normal((B, Hkv, Lmax, d)).astype(np.float32)
    ki, kv = oracle.topk_encode(kk, k)
    v = rng.standard_normal((B, Hkv, Lmax, 8))
    qi, qv = oracle.topk_encode(rng.standard_normal((B, Hq, d)).astype(np.float32), k)
    lens = [Lmax, 37]
    O, L = oracle.attn_decode(qi, qv, ki, kv, v, d, 0.4, seq_len=lens, window=w, n_global=g)
    for b in range(B):
        Lb = lens[b]
        keys = sorted(set(range(max(0, Lb - w), Lb)) | set(range(min(g, Lb))))
        if Lb - 1 < g:
            keys = list(range(Lb))
        for h in range(Hq):
            qd = oracle.densify(qi[b, h][None], qv[b, h][None], d)
            kd = oracle.densify(ki[b, h // 2, keys], kv[b, h // 2, keys], d)
            s = 0.4 * (qd @ kd.T)[0]
            p = np.exp(s - s.max())
            assert np.abs(O[b, h] - p @ v[b, h // 2, keys] / p.sum()).max() < 1e-12
            assert abs(L[b, h] - (s.max() + math.log(p.sum()))) < 1e-12
        # the last row of the windowed forward whose last query is this one
        qs = np.zeros((1, Hq, Lb, k), dtype=np.int64); qsv = np.zeros((1, Hq, Lb, k), np.float32)
        qs[0, :, -1], qsv[0, :, -1] = qi[b], qv[b]
        Of, Lf = oracle.attn_fwd(qs, qsv, ki[b:b + 1, :, :Lb], kv[b:b + 1, :, :Lb],
                                 v[b:b + 1, :, :Lb], d, 0.4, True, window=w, n_global=g)
        assert np.abs(Of[0, :, -1] - O[b]).max() < 1e-12


@pytest.mark.parametrize("causal,w,g", [(True, 6, 0), (True, 5, 3), (False, 4, 2)])
def test_backward_with_window(causal, w, g):
    """The oracle's backward under the token mask: torch autograd (float64)
    through the dense formulation with the band mask built from tril / triu,
    read at the supports (Eq. (6)), and the row / column forms."""
    rng = np.random.default_rng(w + g)
    B, Hq, Hkv, n, d, k = 1, 2, 1, 23, 16, 4
    q = rng.standard_normal((B, Hq, n, d)).astype(np.float32)
    kk = rng.standard_normal((B, Hkv, n, d)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, n, 10))
    do = rng.standard_normal((B, Hq, n, 10))
    qi, qv = oracle.topk_encode(q, k)
    ki, kv = oracle.topk_encode(kk, k)
    dq, dk, dv = oracle.attn_bwd(qi, qv, ki, kv, v, do, d, 0.3, causal, window=w, n_global=g)
    ones = torch.ones(n, n, dtype=torch.bool)
    band = torch.tril(ones, w - 1) & torch.triu(ones, -(w - 1))
    band[:g, :] = True
    band[:, :g] = True
    mask = band & torch.tril(ones) if causal else band
    Qd = torch.tensor(oracle.densify(qi, qv, d), requires_grad=True)
    Kd = torch.tensor(oracle.densify(ki, kv, d), requires_grad=True)
    V = torch.tensor(v, requires_grad=True)
    S = 0.3 * torch.matmul(Qd, Kd.repeat_interleave(2, dim=1).transpose(-1, -2))
    O = torch.matmul(torch.softmax(S.masked_fill(~mask, float("-inf")), -1),
                     V.repeat_interleave(2, dim=1))
    (O * torch.from_numpy(do)).sum().backward()
    assert np.abs(np.take_along_axis(Qd.grad.numpy(), qi.astype(np.int64), -1) - dq).max() < 1e-12
    assert np.abs(np.take_along_axis(Kd.grad.numpy(), ki.astype(np.int64), -1) - dk).max() < 1e-12
    assert np.abs(V.grad.numpy() - dv).max() < 1e-12
    rows, cols = [0, 5, 22], [0, 3, 17, 22]
    got = oracle.attn_bwd_rows(qi[0, 1], qv[0, 1], ki[0, 0], kv[0, 0], v[0, 0], do[0, 1], d, 0.3,
                               causal, rows, window=w, n_global=g)
    assert np.abs(got - dq[0, 1, rows]).max() < 1e-12
    gk, gv = oracle.attn_bwd_cols(qi[0], qv[0], ki[0, 0], kv[0, 0], v[0, 0], do[0], d, 0.3, causal,
                                  cols, window=w, n_global=g)
    assert np.abs(gk - dk[0, 0, cols]).max() < 1e-12 and np.abs(gv - dv[0, 0, cols]).max() < 1e-12
