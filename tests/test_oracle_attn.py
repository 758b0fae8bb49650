"""Pins of the oracle's attention on codes (Sec. 2, Eqs. (1)-(2);
Sec. 3.1 overlap scores; Sec. 3.2 exactness of the tiled result; App. B
decode).

The paper prints no attention outputs, so nothing here compares with paper
values; instead the oracle is pinned by
  * a library routine: with k = d the codes are the dense rows, and SFA is
    plain softmax attention (torch's scaled_dot_product_attention, float64);
  * brute force on tiny inputs with the *sparse* formulation of the scores
    (intersection of supports, pure-Python loops);
  * closed forms: disjoint supports, one shared coordinate, n = 1;
  * invariants: coordinate permutation, rescaling, grouped heads, decode as
    the last forward row, split-context merge.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import logsumexp

import oracle


def _codes(rng, shape, d, k):
    x = rng.standard_normal(shape + (d,)).astype(np.float32)
    return oracle.topk_encode(x, k), x


def test_k_equals_d_is_dense_attention_sdpa():
    rng = np.random.default_rng(0)
    B, Hq, Hkv, n, d = 2, 4, 2, 37, 16
    (qi, qv), q = _codes(rng, (B, Hq, n), d, d)
    (ki, kv), k = _codes(rng, (B, Hkv, n), d, d)
    v = rng.standard_normal((B, Hkv, n, 24)).astype(np.float32)
    scale = 1 / math.sqrt(d)
    for causal in (True, False):
        O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, scale, causal)
        G = Hq // Hkv
        kt = torch.from_numpy(k).double().repeat_interleave(G, dim=1)
        vt = torch.from_numpy(v).double().repeat_interleave(G, dim=1)
        ref = F.scaled_dot_product_attention(torch.from_numpy(q).double(), kt, vt,
                                             is_causal=causal, scale=scale)
        assert np.abs(O - ref.numpy()).max() < 1e-12
        # LSE: library log-sum-exp of the library-computed dense scores
        s = torch.matmul(torch.from_numpy(q).double(), kt.transpose(-1, -2)).numpy() * scale
        if causal:
            s = np.where(np.tril(np.ones((n, n), bool)), s, -np.inf)
        assert np.abs(L - logsumexp(s, axis=-1)).max() < 1e-12


def _brute_force(qi, qv, ki, kv, v, scale, causal):
    """Sparse formulation, pure Python: s_ij = scale * sum over u in S_i cap S_j."""
    n = len(qi)
    O, L = [], []
    for i in range(n):
        qd = {int(u): float(a) for u, a in zip(qi[i], qv[i])}
        scores = []
        for j in range(n):
            if causal and j > i:
                continue
            kd = {int(u): float(b) for u, b in zip(ki[j], kv[j])}
            s = scale * sum(qd[u] * kd[u] for u in set(qd) & set(kd))
            scores.append((j, s))
        m = max(s for _, s in scores)
        w = [(j, math.exp(s - m)) for j, s in scores]
        l = sum(x for _, x in w)
        o = [sum(x * float(v[j][c]) for j, x in w) / l for c in range(len(v[0]))]
        O.append(o)
        L.append(m + math.log(l))
    return np.array(O), np.array(L)


@pytest.mark.parametrize("causal", [True, False])
def test_brute_force_tiny(causal):
    rng = np.random.default_rng(1)
    n, d, k = 9, 12, 4
    (qi, qv), _ = _codes(rng, (1, 1, n), d, k)
    (ki, kv), _ = _codes(rng, (1, 1, n), d, k)
    v = rng.standard_normal((1, 1, n, 5)).astype(np.float32)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.37, causal)
    Ob, Lb = _brute_force(qi[0, 0], qv[0, 0], ki[0, 0], kv[0, 0], v[0, 0], 0.37, causal)
    assert np.abs(O[0, 0] - Ob).max() < 1e-13
    assert np.abs(L[0, 0] - Lb).max() < 1e-13


def test_integer_codes_scores_exact():
    # small-integer values: every score is exact, so LSE of n=1 equals s_00 exactly
    qi = np.array([[[[0, 2, 5]]]]); qv = np.array([[[[3.0, -2.0, 1.0]]]], np.float32)
    ki = np.array([[[[2, 3, 5]]]]); kv = np.array([[[[4.0, 7.0, -5.0]]]], np.float32)
    v = np.array([[[[1.5, -2.5]]]], np.float32)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, 8, 1.0, True)
    assert L[0, 0, 0] == (-2.0 * 4.0) + (1.0 * -5.0)     # shared coords 2 and 5
    assert np.array_equal(O[0, 0, 0], [1.5, -2.5])     # n = 1: O_0 = v_0


@pytest.mark.parametrize("causal", [True, False])
def test_disjoint_supports_closed_form(causal):
    # Q on coordinates [0, k), K on [k, 2k): every score is 0, so every allowed
    # key has weight 1 (dense reading: non-overlapping keys still count).
    rng = np.random.default_rng(2)
    n, d, k = 50, 16, 4
    qi = np.broadcast_to(np.arange(k), (1, 1, n, k)).copy()
    ki = np.broadcast_to(np.arange(k, 2 * k), (1, 1, n, k)).copy()
    qv = rng.standard_normal((1, 1, n, k)).astype(np.float32)
    kv = rng.standard_normal((1, 1, n, k)).astype(np.float32)
    v = rng.standard_normal((1, 1, n, 8)).astype(np.float32)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.25, causal)
    vv = v[0, 0].astype(np.float64)
    if causal:
        want_O = np.cumsum(vv, axis=0) / np.arange(1, n + 1)[:, None]
        want_L = np.log(np.arange(1, n + 1))
    else:
        want_O = np.broadcast_to(vv.mean(axis=0), vv.shape)
        want_L = np.full(n, np.log(n))
    assert np.abs(O[0, 0] - want_O).max() < 1e-13
    assert np.abs(L[0, 0] - want_L).max() < 1e-13


def test_one_shared_coordinate_closed_form():
    # every query holds coordinate 3 with value a, every key holds it with b;
    # other coordinates are disjoint: s_ij = a*b*scale for all pairs.
    rng = np.random.default_rng(3)
    n, d, k, a, b, scale = 40, 32, 4, 1.25, -0.75, 0.3
    qi = np.tile(np.array([3, 10, 11, 12]), (1, 1, n, 1))
    ki = np.tile(np.array([3, 20, 21, 22]), (1, 1, n, 1))
    qv = rng.standard_normal((1, 1, n, k)).astype(np.float32); qv[..., 0] = a
    kv = rng.standard_normal((1, 1, n, k)).astype(np.float32); kv[..., 0] = b
    v = rng.standard_normal((1, 1, n, 6)).astype(np.float32)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, scale, True)
    vv = v[0, 0].astype(np.float64)
    assert np.abs(O[0, 0] - np.cumsum(vv, 0) / np.arange(1, n + 1)[:, None]).max() < 1e-13
    assert np.abs(L[0, 0] - (a * b * scale + np.log(np.arange(1, n + 1)))).max() < 1e-13


def test_invariants_permutation_and_rescale():
    rng = np.random.default_rng(4)
    B, H, n, d, k = 1, 2, 64, 32, 6
    (qi, qv), _ = _codes(rng, (B, H, n), d, k)
    (ki, kv), _ = _codes(rng, (B, H, n), d, k)
    v = rng.standard_normal((B, H, n, 16)).astype(np.float32)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.2, True)
    perm = rng.permutation(d)
    O2, L2 = oracle.attn_fwd(perm[qi], qv, perm[ki], kv, v, d, 0.2, True)
    assert np.abs(O - O2).max() < 1e-12 and np.abs(L - L2).max() < 1e-12
    O3, L3 = oracle.attn_fwd(qi, qv * np.float32(4.0), ki, kv, v, d, 0.05, True)
    assert np.abs(O - O3).max() < 1e-12 and np.abs(L - L3).max() < 1e-12


def test_gqa_equals_repeated_kv_heads():
    rng = np.random.default_rng(5)
    B, Hq, Hkv, n, d, k = 2, 6, 2, 33, 32, 8
    (qi, qv), _ = _codes(rng, (B, Hq, n), d, k)
    (ki, kv), _ = _codes(rng, (B, Hkv, n), d, k)
    v = oracle.bf16_rne(rng.standard_normal((B, Hkv, n, 32)).astype(np.float32))
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.17, True)
    rep = lambda a: np.repeat(a, Hq // Hkv, axis=1)
    O2, L2 = oracle.attn_fwd(qi, qv, rep(ki), rep(kv), rep(v), d, 0.17, True)
    assert np.array_equal(O, O2) and np.array_equal(L, L2)


def test_rows_entry_point_matches_full():
    rng = np.random.default_rng(6)
    n, d, k = 300, 64, 8
    (qi, qv), _ = _codes(rng, (1, 1, n), d, k)
    (ki, kv), _ = _codes(rng, (1, 1, n), d, k)
    v = rng.standard_normal((1, 1, n, 64)).astype(np.float32)
    O, L = oracle.attn_fwd(qi, qv, ki, kv, v, d, 0.125, True)
    rows = [0, 1, 63, 64, 127, 128, 299, 150]
    Or, Lr = oracle.attn_fwd_rows(qi[0, 0], qv[0, 0], ki[0, 0], kv[0, 0], v[0, 0], d, 0.125, True, rows)
    assert np.abs(Or - O[0, 0, rows]).max() < 1e-13
    assert np.abs(Lr - L[0, 0, rows]).max() < 1e-13


def test_decode_is_last_forward_row_and_merges():
    rng = np.random.default_rng(7)
    B, Hq, Hkv, Lmax, d, k = 3, 4, 2, 80, 32, 8
    (ci, cv), _ = _codes(rng, (B, Hkv, Lmax), d, k)
    cvb = oracle.bf16_rne(cv)
    (qi, qv), _ = _codes(rng, (B, Hq), d, k)
    vc = oracle.bf16_rne(rng.standard_normal((B, Hkv, Lmax, 32)).astype(np.float32))
    seq = np.array([80, 1, 47])
    O, L = oracle.attn_decode(qi, qv, ci, cvb, vc, d, 0.177, seq_len=seq)
    G = Hq // Hkv
    for b in range(B):
        Lb = seq[b]
        for h in range(Hq):
            g = h // G
            # forward whose last query row is q: earlier query rows do not matter
            fq_i = np.zeros((Lb, k), np.int64); fq_v = np.zeros((Lb, k), np.float32)
            fq_i[:] = np.arange(k); fq_i[-1] = qi[b, h]; fq_v[-1] = qv[b, h]
            Of, Lf = oracle.attn_fwd_rows(fq_i, fq_v, ci[b, g, :Lb], cvb[b, g, :Lb],
                                          vc[b, g, :Lb], d, 0.177, True, [Lb - 1])
            assert np.abs(O[b, h] - Of[0]).max() < 1e-13
            assert abs(L[b, h] - Lf[0]) < 1e-13
            # split the context in chunks and merge partial results by LSE
            parts = []
            for c0 in range(0, Lb, 16):
                c1 = min(Lb, c0 + 16)
                qd = oracle.densify(qi[b, h][None], qv[b, h][None], d)
                kd = oracle.densify(ci[b, g, c0:c1], cvb[b, g, c0:c1], d)
                parts.append(oracle.softmax_attention(qd, kd, oracle.widen(vc[b, g, c0:c1]), 0.177, False))
            lses = np.array([p[1][0] for p in parts])
            M = lses.max()
            w = np.exp(lses - M)
            Om = sum(wi * p[0][0] for wi, p in zip(w, parts)) / w.sum()
            assert np.abs(O[b, h] - Om).max() < 1e-12
            assert abs(L[b, h] - (M + np.log(w.sum()))) < 1e-12


def test_overlap_count_brute_force():
    rng = np.random.default_rng(8)
    n, d, k = 40, 16, 5
    (qi, _), _ = _codes(rng, (n,), d, k)
    (ki, _), _ = _codes(rng, (n,), d, k)
    for causal in (True, False):
        brute = sum(len(set(qi[i]) & set(ki[j]))
                    for i in range(n) for j in range(n) if (j <= i or not causal))
        assert oracle.overlap_count(qi, ki, causal, d) == brute


def test_overlap_count_matches_k2_over_d_for_uniform_supports():
    # Sec. 3.1 efficiency analysis: with balanced supports E ~ pairs * k^2 / d
    rng = np.random.default_rng(9)
    n, d, k = 2048, 128, 16
    (qi, _), _ = _codes(rng, (n,), d, k)
    (ki, _), _ = _codes(rng, (n,), d, k)
    E = oracle.overlap_count(qi, ki, False, d)
    assert abs(E / (n * n * k * k / d) - 1) < 0.01


def test_csr_bytes_memory_ratio():
    # App. J: int8 indices, int32 indptr, 2-byte values -> ratio ~ 2d / (3k + 4)
    N, d, k = 1 << 20, 128, 16
    ratio = N * d * 2 / oracle.csr_bytes(N, k, 2, 1, 4)
    assert abs(ratio - 2 * d / (3 * k + 4)) < 1e-4
