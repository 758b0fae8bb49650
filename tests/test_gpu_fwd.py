"""GPU parity: sfa_attn_fwd (fed by sfa_topk_encode) against the oracle.

The GPU path codes dense Q and K with its own encoder; the oracle codes the
same dense inputs with its own Top-k and evaluates the plain definition in
float64.  Tolerances: helpers.TOL_* (O 1e-5 float32 path, 5e-3 bf16-V path,
LSE 1e-4)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import (TOL_LSE, TOL_O_BF16V, TOL_O_F32, check_lse, check_o, np_vals,
                     sample_rows)

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _gpu_codes(x, k, idx_dtype=torch.int32, val_dtype=torch.float32):
    return sfa.sfa_topk_encode(x, k, idx_dtype=idx_dtype, val_dtype=val_dtype)


def _run_case(B, Hq, Hkv, n, d, k, causal, v_bf16, seed, idx_dtype=torch.int32,
              val_dtype=torch.float32, zipf_s=0.0, fwd=None, scale=None):
    fwd = fwd or sfa.sfa_attn_fwd
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed,
                            v_dtype=torch.bfloat16 if v_bf16 else torch.float32, device=DEV)
    if zipf_s:
        for b in range(B):
            for h in range(Hq):
                perm = si.zipf_feature_perm(d, seed, h // (Hq // Hkv))
                i_, v_ = si.zipf_codes(n, d, k, zipf_s, perm, seed, "q", b, h, device=DEV)
                q[b, h] = si.dense_from_codes(i_, v_, d)
            for h in range(Hkv):
                perm = si.zipf_feature_perm(d, seed, h)
                i_, v_ = si.zipf_codes(n, d, k, zipf_s, perm, seed, "k", b, h, device=DEV)
                kk[b, h] = si.dense_from_codes(i_, v_, d)
    qi, qv = _gpu_codes(q, k, idx_dtype, val_dtype)
    ki, kv = _gpu_codes(kk, k, idx_dtype, val_dtype)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    o32, lse = fwd(qi, qv, ki, kv, v, causal=causal, scale=scale, o_dtype=torch.float32)
    ob16 = None
    if v_bf16:
        ob16, _ = fwd(qi, qv, ki, kv, v, causal=causal, scale=scale, o_dtype=torch.bfloat16,
                      want_lse=False)
    torch.cuda.synchronize()
    # oracle: its own codes of the same dense inputs
    qn, kn, vn = q.cpu().numpy(), kk.cpu().numpy(), np_vals(v)
    if val_dtype == torch.bfloat16:
        oqi, oqv = oracle.topk_encode_bf16(qn, k)
        oki, okv = oracle.topk_encode_bf16(kn, k)
    else:
        oqi, oqv = oracle.topk_encode(qn, k)
        oki, okv = oracle.topk_encode(kn, k)
    O, L = oracle.attn_fwd(oqi, oqv, oki, okv, vn, d, scale, causal)
    tol = TOL_O_BF16V if v_bf16 else TOL_O_F32
    eo = check_o(o32, O, tol, "O (float32 output)")
    el = check_lse(lse, L, "LSE")
    if ob16 is not None:
        check_o(ob16, O, tol, "O (bf16 output)")
    return eo, el


def test_tiny_workload_fp32():
    w = si.workload("tiny")
    _run_case(w.B, w.Hq, w.Hkv, w.n, w.d, w.k, w.causal, w.v_bf16, w.seed)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16",
    [
        (1, 1, 1, 1, 64, 8, True, False),      # n = 1
        (1, 1, 1, 37, 64, 8, True, False),     # one ragged tile
        (2, 2, 2, 130, 64, 16, True, True),    # ragged tail past two tiles
        (1, 4, 1, 200, 128, 16, True, True),   # GQA 4:1, d = 128
        (1, 8, 1, 100, 128, 16, True, True),   # GQA 8:1 (two heads per wave)
        (1, 2, 1, 257, 128, 8, False, True),   # non-causal
        (1, 1, 1, 300, 64, 1, True, True),     # k = 1
        (1, 2, 2, 150, 64, 64, True, False),   # k = d: dense attention
        (1, 2, 1, 129, 128, 64, True, True),   # largest supported k at d = 128
        (2, 4, 2, 96, 128, 16, False, False),  # float32 V, GQA 2:1
        (1, 16, 1, 70, 64, 8, True, True),     # 16 heads per KV head
        (1, 2, 2, 140, 128, 128, True, True),  # k = d = 128
        (1, 8, 2, 700, 128, 16, True, True),   # GQA 4:1 over eleven key tiles
        (1, 2, 2, 333, 128, 16, True, False),  # float32 V, causal, ragged
    ])
def test_shapes(B, Hq, Hkv, n, d, k, causal, v_bf16):
    _run_case(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=B * 1000 + Hq * 100 + n)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16",
    [
        (1, 1, 1, 37, 64, 8, True, False),
        (2, 2, 2, 130, 64, 16, True, True),
        (1, 4, 1, 200, 128, 16, True, True),
        (1, 2, 1, 257, 128, 8, False, True),
        (1, 2, 2, 150, 64, 64, True, False),
        (1, 16, 1, 70, 64, 8, True, True),
        (1, 2, 1, 300, 128, 32, True, True),   # d = 128, 16 < k <= 64 (the k <= 64 tables)
        (1, 2, 2, 200, 128, 64, True, True),   # d = 128, k = 64, the largest supported
        (1, 32, 1, 150, 128, 16, True, True),  # 32 heads per KV head (4 rows per head and block)
        (1, 128, 1, 70, 128, 8, True, True),   # 128 heads per KV head (1 row per head and block)
        (1, 4, 2, 1000, 128, 4, True, True),   # small k over 16 key tiles
    ])
def test_index_variant(B, Hq, Hkv, n, d, k, causal, v_bf16):
    _run_case(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=B * 1000 + Hq * 100 + n + 7,
              fwd=sfa.sfa_attn_fwd_index)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16",
    [
        (1, 2, 1, 150, 32, 4, True, False),    # d = 32
        (1, 3, 1, 97, 80, 8, True, True),      # d = 80, three query heads per KV head
        (2, 2, 2, 70, 96, 12, False, False),   # d = 96, non-causal
        (1, 2, 2, 65, 256, 16, True, True),    # d = 256, the largest
        (1, 1, 1, 40, 200, 200, True, False),  # k = d = 200
        (1, 2, 1, 35, 16, 1, True, True),      # d = 16, k = 1
        (1, 6, 2, 300, 192, 24, True, True),   # d = 192, ten key tiles
    ])
def test_other_head_dims(B, Hq, Hkv, n, d, k, causal, v_bf16):
    """Head dimensions other than 64 and 128 run on the float32 vector-unit
    forward; any group size."""
    _run_case(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=d * 10 + n)


@pytest.mark.parametrize("scale,v_bf16", [(1.0, True), (-0.5, True), (0.0, True), (1.0, False),
                                           (-1.0 / 128, True), (2.0, True), (-1.0, True)])
def test_scales(scale, v_bf16):
    """Scales other than 1/sqrt(d), of either sign and zero.  At |scale| = 1
    the exponents reach ~50 (base 2), far above the first tiles' maxima: the
    lazily raised maximum and its rescaling run on most rows.  The score
    error is ~3 * 2^-22 of |scale| * sum |q_u k_u| (float16 pieces), so the
    LSE stays within 1e-4 at these scales too."""
    d = 128
    _run_case(1, 4, 1, 1100, d, 16, True, v_bf16, seed=31 + int(8 * abs(scale)), scale=scale)


@pytest.mark.parametrize("side", ["key", "query"])
def test_codes_beyond_float16_pieces(side):
    """Code values too large for the float16 score pieces (|x| >= 65504; for
    queries x includes scale * log2(e)) hand their workgroups to the rerun,
    which splits them into three bf16 pieces.  The scale keeps the scores
    moderate (an LSE in the thousands is not representable to 1e-4 in
    float32), so the ordinary tolerances apply."""
    B, Hq, Hkv, n, d, k = 1, 8, 2, 700, 128, 16
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, 95, v_dtype=torch.bfloat16, device=DEV)
    if side == "key":
        kk[0, 0, 70, 5] = 70000.0      # KV head 0, second tile
        kk[0, 1, 650, 100] = -3.0e5    # KV head 1, last tile
        scale = 1e-4
    else:
        kk *= 1e-5
        q[0, 2, 300, 7] = 70000.0      # x = 70000 * log2(e) > 65504
        q[0, 7, 5, 9] = -1.0e5
        scale = 1.0
    qi, qv = _gpu_codes(q, k)
    ki, kv = _gpu_codes(kk, k)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale, o_dtype=torch.float32)
    torch.cuda.synchronize()
    oqi, oqv = oracle.topk_encode(q.cpu().numpy(), k)
    oki, okv = oracle.topk_encode(kk.cpu().numpy(), k)
    O, L = oracle.attn_fwd(oqi, oqv, oki, okv, np_vals(v), d, scale, True)
    check_o(o32, O, TOL_O_BF16V, f"O with large {side} codes")
    check_lse(lse, L, f"LSE with large {side} codes")


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16",
    [
        (1, 6, 2, 300, 128, 16, True, True),   # groups of 3 query heads
        (1, 5, 1, 200, 128, 16, True, True),   # a group of 5
        (2, 10, 2, 130, 64, 16, False, True),  # groups of 5 at d = 64, non-causal
        (1, 3, 1, 150, 128, 8, True, False),   # group of 3, float32 V
    ])
def test_group_not_power_of_two(B, Hq, Hkv, n, d, k, causal, v_bf16):
    """Group sizes that are not a power of two run the float32 kernel at any
    head dim."""
    _run_case(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=Hq * 10 + n)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16",
    [
        (1, 4, 1, 700, 128, 2, True, True),    # k = 2, eleven key tiles
        (1, 8, 2, 300, 128, 1, True, True),    # k = 1, GQA 4:1
        (2, 2, 2, 257, 128, 2, False, True),   # non-causal, ragged
        (1, 1, 1, 200, 64, 1, True, True),     # d = 64: the dense product (faster there)
        (1, 16, 1, 130, 128, 2, True, True),   # 16 heads per KV head
        (1, 128, 1, 40, 128, 2, True, True),   # 128 heads per KV head (one row per head)
        (1, 2, 1, 1, 128, 2, True, True),      # n = 1
        (1, 6, 2, 300, 128, 2, True, True),    # groups of 3: the float32 kernel
    ])
def test_index_scores_small_k(B, Hq, Hkv, n, d, k, causal, v_bf16):
    """k <= 2 at d = 128 with bf16 V and near-uniform supports: sfa_attn_fwd
    scores through the per-tile inverted indexes (bucket walks) instead of the
    dense product."""
    _run_case(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=k * 100 + n + Hq)


def test_index_scores_skewed_supports():
    """Zipf-skewed supports at k = 2 make long buckets: the data-dependent
    choice may take either mode; the result must match either way."""
    _run_case(1, 4, 2, 1500, 128, 2, True, True, seed=14, zipf_s=1.1)


def test_index_scores_deterministic():
    q, kk, v = si.dense_qkv(1, 4, 1, 2100, 128, 19, device=DEV)
    qi, qv = _gpu_codes(q, 2)
    ki, kv = _gpu_codes(kk, 2)
    o1, l1 = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    o2, l2 = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_index_scores_v_beyond_float16_range():
    """The index mode hands workgroups whose keys reach a V value outside the
    float16 range to the bf16 rerun, like the dense mode."""
    B, Hq, Hkv, n, d, k = 1, 8, 2, 700, 128, 2
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, 97, v_dtype=torch.bfloat16, device=DEV)
    v[0, 0, 70, 5] = 65536.0
    v[0, 1, 650, 100] = -3.0e5
    qi, qv = _gpu_codes(q, k)
    ki, kv = _gpu_codes(kk, k)
    scale = 1.0 / math.sqrt(d)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale, o_dtype=torch.float32)
    torch.cuda.synchronize()
    oqi, oqv = oracle.topk_encode(q.cpu().numpy(), k)
    oki, okv = oracle.topk_encode(kk.cpu().numpy(), k)
    vn = np_vals(v)
    O, L = oracle.attn_fwd(oqi, oqv, oki, okv, vn, d, scale, True)
    tol = TOL_O_BF16V + 2.0 ** -16 * float(np.abs(oracle.widen(vn)).max())
    got = o32.double().cpu().numpy()
    err = np.abs(got - O).max()
    print(f"[parity] index mode, large V: max|O-O_oracle| = {err:.3e} (bound {tol:.3e})", flush=True)
    assert np.isfinite(got).all() and err <= tol
    check_lse(lse, L, "LSE (index mode, large V)")


def test_int16_indices_bf16_values():
    _run_case(1, 4, 2, 190, 128, 16, True, True, seed=77, idx_dtype=torch.int16,
              val_dtype=torch.bfloat16)


def test_zipf_small():
    _run_case(1, 2, 2, 260, 128, 8, True, True, seed=4, zipf_s=1.1)


@pytest.mark.parametrize("where", ["some_tiles", "every_tile"])
def test_v_beyond_float16_range(where):
    """bf16 V values of magnitude >= 65536 do not fit the float16 P.V path;
    the workgroups whose keys reach them are recomputed with bf16 V (P split
    hi + lo).  Some workgroups keep the float16 path, the others are redone:
    every output must match the oracle, to an error bound that scales with
    max|V| (2^-17 per weight, plus the bf16-output half-ulp)."""
    B, Hq, Hkv, n, d, k = 1, 8, 2, 700, 128, 16
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, 91, v_dtype=torch.bfloat16, device=DEV)
    big = [65536.0, -1.0e6, 3.0e5, 2.0e30]
    if where == "some_tiles":
        # KV head 0: key 70 (second tile); KV head 1: key 650 (last tile)
        v[0, 0, 70, 5] = big[0]
        v[0, 0, 70, 77] = big[1]
        v[0, 1, 650, 100] = big[2]
    else:
        for j in range(0, n, 64):
            v[0, j // 64 % Hkv, j, (7 * j) % d] = big[(j // 64) % len(big)]
    qi, qv = _gpu_codes(q, k)
    ki, kv = _gpu_codes(kk, k)
    scale = 1.0 / math.sqrt(d)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale, o_dtype=torch.float32)
    ob16, _ = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale, o_dtype=torch.bfloat16,
                               want_lse=False)
    torch.cuda.synchronize()
    oqi, oqv = oracle.topk_encode(q.cpu().numpy(), k)
    oki, okv = oracle.topk_encode(kk.cpu().numpy(), k)
    vn = np_vals(v)
    O, L = oracle.attn_fwd(oqi, oqv, oki, okv, vn, d, scale, True)
    vmax = float(np.abs(oracle.widen(vn)).max())
    tol = TOL_O_BF16V + 2.0 ** -16 * vmax
    got = o32.double().cpu().numpy()
    assert np.isfinite(got).all()
    err = np.abs(got - O).max()
    print(f"[parity] O with max|V| = {vmax:.3g}: max|O-O_oracle| = {err:.3e} (bound {tol:.3e})", flush=True)
    assert err <= tol
    check_o(ob16, O, tol, "O (bf16 output, large V)")
    check_lse(lse, L, "LSE (large V)")
    # rows whose keys hold no large value are held to the ordinary tolerance
    if where == "some_tiles":
        small = np.abs(O).max(axis=-1) < 100.0
        e_small = np.abs(got - O)[small].max()
        print(f"[parity] rows away from the large values: max|O-O_oracle| = {e_small:.3e}", flush=True)
        assert e_small <= TOL_O_BF16V


def test_gpt2s_workload_full():
    # every output of the GPT-2-small-shaped workload, against the oracle
    w = si.workload("gpt2s")
    _run_case(w.B, w.Hq, w.Hkv, w.n, w.d, w.k, w.causal, w.v_bf16, w.seed)


def _big_case_sampled(w, heads, zipf=False):
    """Full-size workload on the GPU (encode + forward), oracle on sampled rows."""
    G = w.G
    q = torch.empty((1, w.Hq, w.n, w.d), device=DEV)
    kk = torch.empty((1, w.Hkv, w.n, w.d), device=DEV)
    v = torch.empty((1, w.Hkv, w.n, w.d), device=DEV, dtype=torch.bfloat16)
    for h in range(w.Hq):
        if zipf:
            perm = si.zipf_feature_perm(w.d, w.seed, h // G)
            i_, v_ = si.zipf_codes(w.n, w.d, w.k, w.zipf_s, perm, w.seed, "q", 0, h, device=DEV)
            q[0, h] = si.dense_from_codes(i_, v_, w.d)
        else:
            q[0, h] = si.normal((w.n, w.d), w.seed, "q", 0, h, device=DEV)
    for h in range(w.Hkv):
        if zipf:
            perm = si.zipf_feature_perm(w.d, w.seed, h)
            i_, v_ = si.zipf_codes(w.n, w.d, w.k, w.zipf_s, perm, w.seed, "k", 0, h, device=DEV)
            kk[0, h] = si.dense_from_codes(i_, v_, w.d)
        else:
            kk[0, h] = si.normal((w.n, w.d), w.seed, "k", 0, h, device=DEV)
        v[0, h] = si.normal((w.n, w.d), w.seed, "v", 0, h, device=DEV).to(torch.bfloat16)
    qi, qv = _gpu_codes(q, w.k)
    ki, kv = _gpu_codes(kk, w.k)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale,
                                o_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = sample_rows(w.n, extra=(127, 128, 4095, 4096, w.n // 2), count=16, seed=w.seed)
    for h in heads:
        g = h // G
        kn = kk[0, g, : rows.max() + 1].cpu().numpy()
        oki, okv = oracle.topk_encode(kn, w.k)
        oqi, oqv = oracle.topk_encode(q[0, h, torch.from_numpy(rows).to(DEV)].cpu().numpy(), w.k)
        qi_full = np.zeros((w.n, w.k), np.int64); qv_full = np.zeros((w.n, w.k), np.float32)
        qi_full[rows], qv_full[rows] = oqi, oqv
        O, L = oracle.attn_fwd_rows(qi_full, qv_full, oki, okv,
                                    np_vals(v[0, g, : rows.max() + 1]), w.d, w.scale, w.causal, rows)
        sel = torch.from_numpy(rows).to(DEV)
        check_o(o32[0, h, sel], O, TOL_O_BF16V, f"O head {h}")
        check_lse(lse[0, h, sel], L, f"LSE head {h}")


def test_qwen3_32k_full_size_sampled():
    _big_case_sampled(si.workload("qwen3_32k"), heads=(0, 5, 31))


def test_zipf_128k_full_size_sampled():
    _big_case_sampled(si.workload("zipf_128k"), heads=(0, 7), zipf=True)


def test_deterministic():
    # the matrix-core forward has a fixed summation order: bitwise repeatable
    q, kk, v = si.dense_qkv(1, 4, 1, 500, 128, 9, device=DEV)
    qi, qv = _gpu_codes(q, 16)
    ki, kv = _gpu_codes(kk, 16)
    o1, l1 = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    o2, l2 = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_index_variant_repeatable():
    # the inverted-index variant: the order of keys inside a bucket may vary
    # between runs (the counting sort takes slots with atomics), but every
    # score entry has one owner that adds its overlaps in the row's code
    # order, so the results are bitwise repeatable
    q, kk, v = si.dense_qkv(1, 4, 1, 2100, 128, 9, device=DEV)
    qi, qv = _gpu_codes(q, 16)
    ki, kv = _gpu_codes(kk, 16)
    o1, l1 = sfa.sfa_attn_fwd_index(qi, qv, ki, kv, v, o_dtype=torch.float32)
    o2, l2 = sfa.sfa_attn_fwd_index(qi, qv, ki, kv, v, o_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
