"""GPU parity of the forward on 16-bit codes (bfloat16 or float16 values, the
code storage of App. J and of the decode cache) with bf16 V.

These take the one-product score path: the raw query and key values are the
matrix-core operands and the scale is applied to the float32 scores.  The oracle codes the same dense inputs with its own Top-k, rounds the
kept values to the same 16-bit type and evaluates the plain definition in
float64.  Tolerances as for every bf16-V forward: O 5e-3, LSE 1e-4."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import TOL_LSE, TOL_O_BF16V, check_lse, check_o, np_vals, sample_rows

pytestmark = pytest.mark.gpu
DEV = "cuda"
BF16, F16 = torch.bfloat16, torch.float16


def _oracle_codes(x: np.ndarray, k: int, val_dtype):
    return (oracle.topk_encode_f16 if val_dtype == F16 else oracle.topk_encode_bf16)(x, k)


def _case(B, Hq, Hkv, n, d, k, causal, val_dtype, seed, idx_dtype=torch.int32, scale=None,
          window=0, n_global=0):
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed, v_dtype=torch.bfloat16, device=DEV)
    qi, qv = sfa.sfa_topk_encode(q, k, idx_dtype=idx_dtype, val_dtype=val_dtype)
    ki, kv = sfa.sfa_topk_encode(kk, k, idx_dtype=idx_dtype, val_dtype=val_dtype)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale,
                                o_dtype=torch.float32, window=window, n_global=n_global)
    ob16, _ = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale,
                               o_dtype=torch.bfloat16, want_lse=False, window=window,
                               n_global=n_global)
    torch.cuda.synchronize()
    oqi, oqv = _oracle_codes(q.cpu().numpy(), k, val_dtype)
    oki, okv = _oracle_codes(kk.cpu().numpy(), k, val_dtype)
    O, L = oracle.attn_fwd(oqi, oqv, oki, okv, np_vals(v), d, scale, causal, window=window,
                           n_global=n_global)
    check_o(o32, O, TOL_O_BF16V, "O (float32 output)")
    check_o(ob16, O, TOL_O_BF16V, "O (bf16 output)")
    check_lse(lse, L, "LSE")


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,val_dtype",
    [
        (1, 1, 1, 1, 64, 8, True, F16),        # n = 1
        (1, 1, 1, 37, 64, 8, True, BF16),      # one ragged tile
        (2, 2, 2, 130, 64, 16, True, BF16),    # ragged tail past two tiles
        (1, 4, 1, 200, 128, 16, True, F16),    # GQA 4:1, d = 128
        (1, 8, 1, 100, 128, 16, True, BF16),   # GQA 8:1
        (1, 2, 1, 257, 128, 8, False, F16),    # non-causal
        (1, 1, 1, 300, 64, 1, True, BF16),     # k = 1
        (1, 16, 1, 70, 64, 8, True, F16),      # 16 heads per KV head
        (1, 8, 2, 700, 128, 16, True, BF16),   # GQA 4:1 over eleven key tiles
        (1, 8, 2, 700, 128, 16, True, F16),
        (1, 2, 2, 140, 128, 32, True, F16),    # k > 16
        (1, 4, 1, 333, 128, 128, True, BF16),  # k = d: dense attention
        (1, 2, 2, 200, 64, 40, False, F16),    # d = 64, k = 40, non-causal
    ])
def test_shapes(B, Hq, Hkv, n, d, k, causal, val_dtype):
    _case(B, Hq, Hkv, n, d, k, causal, val_dtype, seed=B * 1000 + Hq * 100 + n + 5)


@pytest.mark.parametrize("val_dtype", [BF16, F16])
def test_uint8_indices(val_dtype):
    _case(1, 4, 2, 390, 128, 16, True, val_dtype, seed=57, idx_dtype=torch.uint8)


@pytest.mark.parametrize("scale,val_dtype", [(1.0, BF16), (-0.5, F16), (0.0, BF16),
                                             (-1.0 / 128, BF16), (1.0, F16)])
def test_scales(scale, val_dtype):
    """Either sign (folded into the query operand's sign bit) and zero (the
    piece path).  The products of 16-bit values are exact and the scale is
    one float32 multiply: LSE within 1e-4 at these scales."""
    d = 128
    _case(1, 4, 1, 1100, d, 16, True, val_dtype, seed=41 + int(8 * abs(scale)), scale=scale)


@pytest.mark.parametrize("w,g,val_dtype", [(100, 0, BF16), (257, 64, F16), (128, 3, F16)])
def test_window(w, g, val_dtype):
    _case(1, 4, 2, 1500, 128, 16, True, val_dtype, seed=w + g, window=w, n_global=g)


def test_v_beyond_float16_range():
    """A bf16 V value outside the float16 range hands its workgroups to the
    rerun, which takes the two-piece path on the same 16-bit codes."""
    B, Hq, Hkv, n, d, k = 1, 8, 2, 700, 128, 16
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, 93, v_dtype=torch.bfloat16, device=DEV)
    v[0, 0, 70, 5] = 65536.0
    v[0, 1, 650, 100] = -3.0e5
    qi, qv = sfa.sfa_topk_encode(q, k, val_dtype=BF16)
    ki, kv = sfa.sfa_topk_encode(kk, k, val_dtype=BF16)
    scale = 1.0 / math.sqrt(d)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale, o_dtype=torch.float32)
    torch.cuda.synchronize()
    oqi, oqv = oracle.topk_encode_bf16(q.cpu().numpy(), k)
    oki, okv = oracle.topk_encode_bf16(kk.cpu().numpy(), k)
    vn = np_vals(v)
    O, L = oracle.attn_fwd(oqi, oqv, oki, okv, vn, d, scale, True)
    vmax = float(np.abs(oracle.widen(vn)).max())
    check_o(o32, O, TOL_O_BF16V + 2.0 ** -16 * vmax, "O (large V, 16-bit codes)")
    check_lse(lse, L, "LSE (large V, 16-bit codes)")


def test_deterministic():
    q, kk, v = si.dense_qkv(1, 4, 1, 500, 128, 9, device=DEV, v_dtype=torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, 16, val_dtype=F16)
    ki, kv = sfa.sfa_topk_encode(kk, 16, val_dtype=F16)
    o1, l1 = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    o2, l2 = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("val_dtype", [BF16, F16])
def test_qwen3_32k_full_size_sampled(val_dtype):
    """The 32K GQA workload (8 wavefronts per workgroup) with 16-bit codes:
    every row on the GPU, sampled rows of three heads by the oracle."""
    w = si.workload("qwen3_32k")
    G = w.G
    q = torch.empty((1, w.Hq, w.n, w.d), device=DEV)
    kk = torch.empty((1, w.Hkv, w.n, w.d), device=DEV)
    v = torch.empty((1, w.Hkv, w.n, w.d), device=DEV, dtype=torch.bfloat16)
    for h in range(w.Hq):
        q[0, h] = si.normal((w.n, w.d), w.seed, "q", 0, h, device=DEV)
    for h in range(w.Hkv):
        kk[0, h] = si.normal((w.n, w.d), w.seed, "k", 0, h, device=DEV)
        v[0, h] = si.normal((w.n, w.d), w.seed, "v", 0, h, device=DEV).to(torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, w.k, val_dtype=val_dtype)
    ki, kv = sfa.sfa_topk_encode(kk, w.k, val_dtype=val_dtype)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale,
                                o_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = sample_rows(w.n, extra=(127, 128, 4095, 4096, w.n // 2), count=16, seed=w.seed)
    for h in (0, 6, 31):
        g = h // G
        last = rows.max() + 1
        oki, okv = _oracle_codes(kk[0, g, :last].cpu().numpy(), w.k, val_dtype)
        oqi, oqv = _oracle_codes(q[0, h, torch.from_numpy(rows).to(DEV)].cpu().numpy(), w.k,
                                 val_dtype)
        qi_full = np.zeros((w.n, w.k), np.int64)
        qv_full = np.zeros((w.n, w.k), oqv.dtype)
        qi_full[rows], qv_full[rows] = oqi, oqv
        O, L = oracle.attn_fwd_rows(qi_full, qv_full, oki, okv, np_vals(v[0, g, :last]), w.d,
                                    w.scale, w.causal, rows)
        sel = torch.from_numpy(rows).to(DEV)
        check_o(o32[0, h, sel], O, TOL_O_BF16V, f"O head {h}")
        check_lse(lse[0, h, sel], L, f"LSE head {h}")
