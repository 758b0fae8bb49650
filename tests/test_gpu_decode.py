"""GPU parity: sfa_attn_decode over a sparse-code KV cache against the
oracle.  The cache codes are written by sfa_topk_encode (int16 indices, bf16
values); the oracle codes the same dense keys with its own Top-k and bf16
rounding."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import TOL_O_BF16V, TOL_O_F32, check_lse, check_o, np_vals

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(B, Hq, Hkv, Lmax, d, k, v_bf16, seq, seed, cache_bf16=True):
    kd = torch.empty((B, Hkv, Lmax, d), device=DEV)
    vdt = torch.bfloat16 if v_bf16 else torch.float32
    vc = torch.empty((B, Hkv, Lmax, d), device=DEV, dtype=vdt)
    for b in range(B):
        for h in range(Hkv):
            kd[b, h] = si.normal((Lmax, d), seed, "k", b, h, device=DEV)
            vv = si.normal((Lmax, d), seed, "v", b, h, device=DEV)
            vc[b, h] = vv.to(vdt)
    qd = si.normal((B, Hq, d), seed, "q", device=DEV)
    ci, cv = sfa.sfa_topk_encode(kd, k, idx_dtype=torch.int16,
                                 val_dtype=torch.bfloat16 if cache_bf16 else torch.float32)
    qi, qv = sfa.sfa_topk_encode(qd, k)
    seq_t = None if seq is None else torch.tensor(seq, dtype=torch.int32, device=DEV)
    scale = 1.0 / math.sqrt(d)
    o, lse = sfa.sfa_attn_decode(qi, qv, ci, cv, vc, seq_len=seq_t, scale=scale,
                                 o_dtype=torch.float32)
    torch.cuda.synchronize()
    kn = kd.cpu().numpy()
    oci, ocv = (oracle.topk_encode_bf16 if cache_bf16 else oracle.topk_encode)(kn, k)
    oqi, oqv = oracle.topk_encode(qd.cpu().numpy(), k)
    O, L = oracle.attn_decode(oqi, oqv, oci, ocv, np_vals(vc), d, scale, seq_len=seq)
    check_o(o, O, TOL_O_BF16V if v_bf16 else TOL_O_F32, "decode O")
    check_lse(lse, L, "decode LSE")


@pytest.mark.parametrize(
    "B,Hq,Hkv,Lmax,d,k,v_bf16,seq",
    [
        (3, 8, 2, 300, 128, 16, True, [300, 1, 157]),
        (2, 4, 4, 5000, 64, 8, False, None),         # several context chunks, float32 V
        (2, 8, 1, 4097, 128, 16, True, [4097, 2049]),  # chunk boundaries, 8:1 groups
        (1, 2, 1, 64, 64, 64, False, None),           # k = d
        (2, 2, 2, 100, 128, 1, True, [100, 63]),      # k = 1
        (2, 4, 1, 3000, 128, 8, True, [3000, 1]),     # vectorized codes, k = 8
        (1, 8, 4, 2500, 64, 32, True, [2500]),        # vectorized codes, k = 32, d = 64
        (3, 2, 2, 777, 128, 16, True, [5, 777, 64]),  # vectorized codes, short sequences
    ])
def test_shapes(B, Hq, Hkv, Lmax, d, k, v_bf16, seq):
    _case(B, Hq, Hkv, Lmax, d, k, v_bf16, seq, seed=Lmax + k)


@pytest.mark.parametrize(
    "B,Hq,Hkv,Lmax,d,k,v_bf16,seq",
    [
        (2, 3, 1, 300, 80, 8, True, [300, 37]),          # three query heads per KV head
        (2, 8, 1, 4500, 96, 12, False, [4500, 2049]),    # chunks, 8:1 groups, float32 V
        (1, 2, 2, 100, 256, 16, True, None),             # d = 256
        (2, 4, 2, 129, 32, 32, True, [129, 1]),          # k = d = 32
        (1, 6, 2, 2100, 200, 10, True, [2100]),          # d = 200, group of 3
    ])
def test_other_head_dims(B, Hq, Hkv, Lmax, d, k, v_bf16, seq):
    """Head dimensions other than 64 and 128 run the float32 decode."""
    _case(B, Hq, Hkv, Lmax, d, k, v_bf16, seq, seed=d + Lmax)


@pytest.mark.parametrize(
    "B,Hq,Hkv,Lmax,d,k,v_bf16,seq",
    [
        (2, 6, 2, 5000, 128, 16, True, [5000, 77]),   # groups of 3, two chunks
        (1, 5, 1, 300, 128, 16, True, None),          # a group of 5
        (2, 10, 2, 700, 64, 8, False, [700, 1]),      # groups of 5 at d = 64
    ])
def test_group_not_power_of_two(B, Hq, Hkv, Lmax, d, k, v_bf16, seq):
    """Group sizes that are not a power of two run the float32 decode."""
    _case(B, Hq, Hkv, Lmax, d, k, v_bf16, seq, seed=Hq + Lmax)


def test_float32_cache_values():
    _case(2, 4, 1, 700, 128, 16, True, [700, 333], seed=3, cache_bf16=False)


def test_decode_64k_full_size_sampled():
    """The full 64-sequence x 64K-token cache (int16 indices, bf16 values, bf16
    V), all outputs computed on the GPU; the oracle rebuilds 6 sampled
    (sequence, head) outputs from regenerated dense keys."""
    w = si.workload("decode_64k")
    B, Hq, Hkv, L, d, k = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    ci = torch.empty((B, Hkv, L, k), dtype=torch.int16, device=DEV)
    cv = torch.empty((B, Hkv, L, k), dtype=torch.bfloat16, device=DEV)
    vc = torch.empty((B, Hkv, L, d), dtype=torch.bfloat16, device=DEV)
    for b in range(B):
        for h in range(Hkv):
            kd = si.normal((L, d), w.seed, "k", b, h, device=DEV)
            sfa.sfa_topk_encode(kd, k, idx=ci[b, h], val=cv[b, h])
            vc[b, h] = si.normal((L, d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
    qd = si.normal((B, Hq, d), w.seed, "q", device=DEV)
    qi, qv = sfa.sfa_topk_encode(qd, k)
    o, lse = sfa.sfa_attn_decode(qi, qv, ci, cv, vc, scale=w.scale, o_dtype=torch.float32)
    torch.cuda.synchronize()
    oqi, oqv = oracle.topk_encode(qd.cpu().numpy(), k)
    for (b, h) in [(0, 0), (0, 31), (17, 5), (33, 12), (63, 30), (63, 7)]:
        g = h // w.G
        kd = si.normal((L, d), w.seed, "k", b, g, device=DEV).cpu().numpy()
        oci, ocv = oracle.topk_encode_bf16(kd, k)
        qd1 = oracle.densify(oqi[b, h][None], oqv[b, h][None], d)
        kdd = oracle.densify(oci, ocv, d)
        O, Lse = oracle.softmax_attention(qd1, kdd, oracle.widen(np_vals(vc[b, g])), w.scale, False)
        check_o(o[b, h][None], O, TOL_O_BF16V, f"decode O ({b},{h})")
        check_lse(lse[b, h].reshape(1), Lse, f"decode LSE ({b},{h})")
