"""sfa_attn_decode_noalloc (decode on the library's static device scratch)
against sfa_attn_decode with a caller workspace: the same kernels and
chunking, so the outputs must agree bit for bit; two calls in a row, the
second with a smaller input, so the second reads a scratch the first filled."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import TOL_O_BF16V, check_lse, check_o, np_vals

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _cache(B, Hq, Hkv, L, d, k, seed):
    kd = torch.empty((B, Hkv, L, d), device=DEV)
    vc = torch.empty((B, Hkv, L, d), device=DEV, dtype=torch.bfloat16)
    for b in range(B):
        for h in range(Hkv):
            kd[b, h] = si.normal((L, d), seed, "k", b, h, device=DEV)
            vc[b, h] = si.normal((L, d), seed, "v", b, h, device=DEV).to(torch.bfloat16)
    qd = si.normal((B, Hq, d), seed, "q", device=DEV)
    ci, cv = sfa.sfa_topk_encode(kd, k, idx_dtype=torch.int16, val_dtype=torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(qd, k)
    return kd, vc, qd, ci, cv, qi, qv


def _both(qi, qv, ci, cv, vc, seq, window=0, n_global=0):
    B, Hq, _ = qi.shape
    d = vc.shape[-1]
    o_ref, l_ref = sfa.sfa_attn_decode(qi, qv, ci, cv, vc, seq_len=seq, o_dtype=torch.float32,
                                       window=window, n_global=n_global)
    o = torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=DEV)
    sfa.sfa_attn_decode_noalloc(qi, qv, ci, cv, vc, o, lse, seq_len=seq, window=window,
                                n_global=n_global)
    torch.cuda.synchronize()
    return o_ref, l_ref, o, lse


def _check_against_oracle(kd, vc, qd, o, lse, seq, k):
    d = vc.shape[-1]
    oci, ocv = oracle.topk_encode_bf16(kd.cpu().numpy(), k)
    oqi, oqv = oracle.topk_encode(qd.cpu().numpy(), k)
    O, L = oracle.attn_decode(oqi, oqv, oci, ocv, np_vals(vc), d, 1.0 / math.sqrt(d),
                              seq_len=None if seq is None else seq.cpu().numpy())
    check_o(o, O, TOL_O_BF16V, "noalloc decode O")
    check_lse(lse, L, "noalloc decode LSE")


def test_noalloc_matches_workspace_decode_twice():
    # first call: 3 sequences x 4 query heads over 2 KV heads, 9000-key cache
    # (3 chunks per sequence); second call: a smaller input (2 sequences,
    # 5000 keys) reusing the same scratch
    big = _cache(3, 4, 2, 9000, 128, 16, seed=71)
    kd, vc, qd, ci, cv, qi, qv = big
    seq = torch.tensor([9000, 4097, 1], dtype=torch.int32, device=DEV)
    o_ref, l_ref, o, lse = _both(qi, qv, ci, cv, vc, seq)
    assert torch.equal(o, o_ref) and torch.equal(lse, l_ref)
    _check_against_oracle(kd, vc, qd, o, lse, seq, 16)

    small = _cache(2, 8, 1, 5000, 64, 8, seed=72)
    kd, vc, qd, ci, cv, qi, qv = small
    o_ref, l_ref, o, lse = _both(qi, qv, ci, cv, vc, None)
    assert torch.equal(o, o_ref) and torch.equal(lse, l_ref)
    _check_against_oracle(kd, vc, qd, o, lse, None, 8)


def test_noalloc_window_64k_context():
    # 8 sequences of the 64K-key decode workload's shape (32 query heads over
    # 8 KV heads, d = 128, k = 16), ragged lengths, with a token window and
    # then without; the full 64-sequence step's 17 MB of partials fits too
    w = si.workload("decode_64k")
    B, Hq, Hkv, L, d, k = 8, w.Hq, w.Hkv, w.n, w.d, w.k
    assert sfa.sfa_attn_decode_workspace(64, Hq, L, d) <= 32 << 20
    kd, vc, qd, ci, cv, qi, qv = _cache(B, Hq, Hkv, L, d, k, seed=73)
    seq = torch.tensor([L, 100, 4096, 4097, 30000, 65535, 1, 5000], dtype=torch.int32, device=DEV)
    for window, n_global in ((4096, 4), (0, 0)):
        o_ref, l_ref, o, lse = _both(qi, qv, ci, cv, vc, seq, window, n_global)
        assert torch.equal(o, o_ref) and torch.equal(lse, l_ref), (window, n_global)

