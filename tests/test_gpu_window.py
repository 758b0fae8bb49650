"""GPU parity of SFA composed with token sparsity (App. E): a sliding window
|i - j| < window plus n_global leading global tokens, in the forward (key
tiles outside every row's window skipped), the backward (the same in each
kernel's tile loop) and decode (context outside the window skipped), against
the oracle's token_mask."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import (TOL_GRAD, TOL_O_BF16V, TOL_O_F32, check_grad, check_lse, check_o, np_vals,
                     sample_rows)

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("B,Hq,Hkv,n,d,k,causal,v_bf16,w,g", [
    (1, 4, 1, 700, 128, 16, True, True, 100, 0),     # window edge inside tiles
    (1, 4, 2, 900, 128, 16, True, True, 128, 3),     # global tokens, gap of skipped tiles
    (2, 2, 2, 333, 64, 8, True, False, 64, 70),      # globals past the first tile, float32 V
    (1, 8, 1, 517, 128, 16, False, True, 50, 2),     # non-causal window
    (1, 2, 1, 260, 128, 4, True, True, 1, 0),        # window 1: each query alone
    (1, 4, 4, 300, 64, 16, True, True, 1000, 0),     # window beyond n: plain causal
    (1, 4, 2, 1500, 128, 16, True, True, 257, 64),   # tile-aligned globals, odd window
    (1, 3, 1, 400, 96, 8, True, True, 45, 5),        # head dim 96: float32 vector kernel
    (1, 2, 2, 300, 48, 6, False, False, 33, 0),      # head dim 48, non-causal
    (1, 4, 2, 900, 128, 2, True, True, 128, 3),      # index scores (k <= 2): globals, gap
    (1, 8, 1, 517, 128, 1, False, True, 50, 2),      # index scores, non-causal window
    (1, 4, 1, 1500, 128, 2, True, True, 257, 64),    # index scores, tile-aligned globals
])
def test_fwd_window(B, Hq, Hkv, n, d, k, causal, v_bf16, w, g):
    seed = n + w + g
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed, device=DEV,
                            v_dtype=torch.bfloat16 if v_bf16 else torch.float32)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    scale = 1 / math.sqrt(d)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale,
                              o_dtype=torch.float32, window=w, n_global=g)
    torch.cuda.synchronize()
    O, L = oracle.attn_fwd(qi.cpu().numpy(), qv.cpu().numpy(), ki.cpu().numpy(),
                           kv.cpu().numpy(), np_vals(v), d, scale, causal, window=w, n_global=g)
    check_o(o, O, TOL_O_BF16V if v_bf16 else TOL_O_F32, f"fwd window {w} global {g} O")
    check_lse(lse, L, f"fwd window {w} global {g} LSE")


@pytest.mark.parametrize("val_dtype", [torch.float32, torch.bfloat16])
def test_fwd_window_qwen3_32k_sampled(val_dtype):
    """The 32K GQA workload with a 4096-token window and 4 global tokens: all
    rows on the GPU, sampled rows of two heads by the oracle (32-bit codes, and
    bf16 codes on the one-product score path)."""
    w_ = si.workload("qwen3_32k")
    B, Hq, Hkv, n, d, k, G = w_.B, w_.Hq, w_.Hkv, w_.n, w_.d, w_.k, w_.G
    win, ng = 4096, 4
    q = torch.empty((B, Hq, n, d), device=DEV)
    kk = torch.empty((B, Hkv, n, d), device=DEV)
    v = torch.empty((B, Hkv, n, d), device=DEV, dtype=torch.bfloat16)
    for h in range(Hq):
        q[0, h] = si.normal((n, d), w_.seed, "q", 0, h, device=DEV)
    for h in range(Hkv):
        kk[0, h] = si.normal((n, d), w_.seed, "k", 0, h, device=DEV)
        v[0, h] = si.normal((n, d), w_.seed, "v", 0, h, device=DEV).to(torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, k, val_dtype=val_dtype)
    ki, kv = sfa.sfa_topk_encode(kk, k, val_dtype=val_dtype)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=w_.scale,
                              o_dtype=torch.float32, window=win, n_global=ng)
    torch.cuda.synchronize()
    rows = sample_rows(n, extra=[3, 4, win - 1, win, win + 63, 20000], count=12, seed=4)
    for h in (0, 13):
        g = h // G
        ref = oracle.attn_fwd_rows(qi[0, h].cpu().numpy(), np_vals(qv[0, h]),
                                   ki[0, g].cpu().numpy(), np_vals(kv[0, g]),
                                   np_vals(v[0, g]), d, w_.scale, True, rows, window=win,
                                   n_global=ng)
        sel = torch.from_numpy(rows).to(DEV)
        check_o(o[0, h, sel], ref[0], TOL_O_BF16V, f"qwen3_32k window head {h} O")
        check_lse(lse[0, h, sel], ref[1], f"qwen3_32k window head {h} LSE")


def test_fwd_longest_sequence_window_sampled():
    """The longest sequence the forward takes at d = 128: n = 2^22, so that
    n * d = 2^29, the limit of the kernels' 32-bit per-head offsets.  A
    4096-token window with 4 global tokens keeps the run short; every tile
    image up to the last is read.  Sampled rows are checked against the
    oracle's plain softmax attention over the keys the row may see, gathered
    by hand (no mask): the global tokens and the window."""
    n, d, k, w, g = 1 << 22, 128, 16, 4096, 4
    q = si.normal((1, 1, n, d), 11, "q", device=DEV)
    kk = si.normal((1, 1, n, d), 11, "k", device=DEV)
    v = si.normal((1, 1, n, d), 11, "v", device=DEV).to(torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    del q, kk
    scale = 1 / math.sqrt(d)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale,
                              o_dtype=torch.float32, window=w, n_global=g)
    torch.cuda.synchronize()
    rows = [0, 1, 3, 4, w - 1, w, w + 63, 1 << 21, n - w, n - 65, n - 64, n - 2, n - 1]
    for i in rows:
        keys = sorted(set(range(min(g, i + 1))) | set(range(max(0, i - w + 1), i + 1)))
        kx = torch.tensor(keys, device=DEV)
        qd = oracle.densify(qi[0, 0, i:i + 1].cpu().numpy(), qv[0, 0, i:i + 1].cpu().numpy(), d)
        kd = oracle.densify(ki[0, 0, kx].cpu().numpy(), kv[0, 0, kx].cpu().numpy(), d)
        O, L = oracle.softmax_attention(qd, kd, oracle.widen(np_vals(v[0, 0, kx])), scale,
                                        causal=False)
        check_o(o[0, 0, i:i + 1], O, TOL_O_BF16V, f"n = 2^22 row {i} O")
        check_lse(lse[0, 0, i:i + 1], L, f"n = 2^22 row {i} LSE")


@pytest.mark.parametrize("w,g,seq,d", [(700, 0, [5000, 2500, 700], 128),
                                       (512, 4, [5000, 4097, 3], 128),
                                       (1, 0, [5000, 10, 1], 128),
                                       (3000, 2049, [5000, 2100, 4999], 128),
                                       (600, 3, [5000, 2100, 7], 96)])  # float32 decode
def test_decode_window(w, g, seq, d):
    B, Hq, Hkv, L, k, P = 3, 8, 2, 5000, 16, 64
    seed = w + g
    kd = torch.empty((B, Hkv, L, d), device=DEV)
    vc = torch.empty((B, Hkv, L, d), device=DEV, dtype=torch.bfloat16)
    for b in range(B):
        for h in range(Hkv):
            kd[b, h] = si.normal((L, d), seed, "k", b, h, device=DEV)
            vc[b, h] = si.normal((L, d), seed, "v", b, h, device=DEV).to(torch.bfloat16)
    ci, cv = sfa.sfa_topk_encode(kd, k, idx_dtype=torch.int16, val_dtype=torch.bfloat16)
    qd = si.normal((B, Hq, d), seed, "q", device=DEV)
    qi, qv = sfa.sfa_topk_encode(qd, k)
    seq_t = torch.tensor(seq, dtype=torch.int32, device=DEV)
    scale = 1 / math.sqrt(d)
    o, lse = sfa.sfa_attn_decode(qi, qv, ci, cv, vc, seq_len=seq_t, scale=scale,
                                 o_dtype=torch.float32, window=w, n_global=g)
    mp = (L + P - 1) // P
    pad = mp * P - L

    def paged(a):
        a = torch.cat([a, torch.zeros(a.shape[:2] + (pad,) + a.shape[3:], dtype=a.dtype,
                                      device=DEV)], 2) if pad else a
        return a.reshape(B, Hkv, mp, P, -1).permute(0, 2, 1, 3, 4).reshape(B * mp, Hkv, P, -1) \
                .contiguous()
    table = torch.arange(B * mp, dtype=torch.int32, device=DEV).reshape(B, mp)
    op, lp = sfa.sfa_attn_decode_paged(paged(ci), paged(cv), paged(vc), table, seq_len=seq_t,
                                       q=qd, scale=scale, o_dtype=torch.float32, window=w,
                                       n_global=g)
    torch.cuda.synchronize()
    assert torch.equal(op, o) and torch.equal(lp, lse)
    oci, ocv = oracle.topk_encode_bf16(kd.cpu().numpy(), k)
    oqi, oqv = oracle.topk_encode(qd.cpu().numpy(), k)
    O, Ls = oracle.attn_decode(oqi, oqv, oci, ocv, np_vals(vc), d, scale, seq_len=seq,
                               window=w, n_global=g)
    check_o(o, O, TOL_O_BF16V, f"decode window {w} global {g} O")
    check_lse(lse, Ls, f"decode window {w} global {g} LSE")


@pytest.mark.parametrize("B,Hq,Hkv,n,d,k,causal,v_bf16,w,g", [
    (1, 4, 2, 700, 128, 16, True, True, 100, 0),
    (1, 4, 1, 900, 128, 16, True, True, 200, 3),
    (1, 2, 2, 400, 64, 8, False, False, 60, 40),
    (1, 8, 1, 600, 128, 16, True, True, 1, 0),
    (2, 2, 1, 333, 128, 16, False, True, 45, 0),
    (1, 3, 1, 300, 96, 8, True, True, 40, 3),      # head dim 96: float32 backward
])
def test_bwd_window(B, Hq, Hkv, n, d, k, causal, v_bf16, w, g):
    seed = 3 * n + w + g
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed, device=DEV,
                            v_dtype=torch.bfloat16 if v_bf16 else torch.float32)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    scale = 1 / math.sqrt(d)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale, o_dtype=torch.float32,
                              window=w, n_global=g)
    dout = si.normal((B, Hq, n, d), seed, "dout", device=DEV)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=causal, scale=scale,
                                  window=w, n_global=g)
    torch.cuda.synchronize()
    gq, gk, gv = oracle.attn_bwd(qi.cpu().numpy(), qv.cpu().numpy(), ki.cpu().numpy(),
                                 kv.cpu().numpy(), np_vals(v), np_vals(dout), d, scale, causal,
                                 window=w, n_global=g)
    tol = TOL_GRAD[(v_bf16, False)]
    check_grad(dq, gq, tol, f"dq_val window {w} global {g}")
    check_grad(dk, gk, tol, f"dk_val window {w} global {g}")
    check_grad(dv, gv, tol, f"dv window {w} global {g}")


@pytest.mark.parametrize("Hq,Hkv,n,d,k,causal,v_bf16,o_bf16,w,g", [
    (4, 1, 2048, 128, 16, True, True, False, 128, 4),     # dK / dV kernels, 5 parts
    (2, 2, 2000, 128, 16, False, False, False, 100, 5),   # without causal masking, 2 parts
    (4, 2, 2048, 64, 8, True, True, True, 64, 4),         # fused d = 64 kernel, 3 parts
    (2, 1, 1500, 64, 8, False, True, True, 50, 33),       # fused, global keys in two tiles
    (4, 1, 1200, 128, 16, True, True, False, 100, 300),   # block 0 in 3 parts, block 1 (global
    (8, 1, 1200, 64, 8, True, True, True, 64, 300),       # keys too) whole; fused: 6 parts
])
def test_bwd_window_split(Hq, Hkv, n, d, k, causal, v_bf16, o_bf16, w, g):
    """Token window with global tokens over sequences long enough that key
    block 0's sweep (every query sees the global keys) is split over several
    work items and their partial results summed: every gradient against the
    oracle, and two runs bitwise identical."""
    B = 1
    seed = 7 * n + w + g
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed, device=DEV,
                            v_dtype=torch.bfloat16 if v_bf16 else torch.float32)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    scale = 1 / math.sqrt(d)
    odt = torch.bfloat16 if o_bf16 else torch.float32
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale, o_dtype=odt,
                              window=w, n_global=g)
    dout = si.normal((B, Hq, n, d), seed, "dout", device=DEV).to(odt)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=causal, scale=scale,
                                  window=w, n_global=g)
    dq2, dk2, dv2 = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=causal, scale=scale,
                                     window=w, n_global=g)
    torch.cuda.synchronize()
    assert torch.equal(dq, dq2) and torch.equal(dk, dk2) and torch.equal(dv, dv2)
    gq, gk, gv = oracle.attn_bwd(qi.cpu().numpy(), qv.cpu().numpy(), ki.cpu().numpy(),
                                 kv.cpu().numpy(), np_vals(v), np_vals(dout), d, scale, causal,
                                 window=w, n_global=g, o_store="bf16" if o_bf16 else None)
    tol = TOL_GRAD[(v_bf16, o_bf16)]
    check_grad(dq, gq, tol, f"dq_val window {w} global {g} (split)")
    check_grad(dk, gk, tol, f"dk_val window {w} global {g} (split)")
    check_grad(dv, gv, tol, f"dv window {w} global {g} (split)")


def test_bwd_window_qwen3_32k_sampled():
    """Backward on the 32K GQA workload with a 4096-token window and 4 global
    tokens (bf16 V, O, dO): dq rows of one head and dk, dv keys of one KV head
    against the oracle."""
    w_ = si.workload("qwen3_32k")
    B, Hq, Hkv, n, d, k, G = w_.B, w_.Hq, w_.Hkv, w_.n, w_.d, w_.k, w_.G
    win, ng = 4096, 4
    q = torch.empty((B, Hq, n, d), device=DEV)
    kk = torch.empty((B, Hkv, n, d), device=DEV)
    v = torch.empty((B, Hkv, n, d), device=DEV, dtype=torch.bfloat16)
    dout = torch.empty((B, Hq, n, d), device=DEV, dtype=torch.bfloat16)
    for h in range(Hq):
        q[0, h] = si.normal((n, d), w_.seed, "q", 0, h, device=DEV)
        dout[0, h] = si.normal((n, d), w_.seed, "dout", 0, h, device=DEV).to(torch.bfloat16)
    for h in range(Hkv):
        kk[0, h] = si.normal((n, d), w_.seed, "k", 0, h, device=DEV)
        v[0, h] = si.normal((n, d), w_.seed, "v", 0, h, device=DEV).to(torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=w_.scale,
                              o_dtype=torch.bfloat16, window=win, n_global=ng)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=True, scale=w_.scale,
                                  window=win, n_global=ng)
    torch.cuda.synchronize()
    tol = TOL_GRAD[(True, True)]
    g = 2
    oki, okv = ki[0, g].cpu().numpy(), kv[0, g].cpu().numpy()
    vn, dn = np_vals(v[0, g]), np_vals(dout[0])
    rows = np.array([0, 3, 4, 4095, 4096, 4160, 20000, n - 1])
    h = G * g + 1
    ref = oracle.attn_bwd_rows(qi[0, h].cpu().numpy(), qv[0, h].cpu().numpy(), oki, okv, vn,
                               dn[h], d, w_.scale, True, rows, window=win, n_global=ng,
                               o_store="bf16")
    check_grad(dq[0, h, torch.from_numpy(rows).to(DEV)], ref, tol, f"dq_val window head {h}")
    cols = np.array([0, 3, 4, 100, 4095, 4096, 30000, n - 1])
    hs = slice(G * g, G * g + G)
    gk, gv = oracle.attn_bwd_cols(qi[0, hs].cpu().numpy(), qv[0, hs].cpu().numpy(), oki, okv, vn,
                                  dn[hs], d, w_.scale, True, cols, window=win, n_global=ng,
                                  o_store="bf16")
    sel = torch.from_numpy(cols).to(DEV)
    check_grad(dk[0, g, sel], gk, tol, f"dk_val window KV head {g}")
    check_grad(dv[0, g, sel], gv, tol, f"dv window KV head {g}")
