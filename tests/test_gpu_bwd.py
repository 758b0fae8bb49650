"""GPU parity: sfa_attn_bwd (straight-through estimator, Sec. 3.1 Eq. (6))
against the oracle's backward.

The GPU path codes the dense Q, K with its own encoder, runs its own forward
for O and LSE, and then the backward; the oracle codes the same dense inputs
with its own Top-k and evaluates the plain chain rule in float64.  dO is a
seeded input shared by both.  Gradients are compared as a fraction of the
largest oracle gradient of the same tensor (helpers.TOL_GRAD)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import TOL_GRAD, check_grad, np_vals

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _run(B, Hq, Hkv, n, d, k, causal, v_bf16, seed, o_bf16=False, val_dtype=torch.float32):
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed,
                            v_dtype=torch.bfloat16 if v_bf16 else torch.float32, device=DEV)
    odt = torch.bfloat16 if o_bf16 else torch.float32
    dout = torch.empty((B, Hq, n, d), device=DEV)
    for b in range(B):
        for h in range(Hq):
            dout[b, h] = si.normal((n, d), seed, "dout", b, h, device=DEV)
    dout = dout.to(odt)
    qi, qv = sfa.sfa_topk_encode(q, k, val_dtype=val_dtype)
    ki, kv = sfa.sfa_topk_encode(kk, k, val_dtype=val_dtype)
    scale = 1.0 / math.sqrt(d)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale, o_dtype=odt)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=causal, scale=scale)
    torch.cuda.synchronize()
    enc = oracle.topk_encode_bf16 if val_dtype == torch.bfloat16 else oracle.topk_encode
    oqi, oqv = enc(q.cpu().numpy(), k)
    oki, okv = enc(kk.cpu().numpy(), k)
    # the GPU and oracle codes are bit-identical (encoder parity), so the
    # gradients line up entry by entry
    assert np.array_equal(qi.cpu().numpy(), oqi) and np.array_equal(ki.cpu().numpy(), oki)
    gq, gk, gv = oracle.attn_bwd(oqi, oqv, oki, okv, np_vals(v), np_vals(dout), d, scale, causal,
                                 o_store="bf16" if o_bf16 else None)
    tol = TOL_GRAD[(v_bf16, o_bf16)]
    e = (check_grad(dq, gq, tol, "dq_val"), check_grad(dk, gk, tol, "dk_val"),
         check_grad(dv, gv, tol, "dv"))
    return e


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16",
    [
        (1, 1, 1, 1, 64, 8, True, False),       # n = 1: every gradient but dv is zero
        (1, 1, 1, 37, 64, 8, True, False),      # one ragged tile
        (1, 4, 2, 100, 128, 16, True, True),    # GQA 2:1, ragged
        (2, 4, 1, 161, 128, 16, True, True),    # GQA 4:1, several key blocks
        (1, 2, 2, 130, 64, 16, False, True),    # non-causal
        (1, 1, 1, 70, 64, 1, True, True),       # k = 1
        (1, 2, 2, 96, 64, 64, True, False),     # k = d: dense attention gradients
        (1, 2, 1, 257, 128, 8, True, False),    # float32 V, past two key blocks
        (1, 4, 4, 64, 128, 32, True, True),     # exact tiles, G = 1
    ])
def test_shapes(B, Hq, Hkv, n, d, k, causal, v_bf16):
    _run(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=7 * n + k + Hq)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16,o_bf16",
    [
        (1, 6, 2, 150, 128, 16, True, True, False),  # groups of 3 query heads
        (1, 5, 1, 100, 128, 16, True, True, True),   # a group of 5, bf16 O and dO
        (1, 10, 2, 90, 64, 8, False, False, False),  # groups of 5 at d = 64, non-causal
    ])
def test_group_not_power_of_two(B, Hq, Hkv, n, d, k, causal, v_bf16, o_bf16):
    """Group sizes that are not a power of two run the float32 backward."""
    _run(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=Hq * 7 + n, o_bf16=o_bf16)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,v_bf16,o_bf16",
    [
        (1, 3, 1, 70, 80, 8, True, True, False),     # d = 80, group of 3
        (1, 2, 2, 100, 96, 12, False, False, False),  # d = 96, non-causal
        (1, 2, 1, 45, 256, 16, True, True, True),    # d = 256, bf16 O and dO
        (2, 1, 1, 33, 32, 32, True, False, False),   # k = d = 32
        (1, 4, 2, 130, 200, 20, True, True, False),  # d = 200, several blocks
    ])
def test_other_head_dims(B, Hq, Hkv, n, d, k, causal, v_bf16, o_bf16):
    """Head dimensions other than 64 and 128 run the float32 backward."""
    _run(B, Hq, Hkv, n, d, k, causal, v_bf16, seed=d + n, o_bf16=o_bf16)


def test_bf16_output_and_grad():
    _run(1, 4, 2, 150, 128, 16, True, True, seed=21, o_bf16=True)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal",
    [
        (1, 4, 1, 300, 64, 16, True),     # three 128-key blocks, ragged, GQA 4:1
        (2, 2, 2, 129, 64, 8, False),     # one key past a block, non-causal
        (1, 8, 2, 256, 64, 1, True),      # k = 1, whole blocks
        (1, 2, 1, 200, 64, 64, True),     # k = d: dense attention gradients
        (1, 12, 12, 1024, 64, 16, True),  # the gpt2s head shape, one sequence
    ])
def test_d64_bf16_fused(B, Hq, Hkv, n, d, k, causal):
    """d = 64 with bf16 V, O and dO and 32-bit codes: dk and dv come from
    one S, P, dP, dS per tile pair (the fused key-parallel kernel)."""
    _run(B, Hq, Hkv, n, d, k, causal, True, seed=5 * n + k, o_bf16=True)


def test_d64_bf16_fused_window():
    """The fused d = 64 kernel under a token window with global tokens."""
    B, Hq, Hkv, n, d, k, w, g = 1, 4, 2, 700, 64, 16, 150, 3
    seed = 11
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed, v_dtype=torch.bfloat16, device=DEV)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    scale = 1 / math.sqrt(d)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=scale, o_dtype=torch.bfloat16,
                              window=w, n_global=g)
    dout = si.normal((B, Hq, n, d), seed, "dout", device=DEV).to(torch.bfloat16)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=True, scale=scale,
                                  window=w, n_global=g)
    torch.cuda.synchronize()
    gq, gk, gv = oracle.attn_bwd(qi.cpu().numpy(), qv.cpu().numpy(), ki.cpu().numpy(),
                                 kv.cpu().numpy(), np_vals(v), np_vals(dout), d, scale, True,
                                 window=w, n_global=g, o_store="bf16")
    tol = TOL_GRAD[(True, True)]
    check_grad(dq, gq, tol, "dq_val (fused d = 64, window)")
    check_grad(dk, gk, tol, "dk_val (fused d = 64, window)")
    check_grad(dv, gv, tol, "dv (fused d = 64, window)")


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal",
    [
        (1, 4, 2, 150, 128, 16, True),   # GQA 2:1, ragged
        (2, 4, 1, 161, 64, 16, True),    # GQA 4:1, d = 64
        (1, 2, 2, 130, 64, 8, False),    # non-causal
    ])
def test_float32_v_bf16_o(B, Hq, Hkv, n, d, k, causal):
    """float32 V with bf16 O and dO: the tile images keep both pieces of V
    and the high piece of dO only."""
    _run(B, Hq, Hkv, n, d, k, causal, False, seed=13 * n + k, o_bf16=True)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,o_bf16",
    [
        (1, 4, 2, 150, 128, 16, True, True),   # bf16 codes, V, O, dO: one-piece code products
        (2, 4, 1, 161, 64, 16, True, True),
        (1, 2, 2, 130, 128, 32, False, True),
        (1, 4, 2, 150, 128, 16, True, False),  # float32 O and dO: the piece path
    ])
def test_bf16_codes(B, Hq, Hkv, n, d, k, causal, o_bf16):
    _run(B, Hq, Hkv, n, d, k, causal, True, seed=3 * n + d, o_bf16=o_bf16,
         val_dtype=torch.bfloat16)


def test_bf16_codes_match_widened_codes():
    """bf16 code values have a zero low bf16 piece, so the backward leaves
    their piece products out.  The same values widened to float32 take the
    general path, which adds those products as exact zeros: every gradient
    must be bitwise the same."""
    B, Hq, Hkv, n, d, k = 1, 8, 2, 300, 128, 16
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, 17, v_dtype=torch.bfloat16, device=DEV)
    dout = si.normal((B, Hq, n, d), 17, "dout", device=DEV).to(torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, k, val_dtype=torch.bfloat16)
    ki, kv = sfa.sfa_topk_encode(kk, k, val_dtype=torch.bfloat16)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.bfloat16)
    a = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout)
    b = sfa.sfa_attn_bwd(qi, qv.float(), ki, kv.float(), v, o, lse, dout)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_deterministic():
    torch.manual_seed(0)
    B, Hq, Hkv, n, d, k = 1, 4, 2, 200, 128, 16
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, 5, v_dtype=torch.bfloat16, device=DEV)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, o_dtype=torch.float32)
    dout = si.normal((B, Hq, n, d), 5, "dout", device=DEV)
    a = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout)
    b = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_qwen3_32k_full_size_sampled():
    """The 32K GQA workload in the bench's configuration (bf16 V, O and dO):
    all gradients computed on the GPU; the oracle rebuilds dq for sampled
    query rows of two heads and dk, dv for sampled keys of one KV head (its
    forward over all 32768 rows of the four query heads supplies LSE and O).
    Then every KV head (each runs on its own XCD in the persistent schedule):
    dq for sampled rows of one of its query heads, and dk, dv for sampled
    keys among the last 512, whose causal rows are the last 512."""
    w = si.workload("qwen3_32k")
    B, Hq, Hkv, n, d, k, G = w.B, w.Hq, w.Hkv, w.n, w.d, w.k, w.G
    q = torch.empty((B, Hq, n, d), device=DEV)
    kk = torch.empty((B, Hkv, n, d), device=DEV)
    v = torch.empty((B, Hkv, n, d), device=DEV, dtype=torch.bfloat16)
    dout = torch.empty((B, Hq, n, d), device=DEV, dtype=torch.bfloat16)
    for h in range(Hq):
        q[0, h] = si.normal((n, d), w.seed, "q", 0, h, device=DEV)
        dout[0, h] = si.normal((n, d), w.seed, "dout", 0, h, device=DEV).to(torch.bfloat16)
    for h in range(Hkv):
        kk[0, h] = si.normal((n, d), w.seed, "k", 0, h, device=DEV)
        v[0, h] = si.normal((n, d), w.seed, "v", 0, h, device=DEV).to(torch.bfloat16)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=True, scale=w.scale, o_dtype=torch.bfloat16)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=True, scale=w.scale)
    torch.cuda.synchronize()
    tol = TOL_GRAD[(True, True)]
    g = 5  # KV head under test; query heads 20..23 read it
    oki, okv = oracle.topk_encode(kk[0, g].cpu().numpy(), k)
    vn, dn = np_vals(v[0, g]), np_vals(dout[0])
    rng = np.random.default_rng(1)
    rows = np.unique(np.concatenate([[0, 1, 31, 32, 4095, 16383, n - 1], rng.integers(0, n, 9)]))
    for h in (G * g, G * g + 3):
        oqi, oqv = oracle.topk_encode(q[0, h].cpu().numpy(), k)
        ref = oracle.attn_bwd_rows(oqi, oqv, oki, okv, vn, dn[h], d, w.scale, True, rows,
                                   o_store="bf16")
        check_grad(dq[0, h, torch.from_numpy(rows).to(DEV)], ref, tol, f"dq_val head {h}")
    cols = np.unique(np.concatenate([[0, 1, 63, 127, 128, 20000, n - 1], rng.integers(0, n, 9)]))
    qc = [oracle.topk_encode(q[0, h].cpu().numpy(), k) for h in range(G * g, G * g + G)]
    gk, gv = oracle.attn_bwd_cols(np.stack([c[0] for c in qc]), np.stack([c[1] for c in qc]),
                                  oki, okv, vn, dn[G * g:G * g + G], d, w.scale, True, cols,
                                  o_store="bf16")
    sel = torch.from_numpy(cols).to(DEV)
    check_grad(dk[0, g, sel], gk, tol, f"dk_val KV head {g}")
    check_grad(dv[0, g, sel], gv, tol, f"dv KV head {g}")
    tail = n - 512
    for g2 in range(Hkv):
        oki2, okv2 = oracle.topk_encode(kk[0, g2].cpu().numpy(), k)
        vn2 = np_vals(v[0, g2])
        qc2 = [oracle.topk_encode(q[0, h].cpu().numpy(), k) for h in range(G * g2, G * g2 + G)]
        hq = g2 % G  # one query head of the group
        rows2 = np.unique(np.concatenate([[0, 255, 256, n - 1], rng.integers(0, n, 4)]))
        ref = oracle.attn_bwd_rows(qc2[hq][0], qc2[hq][1], oki2, okv2, vn2, dn[G * g2 + hq], d,
                                   w.scale, True, rows2, o_store="bf16")
        check_grad(dq[0, G * g2 + hq, torch.from_numpy(rows2).to(DEV)], ref, tol,
                   f"dq_val head {G * g2 + hq}")
        cols2 = np.unique(np.concatenate([[tail, n - 257, n - 256, n - 1],
                                          rng.integers(tail, n, 4)]))
        gk2, gv2 = oracle.attn_bwd_cols(np.stack([c[0] for c in qc2]), np.stack([c[1] for c in qc2]),
                                        oki2, okv2, vn2, dn[G * g2:G * g2 + G], d, w.scale, True,
                                        cols2, row_from=tail, o_store="bf16")
        sel2 = torch.from_numpy(cols2).to(DEV)
        check_grad(dk[0, g2, sel2], gk2, tol, f"dk_val KV head {g2} (last keys)")
        check_grad(dv[0, g2, sel2], gv2, tol, f"dv KV head {g2} (last keys)")
    print(f"[parity] qwen3_32k backward: dq rows of 2 + {Hkv} heads, dk / dv keys of every KV head",
          flush=True)


@pytest.mark.parametrize(
    "B,Hq,Hkv,n,d,k,causal,bf16,win,ng",
    [
        (2, 16, 8, 4500, 128, 16, True, True, 0, 0),    # dq: 3 rows of blocks per XCD, dk / dv: 2
        (1, 8, 8, 9000, 64, 8, False, False, 0, 0),     # G = 1, non-causal, float32 V, O and dO
        (1, 16, 8, 9000, 128, 16, False, True, 700, 3),  # token window: one workgroup per block
    ])
def test_persistent_grid_sampled(B, Hq, Hkv, n, d, k, causal, bf16, win, ng):
    """With B * Hkv a multiple of 8 (and no token window) the dq, dk and dv
    kernels run persistent grids; with more blocks than resident workgroups
    each workgroup takes several, in reversed slot order and sweep direction
    on every other row.  Sampled query rows and keys from blocks of every
    row, in the first and the last KV head, against the oracle; the windowed
    case checks the one-workgroup-per-block grid at the same shape."""
    seed = 77
    dt = torch.bfloat16 if bf16 else torch.float32
    q, kk, v = si.dense_qkv(B, Hq, Hkv, n, d, seed, v_dtype=dt, device=DEV)
    dout = torch.empty((B, Hq, n, d), device=DEV)
    for b in range(B):
        for h in range(Hq):
            dout[b, h] = si.normal((n, d), seed, "dout", b, h, device=DEV)
    dout = dout.to(dt)
    qi, qv = sfa.sfa_topk_encode(q, k)
    ki, kv = sfa.sfa_topk_encode(kk, k)
    scale = 1.0 / math.sqrt(d)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=causal, scale=scale, o_dtype=dt,
                              window=win, n_global=ng)
    dq, dk, dv = sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=causal, scale=scale,
                                  window=win, n_global=ng)
    torch.cuda.synchronize()
    tol = TOL_GRAD[(bf16, bf16)]
    G = Hq // Hkv
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([[0, 255, 256, n // 2, n - 1], rng.integers(0, n, 10)]))
    cols = np.unique(np.concatenate([[0, 255, 256, n - 300, n - 1], rng.integers(0, n, 10)]))
    for b, g in ((0, 0), (B - 1, Hkv - 1)):
        oki, okv = oracle.topk_encode(kk[b, g].cpu().numpy(), k)
        vn, dn = np_vals(v[b, g]), np_vals(dout[b])
        qc = [oracle.topk_encode(q[b, h].cpu().numpy(), k) for h in range(G * g, G * g + G)]
        for h in sorted({0, G - 1}):
            ref = oracle.attn_bwd_rows(qc[h][0], qc[h][1], oki, okv, vn, dn[G * g + h], d, scale,
                                       causal, rows, window=win, n_global=ng,
                                       o_store="bf16" if bf16 else None)
            check_grad(dq[b, G * g + h, torch.from_numpy(rows).to(DEV)], ref, tol,
                       f"dq_val batch {b} head {G * g + h}")
        gk, gv = oracle.attn_bwd_cols(np.stack([c[0] for c in qc]), np.stack([c[1] for c in qc]),
                                      oki, okv, vn, dn[G * g:G * g + G], d, scale, causal, cols,
                                      window=win, n_global=ng, o_store="bf16" if bf16 else None)
        sel = torch.from_numpy(cols).to(DEV)
        check_grad(dk[b, g, sel], gk, tol, f"dk_val batch {b} KV head {g}")
        check_grad(dv[b, g, sel], gv, tol, f"dv batch {b} KV head {g}")
