"""GPU parity: the 8-bit cache of "SFA (quant)" (App. E: SFA with 8-bit
activations) -- sfa_kv_append_q8 bit for bit against the oracle's Top-k
coding and per-row int8 quantisation (indices, int8 codes and float32
scales), and sfa_attn_decode_q8 against the oracle's decode of the values
the cache stands for (q * s)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import TOL_O_BF16V, check_lse, check_o, np_vals, oracle_topk_rows

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _q8_cache(B, Hkv, Lmax, d, k, idx_dtype=torch.int16, pages=None):
    rows = (B if pages is None else pages, Hkv, Lmax)
    return (torch.full(rows + (k,), -1, dtype=idx_dtype, device=DEV),
            torch.full(rows + (k,), 99, dtype=torch.int8, device=DEV),
            torch.full(rows, -1.0, dtype=torch.float32, device=DEV),
            torch.full(rows + (d,), 99, dtype=torch.int8, device=DEV),
            torch.full(rows, -1.0, dtype=torch.float32, device=DEV))


def _oracle_q8_rows(kd, vd, k):
    """The oracle's 8-bit cache rows of dense keys kd [R, d] (float32) and
    value rows vd [R, d] (float32, or uint16 bf16 bits)."""
    ci, cv = oracle_topk_rows(kd, k)
    kq, ks = oracle.quant_q8(cv)
    vv = oracle.widen(vd).astype(np.float32) if vd.dtype == np.uint16 else vd
    vq, vs = oracle.quant_q8(vv)
    return ci, kq, ks, vq, vs


@pytest.mark.parametrize(
    "B,Hkv,T,Lmax,d,k,seq,v_bf16,idx_dtype",
    [
        (2, 2, 37, 100, 128, 16, [3, 90], True, torch.int16),   # the second sequence fills up
        (1, 4, 20, 20, 64, 8, [0], False, torch.int16),        # float32 values in
        (3, 1, 9, 64, 128, 32, [10, 0, 55], True, torch.uint8),  # uint8 indices, k = 32
        (1, 1, 5, 8, 80, 5, [1], True, torch.int32),          # d = 80, int32 indices
    ])
def test_append_q8_bit_exact(B, Hkv, T, Lmax, d, k, seq, v_bf16, idx_dtype):
    seed = d + T + k
    kn = si.normal((B, Hkv, T, d), seed, "k_new", device=DEV)
    vn = si.normal((B, Hkv, T, d), seed, "v_new", device=DEV)
    if v_bf16:
        vn = vn.to(torch.bfloat16)
    ci, cv, cs, vc, vs = _q8_cache(B, Hkv, Lmax, d, k, idx_dtype)
    lens = torch.tensor(seq, dtype=torch.int32, device=DEV)
    sfa.sfa_kv_append_q8(kn, vn, lens, ci, cv, cs, vc, vs, k=k)
    torch.cuda.synchronize()
    # the oracle appends into its own copy of the sentinel-filled cache
    oci = np.full((B, Hkv, Lmax, k), -1, np.int64)
    ocv = np.full((B, Hkv, Lmax, k), 99, np.int8)
    ocs = np.full((B, Hkv, Lmax), -1.0, np.float32)
    ovc = np.full((B, Hkv, Lmax, d), 99, np.int8)
    ovs = np.full((B, Hkv, Lmax), -1.0, np.float32)
    new = oracle.kv_append_q8(oci, ocv, ocs, ovc, ovs, kn.cpu().numpy(), np_vals(vn),
                              np.array(seq), k)
    assert lens.cpu().numpy().tolist() == new.tolist()
    got_i = ci.cpu().numpy()
    assert np.array_equal(got_i, oci.astype(got_i.dtype))  # the sentinel -1 in the index type
    assert np.array_equal(cv.cpu().numpy(), ocv)
    assert np.array_equal(cs.cpu().numpy().view(np.uint32), ocs.view(np.uint32))
    assert np.array_equal(vc.cpu().numpy(), ovc)
    assert np.array_equal(vs.cpu().numpy().view(np.uint32), ovs.view(np.uint32))
    print(f"[parity] 8-bit append: {int(new.sum() - sum(seq))} rows x {Hkv} heads bit-exact "
          "(indices, int8 codes, scales)", flush=True)


def _decode_case(B, Hq, Hkv, Lmax, d, k, seq, seed, window=0, n_global=0, dense_q=False,
                 paged=False):
    kn = si.normal((B, Hkv, Lmax, d), seed, "k", device=DEV)
    vn = si.normal((B, Hkv, Lmax, d), seed, "v", device=DEV).to(torch.bfloat16)
    qd = si.normal((B, Hq, d), seed, "q", device=DEV)
    table = None
    if paged:
        P = 64
        max_pages = (Lmax + P - 1) // P
        g = torch.Generator(device="cpu")
        g.manual_seed(seed)
        table = torch.randperm(B * max_pages + 3, generator=g)[:B * max_pages]
        table = table.reshape(B, max_pages).to(torch.int32).to(DEV)
        ci, cv, cs, vc, vs = _q8_cache(B, Hkv, P, d, k, pages=B * max_pages + 3)
    else:
        ci, cv, cs, vc, vs = _q8_cache(B, Hkv, Lmax, d, k)
    lens = torch.zeros(B, dtype=torch.int32, device=DEV)
    sfa.sfa_kv_append_q8(kn, vn, lens, ci, cv, cs, vc, vs, k=k, block_table=table)
    seq_t = torch.tensor(seq, dtype=torch.int32, device=DEV) if seq is not None else None
    scale = 1.0 / math.sqrt(d)
    if dense_q:
        o, lse = sfa.sfa_attn_decode_q8(ci, cv, cs, vc, vs, block_table=table, seq_len=seq_t,
                                        q=qd, scale=scale, window=window, n_global=n_global)
    else:
        qi, qv = sfa.sfa_topk_encode(qd, k)
        o, lse = sfa.sfa_attn_decode_q8(ci, cv, cs, vc, vs, block_table=table, seq_len=seq_t,
                                        q_idx=qi, q_val=qv, scale=scale, window=window,
                                        n_global=n_global)
    torch.cuda.synchronize()
    # oracle: its own 8-bit cache of the same dense keys and values
    kk = kn.cpu().numpy().reshape(-1, d)
    ci_o, kq, ks, vq, vsc = _oracle_q8_rows(kk, np_vals(vn).reshape(-1, d), k)
    shape = (B, Hkv, Lmax)
    kvals = oracle.dequant_q8(kq, ks).reshape(shape + (k,))
    vvals = oracle.dequant_q8(vq, vsc).reshape(shape + (d,))
    oqi, oqv = oracle.topk_encode(qd.cpu().numpy(), k)
    O, L = oracle.attn_decode(oqi, oqv, ci_o.reshape(shape + (k,)), kvals, vvals, d, scale,
                              seq_len=seq, window=window, n_global=n_global)
    check_o(o, O, TOL_O_BF16V, "8-bit cache decode O")
    check_lse(lse, L, "8-bit cache decode LSE")


@pytest.mark.parametrize(
    "B,Hq,Hkv,Lmax,d,k,seq",
    [
        (3, 8, 2, 300, 128, 16, [300, 1, 157]),
        (2, 8, 1, 4097, 128, 16, [4097, 2049]),   # chunk boundaries, 8:1 groups
        (2, 4, 1, 3000, 128, 8, [3000, 1]),      # k = 8
        (1, 8, 4, 2500, 64, 32, [2500]),         # k = 32, d = 64
        (2, 2, 2, 777, 64, 16, None),            # G = 1
    ])
def test_decode_q8(B, Hq, Hkv, Lmax, d, k, seq):
    _decode_case(B, Hq, Hkv, Lmax, d, k, seq, seed=Lmax + k + d)


def test_decode_q8_window_dense_query_paged():
    _decode_case(2, 8, 2, 5000, 128, 16, [5000, 3000], seed=8, window=1000, n_global=3)
    _decode_case(2, 8, 2, 1500, 128, 16, [1500, 700], seed=9, dense_q=True)
    _decode_case(2, 4, 2, 1000, 128, 16, [1000, 333], seed=10, paged=True)


def test_decode_q8_64k_every_sequence():
    """The full 64-sequence x 64K-token step on the 8-bit cache, filled by
    sfa_kv_append_q8 from the same dense keys and values as the bf16 cache;
    for each sequence, every query head of KV head b mod 8 against the
    oracle, whose 8-bit cache rows are also compared bit for bit."""
    w = si.workload("decode_64k")
    B, Hq, Hkv, L, d, k, G = w.B, w.Hq, w.Hkv, w.n, w.d, w.k, w.G
    ci, cv, cs, vc, vs = _q8_cache(B, Hkv, L, d, k)
    for b in range(B):
        kb = torch.empty((1, Hkv, L, d), device=DEV)
        vb = torch.empty((1, Hkv, L, d), device=DEV, dtype=torch.bfloat16)
        for h in range(Hkv):
            kb[0, h] = si.normal((L, d), w.seed, "k", b, h, device=DEV)
            vb[0, h] = si.normal((L, d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
        sfa.sfa_kv_append_q8(kb, vb, torch.zeros(1, dtype=torch.int32, device=DEV), ci[b:b + 1],
                             cv[b:b + 1], cs[b:b + 1], vc[b:b + 1], vs[b:b + 1], k=k)
    del kb, vb
    qd = si.normal((B, Hq, d), w.seed, "q", device=DEV)
    qi, qv = sfa.sfa_topk_encode(qd, k)
    o, lse = sfa.sfa_attn_decode_q8(ci, cv, cs, vc, vs, q_idx=qi, q_val=qv, scale=w.scale)
    torch.cuda.synchronize()
    oqi, oqv = oracle.topk_encode(qd.cpu().numpy(), k)
    for b in range(B):
        g = b % Hkv
        kd = si.normal((L, d), w.seed, "k", b, g, device=DEV).cpu().numpy()
        vd = np_vals(si.normal((L, d), w.seed, "v", b, g, device=DEV).to(torch.bfloat16))
        ci_o, kq, ks, vq, vsc = _oracle_q8_rows(kd, vd, k)
        assert np.array_equal(ci[b, g].cpu().numpy().astype(np.int64), ci_o)
        assert np.array_equal(cv[b, g].cpu().numpy(), kq)
        assert np.array_equal(cs[b, g].cpu().numpy().view(np.uint32), ks.view(np.uint32))
        assert np.array_equal(vc[b, g].cpu().numpy(), vq)
        assert np.array_equal(vs[b, g].cpu().numpy().view(np.uint32), vsc.view(np.uint32))
        hs = list(range(g * G, (g + 1) * G))
        qdd = oracle.densify(oqi[b, hs], oqv[b, hs], d)
        kdd = oracle.densify(ci_o, oracle.dequant_q8(kq, ks), d)
        O, Ls = oracle.softmax_attention(qdd, kdd, oracle.dequant_q8(vq, vsc), w.scale, False)
        check_o(o[b, hs], O, TOL_O_BF16V, f"8-bit decode_64k O seq {b} (KV {g})")
        check_lse(lse[b, hs], Ls, f"8-bit decode_64k LSE seq {b} (KV {g})")
