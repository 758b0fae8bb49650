"""Full-size parity on the long workloads, against the oracle.

* Forward (Sec. 3.1 Eqs. (3)-(5), Sec. 3.2): qwen3_32k (32 query heads over 8
  KV heads, n = 32768) with float32 codes, with int16/bf16 codes and with
  k = 2 (scores through the per-tile inverted indexes), and zipf_128k (8
  heads, n = 131072, Zipf supports), run whole on the GPU; every
  query head is compared with the oracle on >= 4096 rows: rows 0, 1, n-1,
  both sides of every 64-row tile boundary, and random rows.  The float32 and
  bf16 outputs of sfa_attn_fwd and the output of the inverted-index forward
  (sfa_attn_fwd_index) are all compared on those rows.
* Top-k (Sec. 3.1 Eqs. (3)-(4)): every row of Q and K of the forward
  workloads, bit for bit (indices and values; float32 and bf16 values), with
  the rows whose k-th and (k+1)-th magnitudes tie counted.  For the decode
  cache (33.5M key rows) every such tie row and ~1M random rows.
* Decode (App. B): the 64 x 64K cache, every sequence with every query head
  of one KV head (KV head b mod 8, so each KV head is covered 8 times).

The oracle codes the same dense inputs with its own Top-k; nothing it reads
comes from the GPU path.  Its rows are independent and are run in parallel
(tests/helpers.py).
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import (TOL_O_BF16V, boundary_tie_rows, check_lse, check_o, full_size_rows,
                     np_vals, oracle_attn_rows, oracle_topk_rows, par_map)

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _dense_inputs(w):
    """Dense Q, K (float32) and V (bf16) of a forward workload, on the GPU,
    drawn slice by slice exactly as the benchmark draws them."""
    q = torch.empty((w.B, w.Hq, w.n, w.d), device=DEV)
    kk = torch.empty((w.B, w.Hkv, w.n, w.d), device=DEV)
    v = torch.empty((w.B, w.Hkv, w.n, w.d), device=DEV, dtype=torch.bfloat16)
    for b in range(w.B):
        for h in range(w.Hq):
            if w.zipf_s:
                perm = si.zipf_feature_perm(w.d, w.seed, h // w.G)
                i_, v_ = si.zipf_codes(w.n, w.d, w.k, w.zipf_s, perm, w.seed, "q", b, h, device=DEV)
                q[b, h] = si.dense_from_codes(i_, v_, w.d)
            else:
                q[b, h] = si.normal((w.n, w.d), w.seed, "q", b, h, device=DEV)
        for h in range(w.Hkv):
            if w.zipf_s:
                perm = si.zipf_feature_perm(w.d, w.seed, h)
                i_, v_ = si.zipf_codes(w.n, w.d, w.k, w.zipf_s, perm, w.seed, "k", b, h, device=DEV)
                kk[b, h] = si.dense_from_codes(i_, v_, w.d)
            else:
                kk[b, h] = si.normal((w.n, w.d), w.seed, "k", b, h, device=DEV)
            v[b, h] = si.normal((w.n, w.d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
    return q, kk, v


def _run_workload(name, codes16=False, index=True, k=0):
    """Encode + forward on the GPU at full size; keep the dense inputs, the
    GPU codes and the outputs at the sampled rows on the host."""
    w = si.workload(name)
    if k:
        w = dataclasses.replace(w, k=k)
    print(f"[fullsize] {name} codes16={codes16}: GPU encode + forward", flush=True)
    q, kk, v = _dense_inputs(w)
    idt, vdt = (torch.int16, torch.bfloat16) if codes16 else (torch.int32, torch.float32)
    qi, qv = sfa.sfa_topk_encode(q, w.k, idx_dtype=idt, val_dtype=vdt)
    ki, kv = sfa.sfa_topk_encode(kk, w.k, idx_dtype=idt, val_dtype=vdt)
    o32, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale,
                                o_dtype=torch.float32)
    rows = full_size_rows(w.n, w.seed)
    sel = torch.from_numpy(rows).to(DEV)
    out = {"w": w, "rows": rows,
           "o32": o32[0][:, sel].cpu(), "lse": lse[0][:, sel].cpu()}
    del o32, lse
    ob16, _ = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale,
                               o_dtype=torch.bfloat16, want_lse=False)
    out["ob16"] = ob16[0][:, sel].cpu()
    del ob16
    if index:
        oi, li = sfa.sfa_attn_fwd_index(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale,
                                        o_dtype=torch.float32)
        out["oi"], out["li"] = oi[0][:, sel].cpu(), li[0][:, sel].cpu()
        del oi, li
    torch.cuda.synchronize()
    out.update(q=q[0].cpu().numpy(), k=kk[0].cpu().numpy(), v=np_vals(v[0]),
               qi=qi[0].cpu().numpy(), qv=np_vals(qv[0]), ki=ki[0].cpu().numpy(),
               kv=np_vals(kv[0]))
    del q, kk, v, qi, qv, ki, kv
    torch.cuda.empty_cache()
    return out


@pytest.fixture(scope="module")
def qwen3_f32():
    return _run_workload("qwen3_32k")


@pytest.fixture(scope="module")
def qwen3_codes16():
    return _run_workload("qwen3_32k", codes16=True, index=False)


@pytest.fixture(scope="module")
def zipf():
    return _run_workload("zipf_128k")


@pytest.fixture(scope="module")
def qwen3_k2():
    # k = 2: the forward scores through the per-tile inverted indexes
    return _run_workload("qwen3_32k", index=False, k=2)


def _oracle_codes(x, k, bf16):
    i_, v_ = oracle_topk_rows(x, k)
    return (i_, oracle.bf16_rne(v_)) if bf16 else (i_, v_)


def _check_kv_group(run, g, bf16_codes):
    """Compare every query head of KV head g on the sampled rows."""
    w, rows = run["w"], run["rows"]
    oki, okv = _oracle_codes(run["k"][g, : rows.max() + 1], w.k, bf16_codes)
    kd = oracle.densify(oki, okv, w.d)
    vv = oracle.widen(run["v"][g, : rows.max() + 1])
    for h in range(g * w.G, (g + 1) * w.G):
        oqi, oqv = _oracle_codes(run["q"][h, rows], w.k, bf16_codes)
        qd = oracle.densify(oqi, oqv, w.d)
        O, L = oracle_attn_rows(qd, kd, vv, w.scale, w.causal, rows)
        tag = f"{w.name} head {h} (KV {g}), {len(rows)} rows"
        check_o(run["o32"][h], O, TOL_O_BF16V, f"O {tag}")
        check_lse(run["lse"][h], L, f"LSE {tag}")
        check_o(run["ob16"][h], O, TOL_O_BF16V, f"O bf16 output {tag}")
        if "oi" in run:
            check_o(run["oi"][h], O, TOL_O_BF16V, f"index-forward O {tag}")
            check_lse(run["li"][h], L, f"index-forward LSE {tag}")


@pytest.mark.parametrize("g", range(8))
def test_qwen3_32k_every_head(qwen3_f32, g):
    _check_kv_group(qwen3_f32, g, bf16_codes=False)


@pytest.mark.parametrize("g", range(8))
def test_qwen3_32k_codes16_every_head(qwen3_codes16, g):
    _check_kv_group(qwen3_codes16, g, bf16_codes=True)


@pytest.mark.parametrize("h", range(8))
def test_zipf_128k_every_head(zipf, h):
    _check_kv_group(zipf, h, bf16_codes=False)


@pytest.mark.parametrize("g", range(8))
def test_qwen3_32k_k2_index_scores_every_head(qwen3_k2, g):
    _check_kv_group(qwen3_k2, g, bf16_codes=False)


def _check_topk_all(x, gi, gv, k, bf16, what):
    ri, rv = _oracle_codes(x, k, bf16)
    gi = gi.reshape(ri.shape).astype(np.int64)
    gv = gv.reshape(rv.shape)
    ties = boundary_tie_rows(x, k)
    bad_i = np.flatnonzero((gi != ri).any(axis=1))
    bad_v = np.flatnonzero((gv.view(np.uint16 if bf16 else np.uint32) !=
                            rv.view(np.uint16 if bf16 else np.uint32)).any(axis=1))
    print(f"[parity] Top-k {what}: {ri.shape[0]} rows, {ties.size} boundary-tie rows; "
          f"index mismatches {bad_i.size}, value mismatches {bad_v.size}", flush=True)
    assert bad_i.size == 0, f"{what}: indices differ in rows {bad_i[:5]}"
    assert bad_v.size == 0, f"{what}: values differ in rows {bad_v[:5]}"


@pytest.mark.parametrize("which", ["q", "k"])
def test_topk_every_row_qwen3(qwen3_f32, which):
    r = qwen3_f32
    x = r[which].reshape(-1, r["w"].d)
    _check_topk_all(x, r[which + "i"], r[which + "v"], r["w"].k, False, f"qwen3_32k {which}")


@pytest.mark.parametrize("which", ["q", "k"])
def test_topk_every_row_qwen3_bf16(qwen3_codes16, which):
    r = qwen3_codes16
    x = r[which].reshape(-1, r["w"].d)
    _check_topk_all(x, r[which + "i"], r[which + "v"], r["w"].k, True,
                    f"qwen3_32k {which} (int16/bf16)")


@pytest.mark.parametrize("which", ["q", "k"])
def test_topk_every_row_zipf(zipf, which):
    r = zipf
    x = r[which].reshape(-1, r["w"].d)
    _check_topk_all(x, r[which + "i"], r[which + "v"], r["w"].k, False, f"zipf_128k {which}")


@pytest.mark.parametrize("name", ["tiny", "gpt2s"])
def test_topk_every_row_small(name):
    w = si.workload(name)
    q, kk, _ = _dense_inputs(w)
    for which, x in (("q", q), ("k", kk)):
        gi, gv = sfa.sfa_topk_encode(x, w.k)
        torch.cuda.synchronize()
        _check_topk_all(x.reshape(-1, w.d).cpu().numpy(), gi.cpu().numpy(), np_vals(gv), w.k,
                        False, f"{name} {which}")


# ---------------------------------------------------------------------------
# decode cache: 64 sequences x 8 KV heads x 65536 keys
# ---------------------------------------------------------------------------


@pytest.fixture(scope="module")
def decode_cache():
    w = si.workload("decode_64k")
    B, Hq, Hkv, L, d, k = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    print("[fullsize] decode_64k: building the cache on the GPU", flush=True)
    ci = torch.empty((B, Hkv, L, k), dtype=torch.int16, device=DEV)
    cv = torch.empty((B, Hkv, L, k), dtype=torch.bfloat16, device=DEV)
    vc = torch.empty((B, Hkv, L, d), dtype=torch.bfloat16, device=DEV)
    rng = np.random.default_rng(w.seed)
    picked_x, picked_i, picked_v, n_ties = [], [], [], 0
    per_slice = 2048  # random rows per (sequence, KV head): 1,048,576 in all
    for b in range(B):
        for h in range(Hkv):
            kd = si.normal((L, d), w.seed, "k", b, h, device=DEV)
            sfa.sfa_topk_encode(kd, k, idx=ci[b, h], val=cv[b, h])
            vc[b, h] = si.normal((L, d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
            # rows whose k-th and (k+1)-th largest magnitudes tie (found with
            # torch's sort of the magnitudes), plus random rows
            top = torch.topk(kd.abs(), k + 1, dim=1, sorted=True).values
            tie = torch.nonzero(top[:, k - 1] == top[:, k]).flatten()
            n_ties += int(tie.numel())
            rnd = torch.from_numpy(rng.integers(0, L, per_slice)).to(DEV)
            sel = torch.unique(torch.cat([tie, rnd]))
            picked_x.append(kd[sel].cpu().numpy())
            picked_i.append(ci[b, h][sel].cpu().numpy())
            picked_v.append(np_vals(cv[b, h][sel]))
    qd = si.normal((B, Hq, d), w.seed, "q", device=DEV)
    qi, qv = sfa.sfa_topk_encode(qd, k)
    o, lse = sfa.sfa_attn_decode(qi, qv, ci, cv, vc, scale=w.scale, o_dtype=torch.float32)
    ob16, _ = sfa.sfa_attn_decode(qi, qv, ci, cv, vc, scale=w.scale, o_dtype=torch.bfloat16,
                                  want_lse=False)
    torch.cuda.synchronize()
    res = {"w": w, "o": o.cpu(), "lse": lse.cpu(), "ob16": ob16.cpu(), "q": qd.cpu().numpy(),
           "vc": vc, "x": np.concatenate(picked_x), "gi": np.concatenate(picked_i),
           "gv": np.concatenate(picked_v), "n_ties": n_ties}
    del ci, cv, qi, qv, o, lse, ob16
    yield res
    del res["vc"]
    torch.cuda.empty_cache()


def test_decode_cache_topk_ties_and_sample(decode_cache):
    r = decode_cache
    ties = boundary_tie_rows(r["x"], r["w"].k)
    print(f"[parity] decode cache: {r['n_ties']} boundary-tie rows in the 33.5M-row cache "
          f"(found on the GPU), {ties.size} among the {r['x'].shape[0]} rows checked", flush=True)
    assert ties.size >= r["n_ties"]  # every tie row is in the checked set
    _check_topk_all(r["x"], r["gi"], r["gv"], r["w"].k, True, "decode_64k cache (int16/bf16)")


@pytest.mark.parametrize("half", [0, 1])
def test_decode_64k_every_sequence(decode_cache, half):
    r = decode_cache
    w = r["w"]
    L, d, k, G = w.n, w.d, w.k, w.G
    oqi, oqv = oracle.topk_encode(r["q"], k)
    for b in range(half * w.B // 2, (half + 1) * w.B // 2):
        g = b % w.Hkv
        kd = si.normal((L, d), w.seed, "k", b, g, device=DEV).cpu().numpy()
        oci, ocv = _oracle_codes(kd, k, bf16=True)
        kdd = oracle.densify(oci, ocv, d)
        vv = oracle.widen(np_vals(r["vc"][b, g]))
        hs = list(range(g * G, (g + 1) * G))
        qd = oracle.densify(oqi[b, hs], oqv[b, hs], d)
        res = par_map(lambda i: oracle.softmax_attention(qd[i:i + 1], kdd, vv, w.scale, False),
                      range(len(hs)))
        O = np.concatenate([x[0] for x in res])
        Ls = np.concatenate([x[1] for x in res])
        check_o(r["o"][b, hs], O, TOL_O_BF16V, f"decode O seq {b} heads {hs[0]}-{hs[-1]} (KV {g})")
        check_lse(r["lse"][b, hs], Ls, f"decode LSE seq {b} (KV {g})")
        check_o(r["ob16"][b, hs], O, TOL_O_BF16V, f"decode O bf16 output seq {b} (KV {g})")
