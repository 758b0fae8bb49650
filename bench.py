#!/usr/bin/env python3
"""Benchmark of the SFA hot path on one MI355X.

Default workload (the headline metric): Qwen3-like long-context forward,
B=1, 32 query heads over 8 KV heads, n=32768, d=128, k=16, causal, bf16 V and
output.  One step = Top-k coding of the dense fp32 Q and K
(sfa_topk_encode x2) + the fused forward (sfa_attn_fwd), with every input
already resident in HBM.  `--workload decode_64k` times the decode step
(sfa_attn_decode) over the 64-sequence x 64K sparse-code KV cache instead, and
`--pass bwd` the backward with the straight-through estimator (sfa_attn_bwd on
the workload's codes, forward O / LSE and a seeded dO).  `--workload
decode_64k --cache paged` times a serving step over a paged cache: append of
the new token (sfa_kv_append) + decode of the dense query
(sfa_attn_decode_paged), after filling the cache by appends.

Prints ONE JSON line.  Besides the contract fields it carries
  roofline      the dominant kernel's algorithmic rate (from HIP events
                around its own launches) against the MI355X peak, and HBM
                traffic from rocprofv3 counters when a matching summary
                exists under profiles/;
  cpu_baseline  the CPU oracle timed on a bounded sample of the same
                workload on this host, scaled to the metric's unit.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2603_22300_amd as sfa  # noqa: E402
import sfa_inputs as si  # noqa: E402

METRIC = "SFA fwd tokens/s at n=32K,d=128,k=16; % of HBM/MFMA roofline"
PEAK_MFMA_BF16 = 2.5e15      # dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12            # bytes/s
# the decode kernel: its launcher and the header holding the kernel template
DECODE_SRC = "sfa_decode.hip+sfa_decode_kernel.h"
DEV = "cuda"


def _src_hash(name: str) -> str:
    """sha256[:16] of a kernel source, or of several joined by '+' (a source
    and the header that holds its kernel template)."""
    h = hashlib.sha256()
    for part in name.split("+"):
        h.update(open(os.path.join(ROOT, "paper_2603_22300_amd", "csrc", part), "rb").read())
    return h.hexdigest()[:16]


def _traffic(kernel_file: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 PMC summary, if it was
    taken on the current kernel source; else None."""
    p = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(p):
        return None
    try:
        t = json.load(open(p))
    except Exception:
        return None
    if t.get("src_sha256_16") != _src_hash(kernel_file):
        return None
    return t.get("bytes_per_launch")


# ----------------------------------------------------------------------------
# forward workload
# ----------------------------------------------------------------------------

def _fwd_inputs(w):
    q = torch.empty((w.B, w.Hq, w.n, w.d), device=DEV)
    k = torch.empty((w.B, w.Hkv, w.n, w.d), device=DEV)
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
                k[b, h] = si.dense_from_codes(i_, v_, w.d)
            else:
                k[b, h] = si.normal((w.n, w.d), w.seed, "k", b, h, device=DEV)
            v[b, h] = si.normal((w.n, w.d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
    return q, k, v


def _key_ranges(n: int, causal: bool, window: int, n_global: int, device):
    """Per query position i, the keys it may see as two ranges: [lo, hi] and
    the global keys below the window, [0, glob_end)."""
    i = torch.arange(n, device=device)
    hi = i.clone() if causal else torch.full_like(i, n - 1)
    lo = torch.zeros_like(i)
    glob_end = torch.zeros_like(i)
    if window > 0:
        isg = i < n_global
        lo = torch.where(isg, lo, (i - window + 1).clamp(min=0))
        if not causal:
            hi = torch.where(isg, hi, (i + window - 1).clamp(max=n - 1))
        glob_end = torch.where(isg, glob_end, torch.minimum(torch.full_like(i, n_global), lo))
    return lo, hi, glob_end


def _allowed_pairs(n: int, causal: bool, window: int = 0, n_global: int = 0) -> int:
    lo, hi, ge = _key_ranges(n, causal, window, n_global, "cpu")
    return int((hi - lo + 1 + ge).sum().item())


def _overlap_count(qi: torch.Tensor, ki: torch.Tensor, d: int, G: int, causal: bool,
                   window: int = 0, n_global: int = 0) -> int:
    """Exact E = sum over allowed (i, j) of |S_i cap S_j| (accounting only):
    per coordinate, the number of allowed keys holding it (prefix counts over
    the key ranges), summed over the query's coordinates."""
    B, Hq, n, k = qi.shape
    lo, hi, ge = _key_ranges(n, causal, window, n_global, qi.device)
    E = 0
    for b in range(B):
        for g in range(ki.shape[1]):
            km = torch.zeros((n, d), dtype=torch.int32, device=qi.device)
            km.scatter_(1, ki[b, g].long(), 1)
            kc = torch.cat([torch.zeros((1, d), dtype=torch.int32, device=qi.device),
                            torch.cumsum(km, 0, dtype=torch.int32)])  # kc[j] = keys < j
            cnt = kc[hi + 1] - kc[lo] + kc[ge]
            for h in range(g * G, (g + 1) * G):
                E += int(torch.gather(cnt, 1, qi[b, h].long()).sum().item())
    return E


def bench_fwd(w, steps, warmup, want_cpu, window=0, n_global=0, codes="i32f32", fwd="default"):
    q, k, v = _fwd_inputs(w)
    B, Hq, Hkv, n, d, kk = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    idt, vdt = FWD_CODE_FORMATS[codes]
    qi = torch.empty((B, Hq, n, kk), dtype=idt, device=DEV)
    qv = torch.empty((B, Hq, n, kk), dtype=vdt, device=DEV)
    ki = torch.empty((B, Hkv, n, kk), dtype=idt, device=DEV)
    kv = torch.empty((B, Hkv, n, kk), dtype=vdt, device=DEV)
    o = torch.empty((B, Hq, n, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((B, Hq, n), dtype=torch.float32, device=DEV)
    ws = torch.empty(sfa.sfa_attn_fwd_workspace(B, Hkv, n, d, v.dtype), dtype=torch.uint8, device=DEV)

    def step(ev=None):
        if ev is not None:
            ev[2].record()
        sfa.sfa_topk_encode(q, kk, idx=qi, val=qv)
        sfa.sfa_topk_encode(k, kk, idx=ki, val=kv)
        if ev is not None:
            ev[0].record()
        if fwd == "index":
            sfa.sfa_attn_fwd_index(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale, o=o, lse=lse)
        else:
            sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale, o=o, lse=lse,
                             ws=ws, window=window, n_global=n_global)
        if ev is not None:
            ev[1].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record()
    for s in range(steps):
        step(evs[s])
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / steps
    fwd_ms = [e[0].elapsed_time(e[1]) for e in evs]
    fwd_avg = float(np.mean(fwd_ms))
    enc_avg = float(np.mean([e[2].elapsed_time(e[0]) for e in evs]))
    step_ms = [e[2].elapsed_time(e[1]) for e in evs]

    pairs = B * Hq * _allowed_pairs(n, w.causal, window, n_global)
    pv_flops = 2.0 * d * pairs          # P.V: 2 d flops per allowed pair
    E = _overlap_count(qi, ki, d, w.G, w.causal, window, n_global)
    algo_flops = pv_flops + 2.0 * E     # + one multiply-add per overlapping coordinate
    achieved = algo_flops / (fwd_avg * 1e-3)
    tokens = B * n
    metric = METRIC if window == 0 else METRIC + f"; sliding window {window} + {n_global} global tokens"
    if kk != 16 and w.name == "qwen3_32k":
        metric = metric.replace("k=16", f"k={kk}")
    if n != 32768 and w.name == "qwen3_32k":
        metric = metric.replace("n=32K", f"n={n}")
    if fwd == "index":
        metric += "; inverted-index forward (sfa_attn_fwd_index)"
    if codes != "i32f32":
        metric += f"; codes stored as {_CODE_NAMES[codes]}"
        precision = (f"codes {_CODE_NAMES[codes]}; scores fp32 (one exact {vdt_name(vdt)} MFMA product "
                     "per coordinate block, scale applied in fp32); softmax fp32; P.V fp16 MFMA on V "
                     "converted exactly to fp16, fp32 accumulate; O bf16")
    else:
        precision = ("codes fp32; scores fp32 (three products of float16 pieces on MFMA, ~3*2^-22 "
                     "relative); softmax fp32; P.V fp16 MFMA on V converted exactly to fp16, fp32 "
                     "accumulate; O bf16")
    hbm = _fwd_bytes(w, idt, vdt)
    out = {
        "metric": metric,
        "value": tokens / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name, "B": B, "Hq": Hq, "Hkv": Hkv, "n": n, "d": d, "k": kk,
            "causal": w.causal, "seed": w.seed, "window": window, "n_global": n_global,
            "step": "sfa_topk_encode(Q) + sfa_topk_encode(K) + sfa_attn_fwd",
            "codes": codes,
            "precision": precision,
        },
        "roofline": {
            "kernel": "sfa_fwd_index_kernel" if fwd == "index" else "sfa_fwd_kernel",
            "bound": "mfma",
            "achieved": achieved / 1e12,
            "peak": PEAK_MFMA_BF16 / 1e12,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_MFMA_BF16,
            # the committed counter summary is of the fp32-code forward
            "traffic": (_traffic("sfa_fwd.hip", w.name)
                        if codes == "i32f32" and window == 0 and fwd == "default" and kk == 16
                        else None),
            "algorithmic_flops_per_launch": algo_flops,
            "pv_flops_per_launch": pv_flops,
            "fwd_ms_avg": fwd_avg,
            "fwd_ms_min": float(np.min(fwd_ms)),
            "allowed_pairs": pairs,
            "overlap_products_E": E,
            "algorithmic_hbm_bytes_per_launch": hbm,
            "hbm_frac": hbm / (fwd_avg * 1e-3) / PEAK_HBM,
        },
        # the two parts of the step: encoding Q and K, and the forward on
        # codes already in HBM
        "split": {
            "encode_ms": enc_avg,
            "encode_rows_per_s": B * (Hq + Hkv) * n / (enc_avg * 1e-3),
            "fwd_ms": fwd_avg,
            "fwd_tokens_per_s": tokens / (fwd_avg * 1e-3),
        },
        # per-step distribution (each step bracketed by its own events)
        "timing": {"step": _pstats(step_ms), "fwd_call": _pstats(fwd_ms)},
        "wall_s_timed": wall,
    }
    if want_cpu and window == 0 and codes == "i32f32" and fwd == "default":
        out["cpu_baseline"] = cpu_baseline_fwd(w, q, k, v)
    return out


def bench_bwd(w, steps, warmup, want_cpu, window=0, n_global=0, codes="i32f32"):
    """One step = sfa_attn_bwd (codes, O, LSE and dO resident in HBM)."""
    q, k, v = _fwd_inputs(w)
    B, Hq, Hkv, n, d, kk = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    idt, vdt = FWD_CODE_FORMATS[codes]
    qi, qv = sfa.sfa_topk_encode(q, kk, idx_dtype=idt, val_dtype=vdt)
    ki, kv = sfa.sfa_topk_encode(k, kk, idx_dtype=idt, val_dtype=vdt)
    o, lse = sfa.sfa_attn_fwd(qi, qv, ki, kv, v, causal=w.causal, scale=w.scale,
                              o_dtype=torch.bfloat16, window=window, n_global=n_global)
    dout = torch.empty((B, Hq, n, d), dtype=torch.bfloat16, device=DEV)
    for b in range(B):
        for h in range(Hq):
            dout[b, h] = si.normal((n, d), w.seed, "dout", b, h, device=DEV).to(torch.bfloat16)
    dq = torch.empty((B, Hq, n, kk), dtype=torch.float32, device=DEV)
    dk = torch.empty((B, Hkv, n, kk), dtype=torch.float32, device=DEV)
    dv = torch.empty((B, Hkv, n, d), dtype=torch.float32, device=DEV)
    ws = torch.empty(sfa.sfa_attn_bwd_workspace(B, Hq, Hkv, n, d), dtype=torch.uint8, device=DEV)

    def step():
        sfa.sfa_attn_bwd(qi, qv, ki, kv, v, o, lse, dout, causal=w.causal, scale=w.scale,
                         dq=dq, dk=dk, dv=dv, ws=ws, window=window, n_global=n_global)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    wall0 = time.perf_counter()
    for s_ in range(steps):
        evs[s_][0].record()
        step()
        evs[s_][1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = [a.elapsed_time(b_) for a, b_ in evs]
    ms_step = float(np.mean(ms))
    pairs = B * Hq * _allowed_pairs(n, w.causal, window, n_global)
    E = _overlap_count(qi, ki, d, w.G, w.causal, window, n_global)
    # dV and dP: 2d flops per allowed pair each; S, dq~ and dk~ on the
    # supports: 2 flops per shared coordinate each
    algo = 4.0 * d * pairs + 6.0 * E
    out = {
        "metric": "SFA bwd (straight-through estimator) tokens/s at n=32K,d=128,k=16" +
                  (f"; sliding window {window} + {n_global} global tokens" if window else "") +
                  (f"; codes stored as {_CODE_NAMES[codes]}" if codes != "i32f32" else ""),
        "value": B * n / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name, "B": B, "Hq": Hq, "Hkv": Hkv, "n": n, "d": d, "k": kk,
            "causal": w.causal, "seed": w.seed, "window": window, "n_global": n_global,
            "step": "sfa_attn_bwd",
            "codes": codes,
            "precision": "O and dO bf16; products on MFMA with bf16 hi/lo pieces (3 terms; "
                         "pieces that are zero, as for bf16 values, left out), fp32 accumulate; "
                         "gradients fp32",
        },
        "roofline": {
            "kernel": "sfa_bwd_dq_kernel + sfa_bwd_dkv_kernel (+ tile images)",
            "bound": "mfma",
            "achieved": algo / (ms_step * 1e-3) / 1e12,
            "peak": PEAK_MFMA_BF16 / 1e12,
            "unit": "TFLOP/s",
            "frac": algo / (ms_step * 1e-3) / PEAK_MFMA_BF16,
            "traffic": (_traffic("sfa_bwd.hip", f"bwd_{w.name}")
                        if codes == "i32f32" and window == 0 else None),
            "algorithmic_flops_per_launch": algo,
            "allowed_pairs": pairs,
            "overlap_products_E": E,
            "ms_min": float(np.min(ms)),
        },
        "timing": {"step": _pstats(ms)},
        "wall_s_timed": wall,
    }
    if want_cpu and window == 0 and codes == "i32f32":
        out["cpu_baseline"] = cpu_baseline_bwd(w, q, k, v, dout)
    return out


def cpu_baseline_bwd(w, q, k, v, dout, n_sub=3072):
    """The oracle backward (oracle.attn_bwd, float64) on the first n_sub
    positions of one KV head group -- a causal prefix is a sub-problem of the
    same workload -- scaled by the ratio of allowed pairs."""
    import oracle
    G = w.G
    sl = slice(0, n_sub)
    qn = q[:1, :G, sl].cpu().numpy()
    kn = k[:1, :1, sl].cpu().numpy()
    vn = v[:1, :1, sl].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    dn = dout[:1, :G, sl].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    t = time.perf_counter()
    qi, qv = oracle.topk_encode(qn, w.k)
    ki, kv = oracle.topk_encode(kn, w.k)
    oracle.attn_bwd(qi, qv, ki, kv, vn, dn, w.d, w.scale, w.causal)
    dt = time.perf_counter() - t
    sub_pairs = G * (n_sub * (n_sub + 1) // 2 if w.causal else n_sub * n_sub)
    all_pairs = w.B * w.Hq * (w.n * (w.n + 1) // 2 if w.causal else w.n * w.n)
    total = dt * all_pairs / sub_pairs
    return {
        "value": w.B * w.n / total,
        "unit": "tokens/s",
        "cores": _blas_threads(),
        "kind": "oracle",
        "sample": (f"{w.name}: oracle backward (codes, softmax, chain rule in float64) of the "
                   f"first {n_sub} positions of one KV head group ({G} query heads), {dt:.1f} s, "
                   f"scaled x{all_pairs / sub_pairs:.0f} by allowed pairs; extrapolated step "
                   f"{total:.0f} s"),
        "host_cpu_count": os.cpu_count(),
    }


def _fwd_bytes(w, idt=torch.int32, vdt=torch.float32):
    """Compulsory HBM bytes of one forward launch: codes in (index + value
    bytes per entry; int32 + fp32 by default), V in (bf16), O out (bf16), LSE
    out (fp32)."""
    entry = torch.empty((), dtype=idt).element_size() + torch.empty((), dtype=vdt).element_size()
    codes = (w.B * w.Hq * w.n + w.B * w.Hkv * w.n) * w.k * entry
    return codes + w.B * w.Hkv * w.n * w.d * 2 + w.B * w.Hq * w.n * w.d * 2 + w.B * w.Hq * w.n * 4


def _pstats(ms) -> dict:
    """Median, 10th and 90th percentile of per-step times (ms)."""
    a = np.asarray(ms, dtype=np.float64)
    return {"median_ms": float(np.median(a)), "p10_ms": float(np.percentile(a, 10)),
            "p90_ms": float(np.percentile(a, 90)), "mean_ms": float(a.mean()), "n": int(a.size)}


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        return 1


def cpu_baseline_fwd(w, q, k, v, budget_rows=1536, seed=0):
    """The oracle on a bounded sample of the same workload, extrapolated to
    the whole step: Top-k of every key row (timed in full), Top-k of a sample
    of query rows (scaled by the row count), and the attention of `budget_rows`
    random positions for every query head (scaled by the causal row cost,
    proportional to i+1)."""
    import oracle
    rng = np.random.default_rng(seed)
    # key coding, every key row
    kn = k.cpu().numpy()
    t = time.perf_counter()
    kc = [[oracle.topk_encode(kn[b, g], w.k) for g in range(w.Hkv)] for b in range(w.B)]
    t_enck = time.perf_counter() - t
    # query coding, sampled rows
    rows = np.sort(rng.choice(w.n, size=budget_rows, replace=False))
    qs = q[:, :, torch.from_numpy(rows).to(q.device)].cpu().numpy()   # [B,Hq,R,d]
    t = time.perf_counter()
    qc = oracle.topk_encode(qs, w.k)
    t_encq = (time.perf_counter() - t) * (w.n / budget_rows)
    # attention on the sampled rows, all heads
    vn = v.view(torch.int16).cpu().numpy().view(np.uint16)
    t = time.perf_counter()
    for b in range(w.B):
        for h in range(w.Hq):
            g = h // w.G
            qi_full = np.zeros((w.n, w.k), np.int64)
            qv_full = np.zeros((w.n, w.k), np.float32)
            qi_full[rows], qv_full[rows] = qc[0][b, h], qc[1][b, h]
            oracle.attn_fwd_rows(qi_full, qv_full, kc[b][g][0], kc[b][g][1], vn[b, g], w.d,
                                 w.scale, w.causal, rows)
    t_att = time.perf_counter() - t
    if w.causal:
        scale_rows = (w.n * (w.n + 1) / 2) / float(np.sum(rows + 1))
    else:
        scale_rows = w.n / budget_rows
    total = t_enck + t_encq + t_att * scale_rows
    return {
        "value": w.B * w.n / total,
        "unit": "tokens/s",
        "cores": _blas_threads(),
        "kind": "oracle",
        "sample": (f"{w.name}: oracle Top-k of all {w.B * w.Hkv * w.n} key rows ({t_enck:.1f} s), "
                   f"of {budget_rows} query rows x {w.Hq} heads (x{w.n / budget_rows:.0f}), "
                   f"float64 attention of those {budget_rows} random positions x {w.Hq} heads "
                   f"({t_att:.1f} s, scaled x{scale_rows:.1f} by the causal row cost i+1); "
                   f"extrapolated step {total:.0f} s"),
        "host_cpu_count": os.cpu_count(),
    }


# ----------------------------------------------------------------------------
# decode workload
# ----------------------------------------------------------------------------

CODE_FORMATS = {"i16bf16": (torch.int16, torch.bfloat16), "u8f16": (torch.uint8, torch.float16)}
FWD_CODE_FORMATS = dict(CODE_FORMATS, i32f32=(torch.int32, torch.float32))
_CODE_NAMES = {"i16bf16": "int16/bf16", "u8f16": "uint8/float16", "i32f32": "int32/float32"}


def vdt_name(vdt) -> str:
    return {torch.bfloat16: "bf16", torch.float16: "float16"}.get(vdt, str(vdt))


def _decode_keys(L: int, window: int, n_global: int) -> int:
    """Keys the decode query (position L - 1) may see."""
    if window <= 0 or L - 1 < n_global:
        return L
    lo = max(0, L - window)
    return (L - lo) + min(n_global, lo)


def bench_decode(w, steps, warmup, want_cpu, codes="i16bf16", window=0, n_global=0):
    B, Hq, Hkv, L, d, kk = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    idt, vdt = CODE_FORMATS[codes]
    cbytes = kk * (idt.itemsize + vdt.itemsize)  # cache code bytes per key
    ci = torch.empty((B, Hkv, L, kk), dtype=idt, device=DEV)
    cv = torch.empty((B, Hkv, L, kk), dtype=vdt, device=DEV)
    vc = torch.empty((B, Hkv, L, d), dtype=torch.bfloat16, device=DEV)
    for b in range(B):
        for h in range(Hkv):
            kd = si.normal((L, d), w.seed, "k", b, h, device=DEV)
            sfa.sfa_topk_encode(kd, kk, idx=ci[b, h], val=cv[b, h])
            vc[b, h] = si.normal((L, d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
    del kd
    qd = si.normal((B, Hq, d), w.seed, "q", device=DEV)
    qi, qv = sfa.sfa_topk_encode(qd, kk)
    o = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=DEV)
    ws = torch.empty(sfa.sfa_attn_decode_workspace(B, Hq, L, d), dtype=torch.uint8, device=DEV)

    def step():
        sfa.sfa_attn_decode(qi, qv, ci, cv, vc, scale=w.scale, o=o, lse=lse, ws=ws, window=window,
                            n_global=n_global)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    t0.record()
    for s_ in range(steps):
        evs[s_][0].record()
        step()
        evs[s_][1].record()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    step_ms = [a.elapsed_time(b_) for a, b_ in evs]
    algo_bytes = B * Hkv * _decode_keys(L, window, n_global) * (cbytes + d * 2) + \
        B * Hq * (kk * 8 + d * 2 + 4)
    achieved = algo_bytes / (ms * 1e-3)
    out = {
        "metric": f"SFA decode tokens/s, 64 seqs x 64K sparse-code cache (k=16 {_CODE_NAMES[codes]}, "
                  "d=128), 32/8 heads",
        "value": B / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "B": B, "Hq": Hq, "Hkv": Hkv, "L": L, "d": d, "k": kk,
                   "cache_codes": codes, "window": window, "n_global": n_global,
                   "step": "sfa_attn_decode (split context + LSE merge)"},
        "roofline": {"kernel": "sfa_decode_kernel + combine", "bound": "hbm",
                     "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM, "traffic": _traffic(DECODE_SRC, w.name),
                     "algorithmic_bytes_per_launch": algo_bytes},
        "timing": {"step": _pstats(step_ms)},
    }
    return out


def bench_decode_q8(w, steps, warmup, window=0, n_global=0):
    """Decode step over the 8-bit cache of SFA (quant): int16 indices, int8
    code values and int8 value rows with a float32 scale per row, filled by
    sfa_kv_append_q8 from the same dense keys and values as the bf16 cache."""
    B, Hq, Hkv, L, d, kk = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    ci = torch.empty((B, Hkv, L, kk), dtype=torch.int16, device=DEV)
    cv = torch.empty((B, Hkv, L, kk), dtype=torch.int8, device=DEV)
    cs = torch.empty((B, Hkv, L), dtype=torch.float32, device=DEV)
    vc = torch.empty((B, Hkv, L, d), dtype=torch.int8, device=DEV)
    vs = torch.empty((B, Hkv, L), dtype=torch.float32, device=DEV)
    kb = torch.empty((1, Hkv, L, d), device=DEV)
    vb = torch.empty((1, Hkv, L, d), device=DEV, dtype=torch.bfloat16)
    zero = torch.zeros(1, dtype=torch.int32, device=DEV)
    app_ms = 0.0
    for b in range(B):
        for h in range(Hkv):
            kb[0, h] = si.normal((L, d), w.seed, "k", b, h, device=DEV)
            vb[0, h] = si.normal((L, d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
        zero.zero_()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        sfa.sfa_kv_append_q8(kb, vb, zero, ci[b:b + 1], cv[b:b + 1], cs[b:b + 1], vc[b:b + 1],
                             vs[b:b + 1], k=kk)
        e1.record()
        torch.cuda.synchronize()
        if b > 0:
            app_ms += e0.elapsed_time(e1)
    del kb, vb
    qd = si.normal((B, Hq, d), w.seed, "q", device=DEV)
    qi, qv = sfa.sfa_topk_encode(qd, kk)
    o = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=DEV)
    ws = torch.empty(sfa.sfa_attn_decode_workspace(B, Hq, L, d), dtype=torch.uint8, device=DEV)

    def step():
        sfa.sfa_attn_decode_q8(ci, cv, cs, vc, vs, q_idx=qi, q_val=qv, scale=w.scale, o=o,
                               lse=lse, ws=ws, window=window, n_global=n_global)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    t0.record()
    for s_ in range(steps):
        evs[s_][0].record()
        step()
        evs[s_][1].record()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    step_ms = [a.elapsed_time(b_) for a, b_ in evs]
    key_bytes = kk * 2 + kk + 4 + d + 4  # int16 indices, int8 values, scale, int8 V, scale
    algo_bytes = B * Hkv * _decode_keys(L, window, n_global) * key_bytes + \
        B * Hq * (kk * 8 + d * 2 + 4)
    achieved = algo_bytes / (ms * 1e-3)
    app_bytes = Hkv * L * (d * 4 + d * 2 + key_bytes)
    return {
        "metric": "SFA decode tokens/s, 64 seqs x 64K 8-bit cache (SFA (quant): k=16 int16 "
                  "indices + int8 values, int8 V, float32 scale per row; d=128), 32/8 heads",
        "value": B / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int8", "data": "synthetic",
        "config": {"workload": w.name + "_q8", "B": B, "Hq": Hq, "Hkv": Hkv, "L": L, "d": d,
                   "k": kk, "cache": "int16 idx + int8 values + int8 V, float32 scale per row",
                   "window": window, "n_global": n_global,
                   "step": "sfa_attn_decode_q8 (split context + LSE merge)"},
        "roofline": {"kernel": "sfa_decode_kernel (8-bit) + combine", "bound": "hbm",
                     "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM, "traffic": None,
                     "algorithmic_bytes_per_launch": algo_bytes,
                     "bytes_per_cached_key": key_bytes},
        "append_prefill": {"kernel": "sfa_kv_append_kernel (8-bit)", "tokens_per_call": L,
                           "ms_per_call": app_ms / (B - 1), "bytes_per_call": app_bytes,
                           "achieved_GBps": app_bytes / (app_ms / (B - 1) * 1e-3) / 1e9},
        "timing": {"step": _pstats(step_ms)},
    }


def bench_decode_paged(w, steps, warmup, codes="i16bf16"):
    """Serving step over a paged cache: append each sequence's new key (coded on
    append) and value, then decode the new dense query (coded inside the decode
    kernel) over the grown cache.  The cache is first filled by sfa_kv_append,
    one 64K-token prefill per sequence, which is timed as the append rate."""
    B, Hq, Hkv, L, d, kk = w.B, w.Hq, w.Hkv, w.n, w.d, w.k
    P = 256
    if warmup + steps > P:
        raise SystemExit("--cache paged grows each sequence by one token per step: "
                         f"warmup + steps must be <= {P}")
    max_pages = L // P + 1  # one spare page per sequence for the generated tokens
    num_pages = B * max_pages
    g = torch.Generator(device="cpu")
    g.manual_seed(si.slice_seed(w.seed, "block_table"))
    table = torch.randperm(num_pages, generator=g).reshape(B, max_pages).to(torch.int32).to(DEV)
    idt, vdt = CODE_FORMATS[codes]
    cbytes = kk * (idt.itemsize + vdt.itemsize)  # cache code bytes per key
    ci = torch.empty((num_pages, Hkv, P, kk), dtype=idt, device=DEV)
    cv = torch.empty((num_pages, Hkv, P, kk), dtype=vdt, device=DEV)
    vc = torch.empty((num_pages, Hkv, P, d), dtype=torch.bfloat16, device=DEV)
    lens = torch.zeros(B, dtype=torch.int32, device=DEV)
    kb = torch.empty((1, Hkv, L, d), device=DEV)
    vb = torch.empty((1, Hkv, L, d), device=DEV, dtype=torch.bfloat16)
    app_ms = 0.0
    for b in range(B):
        for h in range(Hkv):
            kb[0, h] = si.normal((L, d), w.seed, "k", b, h, device=DEV)
            vb[0, h] = si.normal((L, d), w.seed, "v", b, h, device=DEV).to(torch.bfloat16)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        sfa.sfa_kv_append(kb, vb, lens[b:b + 1], ci, cv, vc, k=kk, block_table=table[b:b + 1])
        e1.record()
        torch.cuda.synchronize()
        if b > 0:  # the first call pays the module load
            app_ms += e0.elapsed_time(e1)
    del kb, vb
    app_bytes = Hkv * L * (d * 4 + d * 2 + cbytes + d * 2)  # per prefill call
    app_rate = app_bytes / (app_ms / (B - 1) * 1e-3)
    # per-step inputs: one new token per sequence, the new dense queries
    kn = si.normal((B, Hkv, 1, d), w.seed, "k_step", device=DEV)
    vn = si.normal((B, Hkv, 1, d), w.seed, "v_step", device=DEV).to(torch.bfloat16)
    qd = si.normal((B, Hq, d), w.seed, "q", device=DEV)
    o = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=DEV)
    ws = torch.empty(sfa.sfa_attn_decode_workspace(B, Hq, max_pages * P, d), dtype=torch.uint8,
                     device=DEV)

    def step(ev=None):
        sfa.sfa_kv_append(kn, vn, lens, ci, cv, vc, k=kk, block_table=table)
        if ev is not None:
            ev[0].record()
        sfa.sfa_attn_decode_paged(ci, cv, vc, table, seq_len=lens, q=qd, scale=w.scale, o=o,
                                  lse=lse, ws=ws)
        if ev is not None:
            ev[1].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for s_ in range(steps):
        step(evs[s_])
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    dec_list = [a.elapsed_time(b) for a, b in evs]
    dec_ms = sum(dec_list) / steps
    ctx = L + warmup + (steps + 1) / 2.0  # mean context length over the timed steps
    dec_bytes = B * Hkv * ctx * (cbytes + d * 2) + B * Hq * (d * 4 + d * 2 + 4)
    achieved = dec_bytes / (dec_ms * 1e-3)
    return {
        "metric": f"SFA decode tokens/s, 64 seqs x 64K sparse-code cache (k=16 {_CODE_NAMES[codes]}, "
                  "d=128), 32/8 heads",
        "value": B / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name + "_paged", "B": B, "Hq": Hq, "Hkv": Hkv, "L": L, "d": d,
                   "k": kk, "page_size": P, "cache_codes": codes,
                   "step": "sfa_kv_append (new token) + sfa_attn_decode_paged (dense query "
                           "coded in-kernel, split context + LSE merge)"},
        "roofline": {"kernel": "sfa_decode_kernel (paged) + combine", "bound": "hbm",
                     "achieved": achieved / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM, "traffic": None,
                     "algorithmic_bytes_per_launch": dec_bytes, "ms_per_launch": dec_ms},
        "append_prefill": {"kernel": "sfa_kv_append_kernel", "tokens_per_call": L,
                           "ms_per_call": app_ms / (B - 1), "bytes_per_call": app_bytes,
                           "achieved_GBps": app_rate / 1e9, "frac": app_rate / PEAK_HBM},
        "timing": {"decode_call": _pstats(dec_list)},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen3_32k", choices=sorted(si.WORKLOADS))
    ap.add_argument("--pass", dest="which", default="fwd", choices=["fwd", "bwd"],
                    help="forward (default, the headline metric) or the backward")
    ap.add_argument("--cache", default="contiguous", choices=["contiguous", "paged"],
                    help="decode workloads: contiguous cache (decode only) or paged cache "
                         "(append of the new token + decode with in-kernel query coding)")
    ap.add_argument("--codes", default=None, choices=sorted(FWD_CODE_FORMATS) + ["q8"],
                    help="code storage: int32 indices + fp32 values (forward default), int16 + "
                         "bf16 (decode default), or the paper's compact uint8 + float16; decode "
                         "takes the two 16-bit formats, and q8: the 8-bit cache of SFA (quant)")
    ap.add_argument("--window", type=int, default=0,
                    help="token sparsity composed with SFA: sliding window (0: none)")
    ap.add_argument("--n-global", type=int, default=0,
                    help="leading global tokens with --window")
    ap.add_argument("--k", type=int, default=0,
                    help="forward workloads: nonzeros per code other than the workload's")
    ap.add_argument("--n", type=int, default=0,
                    help="forward workloads: sequence length other than the workload's")
    ap.add_argument("--fwd", default="default", choices=["default", "index"],
                    help="forward entry point: sfa_attn_fwd, or the inverted-index forward")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run a plain 1 GiB device copy twice (reference for "
                         "the FETCH_SIZE / WRITE_SIZE counters of a profiling run)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the SFA hot path here is built and measured "
              "on a single MI355X (no multi-GPU path); rerun with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    w = si.workload(args.workload)
    if args.k:
        if w.kind != "fwd" or not 1 <= args.k <= w.d:
            print("--k applies to forward workloads, 1 <= k <= d", file=sys.stderr)
            sys.exit(2)
        w = dataclasses.replace(w, k=args.k)
    if args.n:
        if w.kind != "fwd" or args.n < 1:
            print("--n applies to forward workloads, n >= 1", file=sys.stderr)
            sys.exit(2)
        w = dataclasses.replace(w, n=args.n)
    codes = args.codes or ("i16bf16" if w.kind == "decode" else "i32f32")
    if codes == "q8" and w.kind != "decode":
        print("--codes q8 (the 8-bit cache) is a decode format", file=sys.stderr)
        sys.exit(2)
    if w.kind == "decode" and codes not in CODE_FORMATS and codes != "q8":
        print(f"--codes {codes} is not measured for this workload / pass", file=sys.stderr)
        sys.exit(2)
    if codes == "q8":
        out = bench_decode_q8(w, args.steps, args.warmup, args.window, args.n_global)
    elif w.kind == "decode" and args.cache == "paged":
        out = bench_decode_paged(w, args.steps, args.warmup, codes)
    elif w.kind == "decode":
        out = bench_decode(w, args.steps, args.warmup, not args.no_cpu_baseline, codes,
                           args.window, args.n_global)
    elif args.which == "bwd":
        out = bench_bwd(w, args.steps, args.warmup, not args.no_cpu_baseline, args.window,
                        args.n_global, codes)
    else:
        out = bench_fwd(w, args.steps, args.warmup, not args.no_cpu_baseline, args.window,
                        args.n_global, codes, args.fwd)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device=DEV)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = src.numel() * 4
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
