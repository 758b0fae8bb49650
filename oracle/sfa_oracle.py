"""CPU oracle for Sparse Feature Attention (SFA) -- TEST INFRASTRUCTURE ONLY.

Only `tests/`, `__graft_entry__.smoke()` and the `cpu_baseline` leg of
`bench.py` may import or call this module.  The product (the HIP library and
its Python binding) never does, and shares no code with it.

Everything here is the plain definition of what the method computes, written
out in float64 with numpy:

* Top-k coding of a row (Sec. 3.1, Eqs. (3)-(4)):
  keep the k entries of largest magnitude, zero the rest.  The paper leaves
  ties open; this oracle orders by larger |x| first, then lower index, and
  lists the kept pairs by ascending index.
* Sparse scores (Sec. 3.1, Eq. (5)): s_ij = scale * sum over
  coordinates shared by the supports of q_i and k_j of q_iu * k_ju.  On the
  densified codes this is exactly the dense product Q~ K~^T (Sec. 3.1:
  "S = Q~ K~^T"), which is what is computed here.
* Softmax and value aggregation (Sec. 2, Eqs. (1)-(2); Sec. 3.2: the
  tiled result equals softmax(Q~ K~^T / sqrt(d)) V).  Allowed keys under the
  causal mask are j <= i; an allowed key whose support does not overlap the
  query's still enters the softmax with score 0.
* LSE_i = m_i + ln(l_i), natural log (the paper does not define it; this is
  the standard log-sum-exp of the row's scaled scores).
* Decode (App. B, KV-cache latency): one query row against all cached keys.
* Composition with token sparsity (App. E: Longformer, SnapKV and others
  combined with SFA): the causal mask and'ed with a sliding window plus
  leading global tokens, in the forward and in decode.
* KV-cache maintenance: coded keys and their values appended at a
  sequence's next positions, in a contiguous or paged cache (a block table
  maps each run of page_size positions of a sequence to a page of the
  pool), and decode reading each position through that map.
* Backward with the straight-through estimator (Sec. 3.1, Eq. (6)): the
  chain rule of softmax attention on the densified codes, with the gradient
  of a query or key coordinate equal to that of its code value on the
  support and zero elsewhere, i.e. the dense gradient read at the code's
  coordinates.
* bf16 and binary16 storage of code values (round to nearest, ties to even)
  for the KV-cache codes and the compact format of App. J (8-bit indices,
  fp16 values), and CSR rows of variable length (Sec. 2 sparse formats)
  brought to fixed width.
* The 8-bit cache of "SFA (quant)" (App. E: SFA with 8-bit activations):
  symmetric per-row int8 codes with a float32 scale per row, for the key
  codes' values and the value rows; attention reads their values q * s.

Parity pins for every function live in tests/test_oracle_*.py.
"""
from __future__ import annotations

import numpy as np

# --------------------------------------------------------------------------
# value widening (exact)
# --------------------------------------------------------------------------


def widen(a) -> np.ndarray:
    """Exact float64 copy of stored values.

    float32 / float64 arrays widen as usual; uint16 arrays are taken as
    bfloat16 bit patterns (sign, 8 exponent bits, 7 mantissa bits), whose
    value is that of the float32 with the same high 16 bits; float16 arrays
    are binary16 values, widened from their bits by definition."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if a.dtype == np.float16:
        return widen_f16(a.view(np.uint16))
    return a.astype(np.float64)


# --------------------------------------------------------------------------
# Top-k coding, Sec. 3.1 Eqs. (3)-(4)
# --------------------------------------------------------------------------


def topk_select(x: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k kept coordinates of each row of x [..., d], ascending.

    A coordinate u outranks w when |x_u| > |x_w|, or |x_u| == |x_w| and u < w.
    The k highest-ranked coordinates are kept.  Magnitudes are compared
    exactly (float64 of the float32 values; subnormals are not flushed)."""
    x = np.asarray(x)
    d = x.shape[-1]
    if not (1 <= k <= d):
        raise ValueError("need 1 <= k <= d")
    flat = x.reshape(-1, d)
    mag = np.abs(flat.astype(np.float64))
    u = np.broadcast_to(np.arange(d), flat.shape)
    # lexsort: last key is primary -> magnitude descending, then index ascending
    order = np.lexsort((u, -mag), axis=-1)
    kept = np.sort(order[:, :k], axis=-1)
    return kept.reshape(x.shape[:-1] + (k,)).astype(np.int64)


def topk_encode(x: np.ndarray, k: int):
    """(idx int64 [..., k], val float32 [..., k]): the kept coordinates of each
    row, ascending, with the row's float32 values copied bit for bit."""
    x = np.asarray(x, dtype=np.float32)
    idx = topk_select(x, k)
    val = np.take_along_axis(x, idx, axis=-1)
    return idx, val


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values, rounded to nearest with
    ties to even -- written from the definition: of the two bfloat16 values
    that bracket x (the truncation toward zero and the next one away from
    zero), take the nearer; on a tie take the one whose last mantissa bit is
    0.  Finite inputs only; values beyond the largest bfloat16 round to inf."""
    x = np.asarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    trunc = (bits >> 16).astype(np.uint32)          # toward zero
    up = trunc + 1                                   # next one away from zero
    lo_v = widen((trunc & 0xFFFF).astype(np.uint16))
    up_v = widen((up & 0xFFFF).astype(np.uint16))
    # IEEE rounding treats the exponent range as unbounded and overflows to
    # inf afterwards: the neighbour above the largest finite bfloat16 is 2^128.
    past_max = (up & 0x7FFF) == 0x7F80
    up_v = np.where(past_max, np.where((trunc & 0x8000) != 0, -2.0**128, 2.0**128), up_v)
    xv = x.astype(np.float64)
    d_lo = np.abs(xv - lo_v)
    d_up = np.abs(up_v - xv)
    take_up = (d_up < d_lo) | ((d_up == d_lo) & ((trunc & 1) == 1))
    out = np.where(take_up, up, trunc).astype(np.uint16)
    return out


def f16_rne(x: np.ndarray) -> np.ndarray:
    """IEEE binary16 bit patterns (uint16) of float32 values, rounded to nearest
    with ties to even -- written from the definition.  binary16 has a 10-bit
    fraction, exponents -14..15 for normal numbers and subnormals in steps of
    2^-24.  Of the two representable values that bracket x, take the nearer; on
    a tie the one whose last fraction bit is 0.  Magnitudes from
    65504 + 16 (half an ulp past the largest finite value) on round to inf.
    Finite inputs only."""
    x = np.asarray(x, dtype=np.float32)
    xv = np.abs(x.astype(np.float64))
    sign = (x.view(np.uint32) >> 31).astype(np.uint16) << 15
    # spacing of binary16 values at |x|: 2^(e - 10) for e = floor(log2|x|) >= -14,
    # else the subnormal step 2^-24
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(xv > 0, xv, 1.0)))
    e = np.maximum(e, -14.0)
    step = np.exp2(e - 10)
    lo = np.floor(xv / step) * step                  # exact: both are powers of two times integers
    hi = lo + step
    d_lo, d_hi = xv - lo, hi - xv
    lo_units = np.round(lo / step).astype(np.int64)  # last fraction bit parity
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (lo_units % 2 == 1))
    mag = np.where(take_hi, hi, lo)
    # encode the magnitude: subnormal (mag < 2^-14) or normal
    sub = mag < 2.0**-14
    frac_sub = np.round(mag / 2.0**-24).astype(np.int64)
    with np.errstate(divide="ignore"):
        em = np.floor(np.log2(np.where(mag > 0, mag, 1.0)))
    frac_n = np.round((mag / np.exp2(em) - 1.0) * 1024).astype(np.int64)
    bits_n = ((em + 15).astype(np.int64) << 10) | frac_n
    bits = np.where(sub, frac_sub, bits_n)
    bits = np.where(mag > 65504.0, 0x7C00, bits)     # overflow to inf
    return (bits.astype(np.uint16) | sign).astype(np.uint16)


def widen_f16(bits: np.ndarray) -> np.ndarray:
    """Exact float64 value of binary16 bit patterns, from the definition."""
    b = np.asarray(bits).astype(np.int64)
    sign = np.where(b & 0x8000, -1.0, 1.0)
    ex = (b >> 10) & 0x1F
    fr = (b & 0x3FF).astype(np.float64)
    val = np.where(ex == 0, fr * 2.0**-24, (1.0 + fr / 1024.0) * np.exp2(ex - 15.0))
    val = np.where(ex == 0x1F, np.where(fr == 0, np.inf, np.nan), val)
    return sign * val


def topk_encode_f16(x: np.ndarray, k: int):
    """Top-k coding with the kept values stored as binary16 (selection on the
    float32 magnitudes): (idx int64 [..., k], val float16 array)."""
    idx, val = topk_encode(x, k)
    return idx, f16_rne(val).view(np.float16)


def topk_encode_bf16(x: np.ndarray, k: int):
    """Top-k coding with the kept values stored as bfloat16 (selection still on
    the float32 magnitudes): (idx int64 [..., k], val uint16 bf16 bits)."""
    idx, val = topk_encode(x, k)
    return idx, bf16_rne(val)


# --------------------------------------------------------------------------
# attention on codes, Sec. 2 and Sec. 3.1-3.2
# --------------------------------------------------------------------------


# --------------------------------------------------------------------------
# CSR code storage (Sec. 2 sparse formats; App. J memory formula): row r holds
# the entries indptr[r] .. indptr[r+1]-1 of indices / values
# --------------------------------------------------------------------------


def csr_densify(indptr, indices, values, d: int) -> np.ndarray:
    """float64 [rows, d] from a CSR matrix (values widened exactly)."""
    indptr = np.asarray(indptr).astype(np.int64)
    rows = indptr.size - 1
    vals = widen(values)
    out = np.zeros((rows, d))
    for r in range(rows):
        for t in range(indptr[r], indptr[r + 1]):
            out[r, int(indices[t])] = vals[t]
    return out


def csr_to_fixed(indptr, indices, values, d: int, kmax: int):
    """Fixed-width codes [rows, kmax] holding the same matrix as a CSR one whose
    rows have at most kmax entries: each row's own entries, then zero-valued
    entries at the lowest coordinates the row does not hold (the fewer-than-k
    reading of Top-k coding), all sorted by ascending index.  Values keep their
    storage type."""
    indptr = np.asarray(indptr).astype(np.int64)
    rows = indptr.size - 1
    values = np.asarray(values)
    idx = np.empty((rows, kmax), dtype=np.int64)
    val = np.zeros((rows, kmax), dtype=values.dtype)
    for r in range(rows):
        own = [(int(indices[t]), values[t]) for t in range(indptr[r], indptr[r + 1])]
        if len(own) > kmax:
            raise ValueError("row longer than kmax")
        held = {u for u, _ in own}
        pad = [(u, values.dtype.type(0)) for u in range(d) if u not in held][:kmax - len(own)]
        ent = sorted(own + pad, key=lambda e: e[0])
        idx[r] = [u for u, _ in ent]
        val[r] = [v for _, v in ent]
    return idx, val


def densify(idx: np.ndarray, val, d: int) -> np.ndarray:
    """float64 [..., d]: zero except val at the coded coordinates."""
    idx = np.asarray(idx).astype(np.int64)
    v = widen(val)
    out = np.zeros(idx.shape[:-1] + (d,), dtype=np.float64)
    np.put_along_axis(out, idx, v, axis=-1)
    return out


def token_mask(pos, n_k: int, causal: bool, window: int = 0, n_global: int = 0) -> np.ndarray:
    """allowed[a, j] for queries at positions pos[a] and keys 0..n_k-1.

    The causal mask (j <= i) composed with a Longformer-style token pattern
    (App. E): a sliding window |i - j| < window, plus n_global global tokens
    at the start that every query sees and that see every key.  window 0
    means no window (plain causal / full attention)."""
    i = np.asarray(pos, dtype=np.int64)[:, None]
    j = np.arange(n_k)[None, :]
    allowed = (j <= i) if causal else np.ones((i.shape[0], n_k), dtype=bool)
    if window > 0:
        near = np.abs(i - j) < window
        glob = (j < n_global) | (i < n_global)
        allowed = allowed & (near | glob)
    return allowed


def softmax_attention(qd: np.ndarray, kd: np.ndarray, v: np.ndarray, scale: float,
                      causal: bool, pos=None, row_chunk: int = 1024, window: int = 0,
                      n_global: int = 0):
    """Plain softmax attention of one head on dense float64 inputs.

    qd [r, d] are query rows at sequence positions `pos` (default 0..r-1);
    kd [n_k, d] and v [n_k, dv] are the keys and values at positions
    0..n_k-1.  A query at position i sees the keys token_mask allows: j <= i
    when causal, all keys otherwise, further limited by a sliding window and
    global tokens when window > 0.  Rows are independent and are evaluated
    `row_chunk` at a time only to bound memory.  Returns O [r, dv] and LSE [r]
    (natural log)."""
    r = qd.shape[0]
    pos = np.arange(r) if pos is None else np.asarray(pos, dtype=np.int64)
    O = np.empty((r, v.shape[1]), dtype=np.float64)
    L = np.empty(r, dtype=np.float64)
    for s0 in range(0, r, row_chunk):
        pp = pos[s0:s0 + row_chunk]
        last = int(pp.max()) + 1 if causal else kd.shape[0]
        S = scale * (qd[s0:s0 + row_chunk] @ kd[:last].T)   # scores
        if causal or window > 0:
            allowed = token_mask(pp, last, causal, window, n_global)
            S = np.where(allowed, S, -np.inf)
        m = S.max(axis=1)                                    # row max
        P = np.exp(S - m[:, None])                           # unnormalised weights
        l = P.sum(axis=1)                                    # row sum
        O[s0:s0 + len(pp)] = (P @ v[:last]) / l[:, None]
        L[s0:s0 + len(pp)] = m + np.log(l)
    return O, L


def attn_fwd(q_idx, q_val, k_idx, k_val, v, d: int, scale: float, causal: bool,
             window: int = 0, n_global: int = 0):
    """SFA forward on codes.

    q_idx/q_val [B, Hq, n, k], k_idx/k_val [B, Hkv, n, k], v [B, Hkv, n, dv]
    (float32, or uint16 bfloat16 bits).  Query head h reads KV head
    h // (Hq // Hkv).  window / n_global: the token pattern of token_mask.
    Returns O [B, Hq, n, dv] and LSE [B, Hq, n], float64."""
    B, Hq, n, _ = np.shape(q_idx)
    Hkv = np.shape(k_idx)[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    vv = widen(v)
    O = np.empty((B, Hq, n, vv.shape[-1]), dtype=np.float64)
    L = np.empty((B, Hq, n), dtype=np.float64)
    for b in range(B):
        for g in range(Hkv):
            kd = densify(k_idx[b, g], k_val[b, g], d)
            for h in range(g * G, (g + 1) * G):
                qd = densify(q_idx[b, h], q_val[b, h], d)
                O[b, h], L[b, h] = softmax_attention(qd, kd, vv[b, g], scale, causal,
                                                     window=window, n_global=n_global)
    return O, L


def attn_fwd_rows(q_idx_bh, q_val_bh, k_idx_bg, k_val_bg, v_bg, d: int, scale: float,
                  causal: bool, rows, window: int = 0, n_global: int = 0):
    """SFA forward for chosen query rows of one (batch, query head), given the
    codes of that query head [n, k], of its KV head [n, k] and V [n, dv].
    Returns (O [len(rows), dv], LSE [len(rows)])."""
    rows = np.asarray(rows, dtype=np.int64)
    last = int(rows.max()) + 1 if causal else np.shape(k_idx_bg)[0]
    qd = densify(np.asarray(q_idx_bh)[rows], np.asarray(q_val_bh)[rows], d)
    kd = densify(np.asarray(k_idx_bg)[:last], np.asarray(k_val_bg)[:last], d)
    vv = widen(np.asarray(v_bg)[:last])
    return softmax_attention(qd, kd, vv, scale, causal, pos=rows, window=window,
                             n_global=n_global)


def attn_decode(q_idx, q_val, kc_idx, kc_val, v_cache, d: int, scale: float, seq_len=None,
                window: int = 0, n_global: int = 0):
    """SFA decode: each (b, h) query code [B, Hq, k] attends to all cached keys
    j < seq_len[b] of KV head h // G (cache codes [B, Hkv, Lmax, k], V cache
    [B, Hkv, Lmax, dv]).  The query is the token at position seq_len[b] - 1;
    with window > 0 it sees the keys token_mask allows from there.
    Returns O [B, Hq, dv] and LSE [B, Hq], float64."""
    B, Hq, _ = np.shape(q_idx)
    Hkv, Lmax = np.shape(kc_idx)[1], np.shape(kc_idx)[2]
    G = Hq // Hkv
    lens = np.full(B, Lmax) if seq_len is None else np.asarray(seq_len)
    dv = np.shape(v_cache)[-1]
    O = np.empty((B, Hq, dv))
    L = np.empty((B, Hq))
    for b in range(B):
        Lb = int(lens[b])
        for g in range(Hkv):
            kd = densify(np.asarray(kc_idx)[b, g, :Lb], np.asarray(kc_val)[b, g, :Lb], d)
            vv = widen(np.asarray(v_cache)[b, g, :Lb])
            for h in range(g * G, (g + 1) * G):
                qd = densify(np.asarray(q_idx)[b, h][None], np.asarray(q_val)[b, h][None], d)
                O1, L1 = softmax_attention(qd, kd, vv, scale, causal=True, pos=[Lb - 1],
                                           window=window, n_global=n_global)
                O[b, h], L[b, h] = O1[0], L1[0]
    return O, L


# --------------------------------------------------------------------------
# KV-cache maintenance (App. B: decode against a cache of sparse key codes
# and dense V that grows by one coded key per generated token)
# --------------------------------------------------------------------------


def cache_location(block_table, page_size, b: int, j: int):
    """(page, slot) that holds position j of sequence b.

    Paged cache: arrays [num_pages, Hkv, page_size, ...]; position j of
    sequence b sits in page block_table[b][j // page_size] at slot
    j % page_size.  block_table None is the contiguous cache
    [B, Hkv, Lmax, ...]: page b, slot j."""
    if block_table is None:
        return b, j
    return int(np.asarray(block_table)[b][j // page_size]), j % page_size


def cache_capacity(kc_idx, block_table, page_size) -> int:
    """Positions a sequence can hold: Lmax, or max_pages * page_size."""
    if block_table is None:
        return int(np.shape(kc_idx)[2])
    return int(np.shape(block_table)[1]) * int(page_size)


def kv_append(kc_idx, kc_val, v_cache, k_new, v_new, seq_len, k: int, block_table=None,
              page_size=None, n_new=None):
    """Append coded keys and their values to a KV cache, in place.

    For each sequence b and t < n_new[b] (all T when n_new is None), the key
    row k_new[b, h, t] (float32, d wide) is coded by Top-k (Sec. 3.1): kept
    coordinates ascending, values stored as bf16 bits when kc_val holds
    uint16, binary16 when it holds float16, else as float32 copies.  Code and value row v_new[b, h, t] go to
    position seq_len[b] + t of sequence b in every KV head h; a bf16 V cache
    stores bf16_rne of float32 values, a float32 one widens bf16 bits
    exactly.  Positions at or past the capacity, and pages outside the pool,
    are not written.  Returns the new lengths, min(seq_len + n_new,
    capacity)."""
    k_new = np.asarray(k_new, dtype=np.float32)
    B, Hkv, T, _ = k_new.shape
    cap = cache_capacity(kc_idx, block_table, page_size)
    npages = np.shape(kc_idx)[0]
    lens = np.asarray(seq_len).astype(np.int64)
    cnt = np.full(B, T) if n_new is None else np.clip(np.asarray(n_new), 0, T)
    code_dt = np.asarray(kc_val).dtype  # uint16: bf16 bits; float16: binary16
    v_new = np.asarray(v_new)
    for b in range(B):
        for t in range(int(cnt[b])):
            j = int(lens[b]) + t
            if j >= cap:
                break
            page, slot = cache_location(block_table, page_size, b, j)
            if not 0 <= page < npages:
                continue
            for h in range(Hkv):
                if code_dt == np.uint16:
                    ci, cv = topk_encode_bf16(k_new[b, h, t], k)
                elif code_dt == np.float16:
                    ci, cv = topk_encode_f16(k_new[b, h, t], k)
                else:
                    ci, cv = topk_encode(k_new[b, h, t], k)
                kc_idx[page, h, slot] = ci
                kc_val[page, h, slot] = cv
                row = v_new[b, h, t]
                if v_cache.dtype == np.uint16:
                    v_cache[page, h, slot] = row if row.dtype == np.uint16 else bf16_rne(row)
                else:
                    v_cache[page, h, slot] = widen(row).astype(v_cache.dtype)
    return np.minimum(lens + cnt, cap)


def cache_gather(kc_idx, kc_val, v_cache, b: int, L: int, block_table=None, page_size=None):
    """Contiguous copies [Hkv, L, ...] of positions 0..L-1 of sequence b."""
    Hkv = np.shape(kc_idx)[1]
    gi = np.empty((Hkv, L) + np.shape(kc_idx)[3:], dtype=np.asarray(kc_idx).dtype)
    gv = np.empty((Hkv, L) + np.shape(kc_val)[3:], dtype=np.asarray(kc_val).dtype)
    gvv = np.empty((Hkv, L) + np.shape(v_cache)[3:], dtype=np.asarray(v_cache).dtype)
    for j in range(L):
        page, slot = cache_location(block_table, page_size, b, j)
        gi[:, j] = kc_idx[page, :, slot]
        gv[:, j] = kc_val[page, :, slot]
        gvv[:, j] = v_cache[page, :, slot]
    return gi, gv, gvv


def attn_decode_paged(q_idx, q_val, kc_idx, kc_val, v_cache, seq_len, d: int, scale: float,
                      block_table=None, page_size=None, window: int = 0, n_global: int = 0):
    """Decode (App. B) over a paged cache: each sequence's first seq_len[b]
    positions, read through its block table, then the plain decode."""
    B, Hq, _ = np.shape(q_idx)
    dv = np.shape(v_cache)[-1]
    O = np.zeros((B, Hq, dv))
    L = np.full((B, Hq), -np.inf)
    for b in range(B):
        Lb = int(seq_len[b])
        if Lb == 0:
            continue
        gi, gv, gvv = cache_gather(kc_idx, kc_val, v_cache, b, Lb, block_table, page_size)
        Ob, Lsb = attn_decode(np.asarray(q_idx)[b:b + 1], np.asarray(q_val)[b:b + 1],
                              gi[None], gv[None], gvv[None], d, scale, window=window,
                              n_global=n_global)
        O[b], L[b] = Ob[0], Lsb[0]
    return O, L


# --------------------------------------------------------------------------
# 8-bit cache (App. E, "SFA (quant)": SFA combined with 8-bit quantisation
# of the activations; with a KV cache, the cached keys and values are those
# activations): symmetric per-row int8 with one float32 scale per row
# --------------------------------------------------------------------------


def quant_q8(x: np.ndarray):
    """Symmetric 8-bit quantisation of each row of x [..., m] (float32).

    Per row: a = max |x_u|, s = a / 127 as a float32 division, and
    q_u = x_u / s as a float32 division, rounded to the nearest integer with
    ties to even, limited to [-127, 127].  A row of zeros has s = 0 and
    q = 0.  The value code q_u stands for is q_u * s.
    Returns (q int8 [..., m], s float32 [...])."""
    x = np.asarray(x, dtype=np.float32)
    a = np.abs(x).max(axis=-1)
    s = (a / np.float32(127)).astype(np.float32)
    safe = np.where(s > 0, s, np.float32(1)).astype(np.float32)
    r = (x / safe[..., None]).astype(np.float32)
    q = np.clip(np.rint(r), -127, 127)
    q = np.where(s[..., None] > 0, q, 0).astype(np.int8)
    return q, s


def dequant_q8(q, s) -> np.ndarray:
    """float64 values q * s of int8 codes with their row scales."""
    return np.asarray(q).astype(np.float64) * np.asarray(s).astype(np.float64)[..., None]


def kv_append_q8(kc_idx, kc_val, kc_scale, v_cache, v_scale, k_new, v_new, seq_len, k: int,
                 n_new=None):
    """Append to a contiguous 8-bit cache, in place: kc_idx [B, Hkv, Lmax, k],
    kc_val int8 [B, Hkv, Lmax, k], kc_scale float32 [B, Hkv, Lmax], v_cache int8
    [B, Hkv, Lmax, d], v_scale float32 [B, Hkv, Lmax].

    For each sequence b and t < n_new[b] (all T when None), the key row
    k_new[b, h, t] (float32) is coded by Top-k (Sec. 3.1; float32 values) and
    its k kept values quantised as one row (quant_q8); the value row
    v_new[b, h, t] (float32, or uint16 bf16 bits widened exactly) is
    quantised as one row.  Both go to position seq_len[b] + t; positions at
    or past Lmax are not written.  Returns the new lengths."""
    k_new = np.asarray(k_new, dtype=np.float32)
    B, Hkv, T, _ = k_new.shape
    Lmax = np.shape(kc_idx)[2]
    lens = np.asarray(seq_len).astype(np.int64)
    cnt = np.full(B, T) if n_new is None else np.clip(np.asarray(n_new), 0, T)
    vv = np.asarray(v_new)
    vv = widen(vv).astype(np.float32) if vv.dtype == np.uint16 else vv.astype(np.float32)
    for b in range(B):
        for t in range(int(cnt[b])):
            j = int(lens[b]) + t
            if j >= Lmax:
                break
            for h in range(Hkv):
                ci, cv = topk_encode(k_new[b, h, t], k)
                q, sc = quant_q8(cv)
                kc_idx[b, h, j], kc_val[b, h, j], kc_scale[b, h, j] = ci, q, sc
                q, sc = quant_q8(vv[b, h, t])
                v_cache[b, h, j], v_scale[b, h, j] = q, sc
    return np.minimum(lens + cnt, Lmax)


# --------------------------------------------------------------------------
# accounting (Sec. 3.1 efficiency analysis; App. J memory formula)
# --------------------------------------------------------------------------


# --------------------------------------------------------------------------
# backward (straight-through estimator, Sec. 3.1, Eq. (6))
# --------------------------------------------------------------------------


def stored_output(o: np.ndarray, o_store) -> np.ndarray:
    """The forward's output O as the backward receives it: o_store None keeps
    it exact, "bf16" rounds it to the nearest bfloat16 (ties to even) through
    float32, as a forward that writes O in bfloat16 stores it."""
    if o_store is None:
        return o
    assert o_store == "bf16", o_store
    return widen(bf16_rne(np.asarray(o, dtype=np.float64).astype(np.float32)))


def softmax_attention_grad(qd: np.ndarray, kd: np.ndarray, v: np.ndarray, do: np.ndarray,
                           scale: float, causal: bool, window: int = 0, n_global: int = 0,
                           o_store=None):
    """Gradients of O = softmax(scale * qd kd^T, mask) v for one head, dense
    float64, queries at positions 0..r-1 and keys at 0..n_k-1; the mask is
    token_mask (causal, window, global tokens).

    With P the row-normalised weights: dV = P^T dO, dP = dO V^T,
    dS = P * (dP - D), dQ = scale dS K, dK = scale dS^T Q, where
    D_i = dO_i . O_i = rowsum(dP * P)_i.  With o_store the backward takes O
    as the forward stored it (stored_output), and D_i = dO_i . O_i uses that.
    Returns (dQ [r, d], dK [n_k, d], dV [n_k, dv])."""
    S = scale * (qd @ kd.T)
    if causal or window > 0:
        allowed = token_mask(np.arange(qd.shape[0]), kd.shape[0], causal, window, n_global)
        S = np.where(allowed, S, -np.inf)
    P = np.exp(S - S.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    dV = P.T @ do
    dP = do @ v.T
    if o_store is None:
        D = (dP * P).sum(axis=1, keepdims=True)
    else:
        D = (do * stored_output(P @ v, o_store)).sum(axis=1, keepdims=True)
    dS = P * (dP - D)
    return scale * (dS @ kd), scale * (dS.T @ qd), dV


def attn_bwd(q_idx, q_val, k_idx, k_val, v, do, d: int, scale: float, causal: bool,
             window: int = 0, n_global: int = 0, o_store=None):
    """SFA backward on codes (Sec. 3.1, Eq. (6)).

    Inputs as attn_fwd, plus do [B, Hq, n, dv] (float32, or uint16 bf16
    bits).  The gradient of query i's coordinate u is the dense dQ~[i, u] on
    its support and 0 elsewhere, so it is returned in code form:
    dq_val [B, Hq, n, k] with dq_val[..., t] the gradient at q_idx[..., t];
    likewise dk_val [B, Hkv, n, k].  dv [B, Hkv, n, dv].  A KV head's
    gradients sum over the query heads that read it.  o_store: the stored
    form of the forward's output that D_i = dO_i . O_i uses (stored_output).
    float64."""
    B, Hq, n, k = np.shape(q_idx)
    Hkv = np.shape(k_idx)[1]
    G = Hq // Hkv
    vv, dd = widen(v), widen(do)
    dq = np.empty((B, Hq, n, k), dtype=np.float64)
    dk = np.zeros((B, Hkv, n, k), dtype=np.float64)
    dv = np.zeros((B, Hkv, n, vv.shape[-1]), dtype=np.float64)
    for b in range(B):
        for g in range(Hkv):
            kd = densify(k_idx[b, g], k_val[b, g], d)
            dkd = np.zeros_like(kd)
            for h in range(g * G, (g + 1) * G):
                qd = densify(q_idx[b, h], q_val[b, h], d)
                gq, gk, gv = softmax_attention_grad(qd, kd, vv[b, g], dd[b, h], scale, causal,
                                                    window, n_global, o_store)
                dq[b, h] = np.take_along_axis(gq, np.asarray(q_idx[b, h], dtype=np.int64), 1)
                dkd += gk
                dv[b, g] += gv
            dk[b, g] = np.take_along_axis(dkd, np.asarray(k_idx[b, g], dtype=np.int64), 1)
    return dq, dk, dv


def attn_bwd_rows(q_idx_bh, q_val_bh, k_idx_bg, k_val_bg, v_bg, do_bh, d: int, scale: float,
                  causal: bool, rows, window: int = 0, n_global: int = 0, o_store=None):
    """dq_val (Eq. (6)) of the selected query rows of one head, each row on
    its own: p = softmax over the row's allowed keys, dp = V do_i,
    ds = p * (dp - D_i) with D_i = p.dp = do_i . o_i (o_i = p V, in its stored
    form with o_store), dq~ = scale ds K~, read at the row's support.
    Returns [len(rows), k], float64."""
    kd = densify(k_idx_bg, k_val_bg, d)
    vv, dd = widen(v_bg), widen(do_bh)
    out = np.empty((len(rows), np.shape(q_idx_bh)[1]), dtype=np.float64)
    for r, i in enumerate(rows):
        qd = densify(q_idx_bh[i][None], q_val_bh[i][None], d)[0]
        keys = np.flatnonzero(token_mask([int(i)], kd.shape[0], causal, window, n_global)[0])
        s = scale * (kd[keys] @ qd)
        p = np.exp(s - s.max())
        p /= p.sum()
        dp = vv[keys] @ dd[i]
        Di = p @ dp if o_store is None else dd[i] @ stored_output(p @ vv[keys], o_store)
        ds = p * (dp - Di)
        out[r] = (scale * (ds @ kd[keys]))[np.asarray(q_idx_bh[i], dtype=np.int64)]
    return out


def attn_bwd_cols(q_idx_bg, q_val_bg, k_idx_bg, k_val_bg, v_bg, do_bg, d: int, scale: float,
                  causal: bool, cols, row_chunk: int = 1024, window: int = 0, n_global: int = 0,
                  row_from: int = 0, o_store=None):
    """dk_val and dv (Eq. (6)) of the selected keys of one KV head, summed
    over its query heads: q_*_bg [G, n, k], do_bg [G, n, dv].  Each query
    row's LSE_i and D_i = dO_i . O_i come from the plain forward
    (softmax_attention); then for key j and every query i that sees it,
    P_ij = exp(s_ij - LSE_i), dS_ij = P_ij (dO_i . v_j - D_i),
    dv_j = sum_i P_ij dO_i and dk~_j = scale sum_i dS_ij q~_i; with o_store,
    D_i takes O in its stored form (stored_output).
    row_from > 0 (causal, no window, every column >= row_from): only query
    rows from row_from on are evaluated; the rows below see none of the
    columns (j <= i fails), so they would add only zeros.
    Returns (dk [len(cols), k], dv [len(cols), dv]), float64."""
    kd = densify(k_idx_bg, k_val_bg, d)
    vv, dd = widen(v_bg), widen(do_bg)
    n = kd.shape[0]
    cols = np.asarray(cols, dtype=np.int64)
    if row_from > 0:
        assert causal and window == 0 and int(cols.min()) >= row_from
    pos = np.arange(row_from, n)
    dk = np.zeros((len(cols), np.shape(k_idx_bg)[1]), dtype=np.float64)
    dv = np.zeros((len(cols), vv.shape[1]), dtype=np.float64)
    dkd = np.zeros((len(cols), d), dtype=np.float64)
    for h in range(np.shape(q_idx_bg)[0]):
        qd = densify(q_idx_bg[h], q_val_bg[h], d)[row_from:]
        do_h = dd[h][row_from:]
        O, L = softmax_attention(qd, kd, vv, scale, causal, pos=pos, row_chunk=row_chunk,
                                 window=window, n_global=n_global)
        D = (do_h * stored_output(O, o_store)).sum(axis=1)
        S = scale * (qd @ kd[cols].T)                      # [rows, len(cols)]
        if causal or window > 0:
            allowed = token_mask(pos, n, causal, window, n_global)[:, cols]
            S = np.where(allowed, S, -np.inf)
        P = np.exp(S - L[:, None])
        dS = P * (do_h @ vv[cols].T - D[:, None])
        dv += P.T @ do_h
        dkd += scale * (dS.T @ qd)
    for c, j in enumerate(cols):
        dk[c] = dkd[c][np.asarray(k_idx_bg[j], dtype=np.int64)]
    return dk, dv


def overlap_count(q_idx_bh, k_idx_bg, causal: bool, d: int) -> int:
    """E = number of (allowed pair, shared coordinate) triples of one head:
    sum over coordinates u of #{(i, j) allowed : u in S_i and u in S_j}."""
    q = np.asarray(q_idx_bh)
    kk = np.asarray(k_idx_bg)
    n = q.shape[0]
    qm = np.zeros((n, d), dtype=np.int64)
    km = np.zeros((n, d), dtype=np.int64)
    np.put_along_axis(qm, q.astype(np.int64), 1, axis=1)
    np.put_along_axis(km, kk.astype(np.int64), 1, axis=1)
    if causal:
        kc = np.cumsum(km, axis=0)          # keys j <= i holding u
        return int((qm * kc).sum())
    return int((qm * km.sum(axis=0)[None, :]).sum())


def csr_bytes(N: int, k: int, s_val: int, s_idx: int, s_ptr: int) -> int:
    """Bytes of an N-row CSR matrix with k nonzeros per row (App. J)."""
    return N * k * (s_val + s_idx) + (N + 1) * s_ptr
