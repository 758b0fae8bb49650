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
* bf16 storage of code values (round to nearest, ties to even) for the
  KV-cache codes.

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
    value is that of the float32 with the same high 16 bits."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
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


def topk_encode_bf16(x: np.ndarray, k: int):
    """Top-k coding with the kept values stored as bfloat16 (selection still on
    the float32 magnitudes): (idx int64 [..., k], val uint16 bf16 bits)."""
    idx, val = topk_encode(x, k)
    return idx, bf16_rne(val)


# --------------------------------------------------------------------------
# attention on codes, Sec. 2 and Sec. 3.1-3.2
# --------------------------------------------------------------------------


def densify(idx: np.ndarray, val, d: int) -> np.ndarray:
    """float64 [..., d]: zero except val at the coded coordinates."""
    idx = np.asarray(idx).astype(np.int64)
    v = widen(val)
    out = np.zeros(idx.shape[:-1] + (d,), dtype=np.float64)
    np.put_along_axis(out, idx, v, axis=-1)
    return out


def softmax_attention(qd: np.ndarray, kd: np.ndarray, v: np.ndarray, scale: float,
                      causal: bool, pos=None, row_chunk: int = 1024):
    """Plain softmax attention of one head on dense float64 inputs.

    qd [r, d] are query rows at sequence positions `pos` (default 0..r-1);
    kd [n_k, d] and v [n_k, dv] are the keys and values at positions
    0..n_k-1.  A query at position i sees keys j <= i when causal, all keys
    otherwise.  Rows are independent and are evaluated `row_chunk` at a time
    only to bound memory.  Returns O [r, dv] and LSE [r] (natural log)."""
    r = qd.shape[0]
    pos = np.arange(r) if pos is None else np.asarray(pos, dtype=np.int64)
    O = np.empty((r, v.shape[1]), dtype=np.float64)
    L = np.empty(r, dtype=np.float64)
    for s0 in range(0, r, row_chunk):
        pp = pos[s0:s0 + row_chunk]
        last = int(pp.max()) + 1 if causal else kd.shape[0]
        S = scale * (qd[s0:s0 + row_chunk] @ kd[:last].T)   # scores
        if causal:
            allowed = np.arange(last)[None, :] <= pp[:, None]
            S = np.where(allowed, S, -np.inf)
        m = S.max(axis=1)                                    # row max
        P = np.exp(S - m[:, None])                           # unnormalised weights
        l = P.sum(axis=1)                                    # row sum
        O[s0:s0 + len(pp)] = (P @ v[:last]) / l[:, None]
        L[s0:s0 + len(pp)] = m + np.log(l)
    return O, L


def attn_fwd(q_idx, q_val, k_idx, k_val, v, d: int, scale: float, causal: bool):
    """SFA forward on codes.

    q_idx/q_val [B, Hq, n, k], k_idx/k_val [B, Hkv, n, k], v [B, Hkv, n, dv]
    (float32, or uint16 bfloat16 bits).  Query head h reads KV head
    h // (Hq // Hkv).  Returns O [B, Hq, n, dv] and LSE [B, Hq, n], float64."""
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
                O[b, h], L[b, h] = softmax_attention(qd, kd, vv[b, g], scale, causal)
    return O, L


def attn_fwd_rows(q_idx_bh, q_val_bh, k_idx_bg, k_val_bg, v_bg, d: int, scale: float,
                  causal: bool, rows):
    """SFA forward for chosen query rows of one (batch, query head), given the
    codes of that query head [n, k], of its KV head [n, k] and V [n, dv].
    Returns (O [len(rows), dv], LSE [len(rows)])."""
    rows = np.asarray(rows, dtype=np.int64)
    last = int(rows.max()) + 1 if causal else np.shape(k_idx_bg)[0]
    qd = densify(np.asarray(q_idx_bh)[rows], np.asarray(q_val_bh)[rows], d)
    kd = densify(np.asarray(k_idx_bg)[:last], np.asarray(k_val_bg)[:last], d)
    vv = widen(np.asarray(v_bg)[:last])
    return softmax_attention(qd, kd, vv, scale, causal, pos=rows)


def attn_decode(q_idx, q_val, kc_idx, kc_val, v_cache, d: int, scale: float, seq_len=None):
    """SFA decode: each (b, h) query code [B, Hq, k] attends to all cached keys
    j < seq_len[b] of KV head h // G (cache codes [B, Hkv, Lmax, k], V cache
    [B, Hkv, Lmax, dv]).  Returns O [B, Hq, dv] and LSE [B, Hq], float64."""
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
                O1, L1 = softmax_attention(qd, kd, vv, scale, causal=False)
                O[b, h], L[b, h] = O1[0], L1[0]
    return O, L


# --------------------------------------------------------------------------
# accounting (Sec. 3.1 efficiency analysis; App. J memory formula)
# --------------------------------------------------------------------------


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
