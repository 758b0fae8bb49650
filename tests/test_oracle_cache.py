"""Pins of the oracle's KV-cache maintenance (decode of App. B over a cache
that grows by coded keys).

The append / gather / paged-decode functions are pinned against things that
do not share their indexing:
  * appending in several ragged calls through a shuffled block table, then
    reading back, gives the one-shot Top-k coding of each sequence's whole
    key stream (already pinned in test_oracle_topk.py) and its bf16 V;
  * slots no append reached keep their sentinel, and a full cache stops at
    its capacity;
  * decode of a query against the first L positions equals the last row of
    the causal forward whose last query is that query (A-13 of the decode
    reading: the new token's own key is already in the cache);
  * a contiguous cache is the paged cache with one page per sequence.
"""
import math

import numpy as np

import oracle


def _pool(num_pages, Hkv, P, k, d, v_bf16=True):
    kc_idx = np.full((num_pages, Hkv, P, k), -1, dtype=np.int16)
    kc_val = np.full((num_pages, Hkv, P, k), 0xFFFF, dtype=np.uint16)
    v = np.full((num_pages, Hkv, P, d), 0xFFFF if v_bf16 else np.nan,
                dtype=np.uint16 if v_bf16 else np.float32)
    return kc_idx, kc_val, v


def test_ragged_appends_equal_one_shot_coding():
    rng = np.random.default_rng(1)
    B, Hkv, d, k, P, max_pages = 3, 2, 32, 4, 8, 6
    num_pages = B * max_pages + 5
    table = rng.permutation(num_pages)[:B * max_pages].reshape(B, max_pages)
    kc_idx, kc_val, vc = _pool(num_pages, Hkv, P, k, d)
    lens = np.zeros(B, dtype=np.int64)
    keys = [[] for _ in range(B)]
    vals = [[] for _ in range(B)]
    for step, T in enumerate((7, 1, 13, 5)):
        kn = rng.standard_normal((B, Hkv, T, d)).astype(np.float32)
        vn = rng.standard_normal((B, Hkv, T, d)).astype(np.float32)
        n_new = rng.integers(0, T + 1, B)
        n_new[step % B] = T
        new = oracle.kv_append(kc_idx, kc_val, vc, kn, vn, lens, k, table, P, n_new)
        assert np.array_equal(new, lens + n_new)
        for b in range(B):
            keys[b].append(kn[b, :, :n_new[b]])
            vals[b].append(vn[b, :, :n_new[b]])
        lens = new
    used = np.zeros((num_pages, P), dtype=bool)
    for b in range(B):
        kall = np.concatenate(keys[b], axis=1)
        vall = np.concatenate(vals[b], axis=1)
        gi, gv, gvv = oracle.cache_gather(kc_idx, kc_val, vc, b, int(lens[b]), table, P)
        wi, wv = oracle.topk_encode_bf16(kall, k)
        assert np.array_equal(gi, wi) and np.array_equal(gv, wv)
        assert np.array_equal(gvv, oracle.bf16_rne(vall))
        for j in range(int(lens[b])):
            used[table[b, j // P], j % P] = True
    # every slot no append reached still holds the sentinel
    slot_major = lambda a: a.transpose(0, 2, 1, 3)  # [page, slot, head, ...]
    assert (slot_major(kc_idx)[~used] == -1).all() and (slot_major(kc_val)[~used] == 0xFFFF).all()
    assert (slot_major(vc)[~used] == 0xFFFF).all()
    assert used.sum() == lens.sum()


def test_capacity_and_skipped_pages():
    rng = np.random.default_rng(2)
    B, Hkv, d, k, P, max_pages = 2, 1, 16, 3, 4, 2
    table = np.array([[0, 1], [2, 9]])  # page 9 is outside a 3-page pool
    kc_idx, kc_val, vc = _pool(3, Hkv, P, k, d, v_bf16=False)
    kn = rng.standard_normal((B, Hkv, 11, d)).astype(np.float32)
    vn = rng.standard_normal((B, Hkv, 11, d)).astype(np.float32)
    lens = oracle.kv_append(kc_idx, kc_val, vc, kn, vn, np.array([3, 0]), k, table, P)
    assert list(lens) == [8, 8]  # capacity 2 pages x 4 slots
    # sequence 0: positions 3..7 hold keys 0..4
    gi, _, gvv = oracle.cache_gather(kc_idx, kc_val, vc, 0, 8, table, P)
    assert np.array_equal(gi[:, 3:], oracle.topk_encode(kn[0, :, :5], k)[0])
    assert np.array_equal(gvv[:, 3:], vn[0, :, :5])
    assert (kc_idx[0, :, :3] == -1).all()
    # sequence 1: positions 0..3 in page 2; positions 4..7 map outside the pool
    assert np.array_equal(kc_idx[2, :, :], oracle.topk_encode(kn[1, :, :4], k)[0])


def test_decode_paged_is_last_row_of_the_forward():
    rng = np.random.default_rng(3)
    Hq, Hkv, d, k, P, L = 4, 2, 32, 5, 16, 45
    G = Hq // Hkv
    table = np.array([[4, 0, 2, 5]])
    kc_idx, kc_val, vc = _pool(6, Hkv, P, k, d)
    kd = rng.standard_normal((1, Hkv, L, d)).astype(np.float32)
    vd = rng.standard_normal((1, Hkv, L, d)).astype(np.float32)
    # the cache grows by a prompt of 30 tokens, then one token at a time
    lens = oracle.kv_append(kc_idx, kc_val, vc, kd[:, :, :30], vd[:, :, :30], [0], k, table, P)
    for t in range(30, L):
        lens = oracle.kv_append(kc_idx, kc_val, vc, kd[:, :, t:t + 1], vd[:, :, t:t + 1], lens,
                                k, table, P)
    assert lens[0] == L
    qd = rng.standard_normal((1, Hq, L, d)).astype(np.float32)
    qi, qv = oracle.topk_encode(qd, k)
    scale = 1 / math.sqrt(d)
    O, Ls = oracle.attn_decode_paged(qi[:, :, L - 1], qv[:, :, L - 1], kc_idx, kc_val, vc,
                                     lens, d, scale, table, P)
    ki, kv = oracle.topk_encode_bf16(kd, k)
    Of, Lf = oracle.attn_fwd(qi, qv, ki, kv, oracle.bf16_rne(vd), d, scale, causal=True)
    assert np.abs(O[0] - Of[0, :, L - 1]).max() < 1e-12
    assert np.abs(Ls[0] - Lf[0, :, L - 1]).max() < 1e-12
    assert G == 2


def test_contiguous_is_one_page_per_sequence():
    rng = np.random.default_rng(4)
    B, Hq, Hkv, d, k, Lmax = 2, 2, 1, 16, 4, 20
    ci = np.full((B, Hkv, Lmax, k), -1, dtype=np.int16)
    cv = np.zeros((B, Hkv, Lmax, k), dtype=np.float32)
    vc = np.zeros((B, Hkv, Lmax, d), dtype=np.float32)
    kn = rng.standard_normal((B, Hkv, 9, d)).astype(np.float32)
    vn = rng.standard_normal((B, Hkv, 9, d)).astype(np.float32)
    lens = oracle.kv_append(ci, cv, vc, kn, vn, [0, 11], k)
    assert list(lens) == [9, 20]
    pi, pv, pvv = ci.copy(), cv.copy(), vc.copy()
    ci2 = np.full_like(ci, -1); cv2 = np.zeros_like(cv); vc2 = np.zeros_like(vc)
    lens2 = oracle.kv_append(ci2, cv2, vc2, kn, vn, [0, 11], k, np.arange(B)[:, None], Lmax)
    assert list(lens2) == [9, 20]
    assert np.array_equal(ci2, pi) and np.array_equal(cv2, pv) and np.array_equal(vc2, pvv)
    qi, qv = oracle.topk_encode(rng.standard_normal((B, Hq, d)).astype(np.float32), k)
    O1, L1 = oracle.attn_decode(qi, qv, ci, cv, vc, d, 0.3, seq_len=lens)
    O2, L2 = oracle.attn_decode_paged(qi, qv, ci, cv, vc, lens, d, 0.3)
    assert np.array_equal(O1, O2) and np.array_equal(L1, L2)
