"""Pins of the oracle's compact code storage (App. J: 8-bit indices, fp16
values, CSR rows with an int32 indptr).

  * binary16 rounding, written from its definition, equals numpy's float16
    conversion (a library routine, IEEE round-to-nearest-even) on random values
    and on the edges: ties in the normal and subnormal range, the subnormal
    boundary, the largest finite value and overflow;
  * binary16 widening, from the definition, equals numpy's float16 -> float64;
  * CSR -> fixed rows keeps the matrix (densified by a loop over the CSR
    entries, written here independently), pads at the lowest free
    coordinates (brute force), and leaves full rows as they were;
  * attention on the fixed rows equals plain softmax attention on the
    densified CSR matrices.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F

import oracle


def _edges():
    ulp = 2.0 ** -10
    vals = [0.0, -0.0, 1.0, 1 + ulp / 2, 1 + 3 * ulp / 2, 1 + ulp / 2 + 2 ** -20,
            2.0 ** -14, 2.0 ** -14 - 2.0 ** -25, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -25,
            2.0 ** -26, 5 * 2.0 ** -26, 65504.0, 65519.0, 65520.0, 1e6, 2.0 ** -14 * 1.5,
            0.1, 1 / 3, 3.14159]
    v = np.array(vals, dtype=np.float32)
    return np.concatenate([v, -v])


def test_f16_rounding_matches_ieee_conversion():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200000).astype(np.float32) * np.float32(4.0),
                        (rng.standard_normal(20000) * 1e-5).astype(np.float32),
                        (rng.standard_normal(20000) * 3e4).astype(np.float32), _edges()])
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    got = oracle.f16_rne(x)
    assert np.array_equal(got, want), np.flatnonzero(got != want)[:5]


def test_f16_widening_is_exact():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    want = bits.view(np.float16).astype(np.float64)
    got = oracle.widen_f16(bits)
    fin = np.isfinite(want)
    assert np.array_equal(got[fin], want[fin])
    assert np.array_equal(np.isinf(got), np.isinf(want))
    assert np.array_equal(np.isnan(got), np.isnan(want))


def test_topk_encode_f16():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((300, 64)).astype(np.float32)
    i, v = oracle.topk_encode_f16(x, 8)
    i32, v32 = oracle.topk_encode(x, 8)
    assert np.array_equal(i, i32)
    with np.errstate(over="ignore"):
        assert np.array_equal(v.view(np.uint16), v32.astype(np.float16).view(np.uint16))
    assert v.dtype == np.float16


def _random_csr(rng, rows, d, kmax, dtype=np.float32):
    lens = rng.integers(0, kmax + 1, rows)
    lens[0], lens[-1] = 0, kmax
    indptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    indices = np.concatenate([rng.permutation(d)[:m] for m in lens]).astype(np.int64)
    values = rng.standard_normal(int(indptr[-1])).astype(dtype)
    return indptr, indices, values


def test_csr_to_fixed():
    rng = np.random.default_rng(2)
    rows, d, kmax = 60, 32, 7
    indptr, indices, values = _random_csr(rng, rows, d, kmax)
    idx, val = oracle.csr_to_fixed(indptr, indices, values, d, kmax)
    dense = np.zeros((rows, d))
    for r in range(rows):                      # the CSR matrix, entry by entry
        for t in range(indptr[r], indptr[r + 1]):
            dense[r, indices[t]] = values[t]
    assert np.array_equal(oracle.csr_densify(indptr, indices, values, d), dense)
    assert np.array_equal(oracle.densify(idx, val, d), dense)
    for r in range(rows):
        assert list(idx[r]) == sorted(set(idx[r].tolist())) and len(idx[r]) == kmax
        own = set(indices[indptr[r]:indptr[r + 1]].tolist())
        free = [u for u in range(d) if u not in own]
        assert set(idx[r].tolist()) == own | set(free[:kmax - len(own)])
        if len(own) == kmax:
            order = np.argsort(indices[indptr[r]:indptr[r + 1]])
            assert np.array_equal(val[r], values[indptr[r]:indptr[r + 1]][order])


def test_attention_on_csr_rows():
    rng = np.random.default_rng(3)
    n, d, kmax = 40, 16, 5
    qp, qi, qv = _random_csr(rng, n, d, kmax, np.float16)
    kp, ki, kv = _random_csr(rng, n, d, kmax, np.float16)
    v = rng.standard_normal((n, d)).astype(np.float32)
    fq, fqv = oracle.csr_to_fixed(qp, qi, qv, d, kmax)
    fk, fkv = oracle.csr_to_fixed(kp, ki, kv, d, kmax)
    for causal in (True, False):
        O, L = oracle.attn_fwd(fq[None, None], fqv[None, None], fk[None, None], fkv[None, None],
                               v[None, None], d, 0.4, causal)
        qd = torch.from_numpy(oracle.csr_densify(qp, qi, qv, d))
        kd = torch.from_numpy(oracle.csr_densify(kp, ki, kv, d))
        ref = F.scaled_dot_product_attention(qd[None], kd[None], torch.from_numpy(v).double()[None],
                                             is_causal=causal, scale=0.4)[0].numpy()
        assert np.abs(O[0, 0] - ref).max() < 1e-12
        s = 0.4 * (qd @ kd.T).numpy()
        if causal:
            s = np.where(np.tril(np.ones((n, n))) > 0, s, -np.inf)
        m = s.max(1)
        assert np.abs(L[0, 0] - (m + np.log(np.exp(s - m[:, None]).sum(1)))).max() < 1e-12
