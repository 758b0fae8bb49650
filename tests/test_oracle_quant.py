"""Pins of the oracle's 8-bit cache ("SFA (quant)", App. E: SFA with 8-bit
activations; with a KV cache the cached keys and values are those
activations): symmetric per-row int8 codes with a float32 scale.

  * hand-worked rows (tests/golden/q8_quant.json) whose scale is a power of
    two, so every division is exact: the codes, halves to even included;
  * invariants on random rows: |q| <= 127, the largest |x| maps to +-127
    with its sign, |x - q s| <= s / 2 (plus float32 rounding of x / s),
    quant(-x) = -quant(x), and scaling a row by 2^j scales s by 2^j and
    keeps q (all float32 operations then scale exactly);
  * the 8-bit append: indices equal the Top-k coding, the stored codes stand
    for the coded values and the value rows within half a step, positions
    past the capacity are not written.
"""
import json
import os

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def test_hand_worked_rows():
    fx = json.load(open(os.path.join(HERE, "golden", "q8_quant.json")))
    for row in fx["rows"]:
        q, s = oracle.quant_q8(np.array([row["x"]], dtype=np.float32))
        assert q.dtype == np.int8
        assert float(s[0]) == row["s"], row["why"]
        assert q[0].tolist() == row["q"], row["why"]


@pytest.mark.parametrize("m", [8, 16, 64, 128])
def test_invariants_on_random_rows(m):
    rng = np.random.default_rng(m)
    x = (rng.standard_normal((2000, m)) * np.exp(rng.uniform(-20, 20, (2000, 1)))).astype(np.float32)
    q, s = oracle.quant_q8(x)
    assert np.abs(q.astype(np.int32)).max() <= 127
    am = np.abs(x).argmax(axis=1)
    top = q[np.arange(len(x)), am].astype(np.int32)
    assert np.array_equal(top, np.where(x[np.arange(len(x)), am] > 0, 127, -127))
    err = np.abs(x.astype(np.float64) - oracle.dequant_q8(q, s))
    assert (err <= s.astype(np.float64)[:, None] * (0.5 + 2.0 ** -20)).all()
    qn, sn = oracle.quant_q8(-x)
    assert np.array_equal(qn, -q) and np.array_equal(sn, s)
    for j in (-7, 3, 11):
        qj, sj = oracle.quant_q8((x * np.float32(2.0 ** j)).astype(np.float32))
        assert np.array_equal(qj, q) and np.array_equal(sj, (s * np.float32(2.0 ** j)))


def test_step_is_max_over_127_not_128():
    # a row whose other entries sit exactly on the 127-step grid: q is the
    # grid index, which a 128-step or truncating quantiser would miss
    x = np.array([[127.0, 64.0, -1.0, 126.0, -127.0]], dtype=np.float32) * np.float32(0.25)
    q, s = oracle.quant_q8(x)
    assert float(s[0]) == 0.25 and q[0].tolist() == [127, 64, -1, 126, -127]


def test_append_q8_codes_and_capacity():
    rng = np.random.default_rng(5)
    B, Hkv, T, d, k, Lmax = 3, 2, 6, 32, 4, 9
    kn = rng.standard_normal((B, Hkv, T, d)).astype(np.float32)
    vn = oracle.bf16_rne(rng.standard_normal((B, Hkv, T, d)).astype(np.float32))
    ci = np.full((B, Hkv, Lmax, k), -1, np.int16)
    cv = np.full((B, Hkv, Lmax, k), 99, np.int8)
    cs = np.full((B, Hkv, Lmax), -1.0, np.float32)
    vc = np.full((B, Hkv, Lmax, d), 99, np.int8)
    vs = np.full((B, Hkv, Lmax), -1.0, np.float32)
    lens = np.array([0, 5, 8])
    new = oracle.kv_append_q8(ci, cv, cs, vc, vs, kn, vn, lens, k, n_new=np.array([6, 2, 6]))
    assert new.tolist() == [6, 7, 9]
    for b, (l0, cnt) in enumerate(((0, 6), (5, 2), (8, 1))):
        for t in range(cnt):
            j = l0 + t
            for h in range(Hkv):
                ti, tv = oracle.topk_encode(kn[b, h, t], k)
                assert np.array_equal(ci[b, h, j], ti)
                step = float(cs[b, h, j])
                assert step == np.float32(np.abs(tv).max() / np.float32(127))
                assert np.abs(oracle.dequant_q8(cv[b, h, j], cs[b, h, j]) - tv).max() <= step / 2 * (1 + 2 ** -20)
                vrow = oracle.widen(vn[b, h, t])
                assert np.abs(oracle.dequant_q8(vc[b, h, j], vs[b, h, j]) - vrow).max() <= float(vs[b, h, j]) / 2 * (1 + 2 ** -20)
    # untouched slots keep their sentinels: before each sequence's start and
    # past its end
    assert (cs[1, :, :5] == -1).all() and (cs[1, :, 7:] == -1).all() and (cs[0, :, 6:] == -1).all()
