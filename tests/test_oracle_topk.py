"""Pins of the oracle's Top-k coding (Sec. 3.1, Eqs. (3)-(4)) and bf16 rounding.

Each test checks the oracle against something other than itself: a
hand-worked fixture, a brute-force enumeration of subsets, a library routine
on inputs where it is unambiguous, or an invariant of the definition.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle
from sfa_inputs import tie_rows

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _f(v):
    return np.float32(-0.0) if v == "-0.0" else np.float32(v)


def test_golden_ties():
    g = json.load(open(os.path.join(GOLDEN, "topk_ties.json")))
    x = np.array([_f(v) for v in g["x"]], dtype=np.float32)
    for case in g["cases"]:
        idx, val = oracle.topk_encode(x[None], case["k"])
        assert idx[0].tolist() == case["idx"]
        want = np.array([_f(v) for v in case["val"]], dtype=np.float32)
        assert val[0].view(np.uint32).tolist() == want.view(np.uint32).tolist()


def _brute_force_subset(x, k):
    """The unique k-subset S such that every kept u and every dropped w satisfy
    |x_u| > |x_w| or (|x_u| == |x_w| and u < w): found by enumeration."""
    d = len(x)
    mag = np.abs(x.astype(np.float64))
    found = []
    for S in itertools.combinations(range(d), k):
        Sset = set(S)
        ok = all(
            (mag[u] > mag[w]) or (mag[u] == mag[w] and u < w)
            for u in S for w in range(d) if w not in Sset
        )
        if ok:
            found.append(list(S))
    assert len(found) == 1
    return found[0]


def test_brute_force_small_rows():
    rng = np.random.default_rng(11)
    for trial in range(300):
        d = int(rng.integers(1, 9))
        k = int(rng.integers(1, d + 1))
        # few distinct magnitudes so that ties are common
        x = (rng.integers(-3, 4, size=d)).astype(np.float32)
        if trial % 3 == 0:
            x = rng.standard_normal(d).astype(np.float32)
        idx, val = oracle.topk_encode(x[None], k)
        assert idx[0].tolist() == _brute_force_subset(x, k)
        assert val[0].view(np.uint32).tolist() == x[idx[0]].view(np.uint32).tolist()


def test_matches_stable_argsort_on_tie_free_rows():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2000, 128)).astype(np.float32)
    mags = np.abs(x)
    tie_free = np.array([len(np.unique(r)) == r.size for r in mags])
    x = x[tie_free]
    for k in (1, 8, 16, 64, 128):
        idx, _ = oracle.topk_encode(x, k)
        ref = np.sort(np.argsort(-np.abs(x), axis=1, kind="stable")[:, :k], axis=1)
        assert np.array_equal(idx, ref)


def test_k1_is_argmax_lowest_index():
    rows = tie_rows(64, seed=3)
    idx, _ = oracle.topk_encode(rows, 1)
    # np.argmax returns the first (lowest-index) maximum
    assert np.array_equal(idx[:, 0], np.argmax(np.abs(rows.astype(np.float64)), axis=1))


def test_k_equals_d_keeps_everything():
    rows = tie_rows(32, seed=4)
    idx, val = oracle.topk_encode(rows, 32)
    assert np.array_equal(idx, np.broadcast_to(np.arange(32), idx.shape))
    assert np.array_equal(val.view(np.uint32), rows.view(np.uint32))


@pytest.mark.parametrize("d,k", [(64, 8), (64, 16), (128, 16), (128, 8), (128, 1), (64, 63)])
def test_invariants_on_tie_suite(d, k):
    rows = np.concatenate([tie_rows(d, seed=d + k),
                           np.random.default_rng(d * k).standard_normal((64, d)).astype(np.float32)])
    idx, val = oracle.topk_encode(rows, k)
    assert idx.shape == (rows.shape[0], k)
    assert np.all(np.diff(idx, axis=1) > 0)          # distinct and ascending
    assert idx.min() >= 0 and idx.max() < d
    assert np.array_equal(val.view(np.uint32),
                          np.take_along_axis(rows, idx, 1).view(np.uint32))
    mag = np.abs(rows.astype(np.float64))
    for r in range(rows.shape[0]):
        kept = set(idx[r].tolist())
        min_kept = min((mag[r, u], -u) for u in kept)
        for w in range(d):
            if w not in kept:
                assert (mag[r, w], -w) < min_kept


def test_subnormals_are_ordered_not_flushed():
    x = np.array([[1e-45, 2e-45, 0.0, -3e-45, 1e-44, -0.0, 5e-45, 1e-45]], np.float32)
    idx, _ = oracle.topk_encode(x, 3)
    assert idx[0].tolist() == [3, 4, 6]


def test_bf16_golden():
    g = json.load(open(os.path.join(GOLDEN, "bf16_rne.json")))
    src = np.array([int(c[0], 16) for c in g["cases"]], dtype=np.uint32).view(np.float32)
    want = [int(c[1], 16) for c in g["cases"]]
    assert oracle.bf16_rne(src).tolist() == want


def test_bf16_matches_torch_rounding():
    rng = np.random.default_rng(9)
    bits = rng.integers(0, 1 << 32, size=200000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    got = oracle.bf16_rne(x)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, ref)


def test_topk_bf16_selects_on_fp32_magnitudes():
    # 1.0 and 1.00390625 round to the same bf16 value; selection must still
    # prefer the larger float32 magnitude.
    x = np.array([[1.0, 1.00390625, 0.5, 0.25]], np.float32)
    idx, val = oracle.topk_encode_bf16(x, 1)
    assert idx[0].tolist() == [1]
    assert val[0].tolist() == [0x3F80]
