"""The seeded input generator: determinism, per-slice regeneration, and the
Zipf support sampler's marginals."""
import numpy as np
import torch

import oracle
import sfa_inputs as si


def test_slices_are_deterministic_and_independent():
    a = si.normal((4, 8), 3, "q", 0, 1)
    b = si.normal((4, 8), 3, "q", 0, 1)
    c = si.normal((4, 8), 3, "q", 0, 2)
    assert torch.equal(a, b) and not torch.equal(a, c)
    q, k, v = si.dense_qkv(2, 4, 2, 16, 8, seed=7)
    assert torch.equal(q[1, 3], si.normal((16, 8), 7, "q", 1, 3))
    assert torch.equal(v[0, 1], si.normal((16, 8), 7, "v", 0, 1).to(torch.bfloat16))


def test_zipf_first_draw_marginal():
    # the first feature of a row is drawn with probability w_r / sum(w)
    d, s = 16, 1.1
    perm = torch.arange(d)
    rows = 200000
    idx, _ = si.zipf_codes(rows, d, 1, s, perm, 1, "t")
    w = np.arange(1, d + 1, dtype=np.float64) ** -s
    p = w / w.sum()
    freq = np.bincount(idx[:, 0].numpy(), minlength=d) / rows
    sd = np.sqrt(p * (1 - p) / rows)
    assert np.all(np.abs(freq - p) < 5 * sd)


def test_zipf_second_draw_is_without_replacement():
    # P(rank 0 and rank 1 are the two picks of k=2) = p0*p1/(1-p0) + p1*p0/(1-p1)
    d, s = 8, 1.1
    rows = 200000
    idx, _ = si.zipf_codes(rows, d, 2, s, torch.arange(d), 2, "t")
    w = np.arange(1, d + 1, dtype=np.float64) ** -s
    p = w / w.sum()
    want = p[0] * p[1] / (1 - p[0]) + p[1] * p[0] / (1 - p[1])
    pairs = np.sort(idx.numpy(), axis=1)
    got = np.mean((pairs[:, 0] == 0) & (pairs[:, 1] == 1))
    assert abs(got - want) < 5 * np.sqrt(want * (1 - want) / rows)
    assert np.all(pairs[:, 0] != pairs[:, 1])


def test_dense_rows_from_codes_reencode_to_the_codes():
    d, k = 128, 8
    perm = si.zipf_feature_perm(d, 4, 0)
    idx, val = si.zipf_codes(500, d, k, 1.1, perm, 4, "k", 0, 0)
    x = si.dense_from_codes(idx, val, d).numpy()
    oi, ov = oracle.topk_encode(x, k)
    order = np.argsort(idx.numpy(), axis=1)
    assert np.array_equal(oi, np.take_along_axis(idx.numpy(), order, 1))
    assert np.array_equal(ov, np.take_along_axis(val.numpy(), order, 1))
