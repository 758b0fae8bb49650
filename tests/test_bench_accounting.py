"""The benchmark's algorithmic accounting (allowed pairs, overlap products E,
decode keys) against the oracle's token mask, counted pair by pair on small
inputs."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


@pytest.mark.parametrize("causal,w,g", [(True, 0, 0), (False, 0, 0), (True, 50, 0), (True, 50, 7),
                                        (False, 40, 3), (True, 1, 0), (True, 50, 80)])
def test_pairs_and_overlaps(causal, w, g):
    n, d, k, G = 300, 32, 4, 2
    gen = torch.Generator().manual_seed(w + g)
    qi = torch.stack([torch.randperm(d, generator=gen)[:k] for _ in range(2 * n)]).reshape(1, 2, n, k)
    ki = torch.stack([torch.randperm(d, generator=gen)[:k] for _ in range(n)]).reshape(1, 1, n, k)
    m = oracle.token_mask(np.arange(n), n, causal, w, g)
    qd = np.zeros((2, n, d)); kd = np.zeros((n, d))
    np.put_along_axis(qd, qi[0].numpy(), 1, -1)
    np.put_along_axis(kd, ki[0, 0].numpy(), 1, -1)
    E = int(sum(((qd[h] @ kd.T) * m).sum() for h in range(2)))
    assert bench._overlap_count(qi, ki, d, G, causal, w, g) == E
    assert bench._allowed_pairs(n, causal, w, g) == int(m.sum())


@pytest.mark.parametrize("L,w,g", [(100, 0, 0), (100, 30, 0), (100, 30, 5), (100, 30, 80), (3, 30, 5)])
def test_decode_keys(L, w, g):
    assert bench._decode_keys(L, w, g) == int(oracle.token_mask([L - 1], L, True, w, g).sum())
