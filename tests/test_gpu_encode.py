"""GPU parity: sfa_topk_encode against the oracle's Top-k, bit for bit
(indices and values), through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_22300_amd as sfa
import sfa_inputs as si
from helpers import np_vals

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _encode_and_check(x_cpu: np.ndarray, k: int):
    x = torch.from_numpy(x_cpu).to(DEV)
    ri, rv = oracle.topk_encode(x_cpu, k)
    bi, bv = oracle.topk_encode_bf16(x_cpu, k)
    gi, gv = sfa.sfa_topk_encode(x, k)
    hi, hv = sfa.sfa_topk_encode(x, k, idx_dtype=torch.int16, val_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert np.array_equal(gi.cpu().numpy(), ri)
    assert np.array_equal(np_vals(gv).view(np.uint32), rv.view(np.uint32))
    assert np.array_equal(hi.cpu().numpy().astype(np.int64), bi)
    assert np.array_equal(np_vals(hv), bv)


@pytest.mark.parametrize("d,k", [(64, 8), (64, 16), (128, 16), (128, 8), (128, 1), (128, 128),
                                 (64, 64), (100, 7), (256, 32), (33, 33), (1, 1), (200, 199)])
def test_random_rows(d, k):
    x = si.normal((3001, d), 17, "enc", d, k).numpy()
    _encode_and_check(x, k)


@pytest.mark.parametrize("d,k", [(64, 1), (64, 8), (64, 16), (128, 16), (128, 64), (128, 127),
                                 (256, 40)])
def test_tie_suite(d, k):
    _encode_and_check(si.tie_rows(d, seed=d * 1000 + k), k)


def test_empty_is_noop():
    x = torch.empty((0, 64), device=DEV)
    gi, gv = sfa.sfa_topk_encode(x, 8)
    assert gi.shape == (0, 8)


def test_qwen3_queries_full_size_sampled():
    # the full 32-head x 32K x 128 query tensor of the 32K workload, coded on
    # the GPU; 20000 random rows + the first rows of every head are checked
    w = si.workload("qwen3_32k")
    q = torch.empty((w.Hq, w.n, w.d), device=DEV)
    for h in range(w.Hq):
        q[h] = si.normal((w.n, w.d), w.seed, "q", 0, h, device=DEV)
    gi, gv = sfa.sfa_topk_encode(q, w.k)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    flat = q.view(-1, w.d)
    rows = np.unique(np.concatenate([rng.integers(0, flat.shape[0], 20000),
                                     (np.arange(w.Hq)[:, None] * w.n + np.arange(64)[None]).ravel()]))
    xr = flat[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    ri, rv = oracle.topk_encode(xr, w.k)
    gi_s = gi.view(-1, w.k)[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    gv_s = np_vals(gv.view(-1, w.k)[torch.from_numpy(rows).to(DEV)])
    assert np.array_equal(gi_s, ri)
    assert np.array_equal(gv_s.view(np.uint32), rv.view(np.uint32))
