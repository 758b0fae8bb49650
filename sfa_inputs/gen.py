"""Seeded generators (see package docstring).  No method arithmetic here."""
from __future__ import annotations

import hashlib
import struct

import numpy as np
import torch

_MASK63 = (1 << 63) - 1


def slice_seed(seed: int, *tags) -> int:
    """Stable 63-bit seed for one tensor slice: sha256 of the seed and tags."""
    h = hashlib.sha256()
    h.update(struct.pack("<q", int(seed)))
    for t in tags:
        h.update(b"|")
        h.update(str(t).encode())
    return int.from_bytes(h.digest()[:8], "little") & _MASK63


def _gen(device, seed: int, *tags) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(slice_seed(seed, *tags))
    return g


def normal(shape, seed: int, *tags, device="cpu") -> torch.Tensor:
    """float32 N(0,1) tensor of `shape`, reproducible from (seed, tags, device)."""
    g = _gen(device, seed, *tags)
    return torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)


def to_bf16(x: torch.Tensor) -> torch.Tensor:
    """Input preparation: store a float32 draw as bfloat16 (torch rounds to
    nearest even).  Used for V and for V caches, whose *input* format is bf16."""
    return x.to(torch.bfloat16)


def dense_qkv(B, Hq, Hkv, n, d, seed, v_dtype=torch.bfloat16, device="cpu"):
    """Dense fp32 Q [B,Hq,n,d], K [B,Hkv,n,d] and V [B,Hkv,n,d] (v_dtype),
    each (b, h) slice drawn from its own seeded generator."""
    q = torch.empty((B, Hq, n, d), dtype=torch.float32, device=device)
    k = torch.empty((B, Hkv, n, d), dtype=torch.float32, device=device)
    v = torch.empty((B, Hkv, n, d), dtype=v_dtype, device=device)
    for b in range(B):
        for h in range(Hq):
            q[b, h] = normal((n, d), seed, "q", b, h, device=device)
        for h in range(Hkv):
            k[b, h] = normal((n, d), seed, "k", b, h, device=device)
            vv = normal((n, d), seed, "v", b, h, device=device)
            v[b, h] = vv if v_dtype == torch.float32 else vv.to(v_dtype)
    return q, k, v


def zipf_feature_perm(d: int, seed: int, head: int) -> torch.Tensor:
    """Per-head map from popularity rank (0 = most popular) to feature id."""
    g = _gen("cpu", seed, "zipf_perm", head)
    return torch.randperm(d, generator=g)


def zipf_codes(rows: int, d: int, k: int, s: float, perm: torch.Tensor,
               seed: int, *tags, device="cpu"):
    """k distinct feature ids per row, drawn without replacement with
    popularity weight w_r = (r+1)^-s over rank r, mapped through `perm`;
    values N(0,1) float32 with exact zeros replaced by 1.0.

    Sampling without replacement uses the Gumbel-top-k construction (keys
    log w_r + Gumbel noise, keep the k largest), which has the same
    distribution as drawing one feature at a time with probability
    proportional to the remaining weights.  Returns (idx int64 [rows,k]
    unsorted, val float32 [rows,k])."""
    g = _gen(device, seed, "zipf", *tags)
    ranks = torch.arange(1, d + 1, dtype=torch.float64, device=device)
    logw = (-s * torch.log(ranks)).to(torch.float32)
    u = torch.rand((rows, d), generator=g, device=device, dtype=torch.float32)
    u = u.clamp_(min=1e-30)
    gumbel = -torch.log(-torch.log(u).clamp_(max=-1e-30))
    keys = logw.unsqueeze(0) + gumbel
    rank_sel = torch.topk(keys, k, dim=1).indices
    idx = perm.to(device)[rank_sel]
    val = torch.randn((rows, k), generator=g, device=device, dtype=torch.float32)
    val = torch.where(val == 0, torch.ones_like(val), val)
    return idx, val


def dense_from_codes(idx: torch.Tensor, val: torch.Tensor, d: int) -> torch.Tensor:
    """Input construction: dense float32 rows that are zero off the given
    support and carry `val` on it."""
    out = torch.zeros(idx.shape[:-1] + (d,), dtype=torch.float32, device=idx.device)
    out.scatter_(-1, idx.long(), val)
    return out


def tie_rows(d: int, seed: int) -> np.ndarray:
    """A float32 [R, d] matrix of adversarial rows for the Top-k tie rule:
    all zeros, all equal, +-x pairs, +0/-0 mixes, subnormals, repeated
    magnitudes straddling every boundary, powers of two, and max floats."""
    rng = np.random.default_rng(slice_seed(seed, "ties"))
    rows = []
    rows.append(np.zeros(d, np.float32))
    rows.append(np.full(d, 1.5, np.float32))
    r = np.full(d, -2.0, np.float32); r[::2] = 2.0; rows.append(r)
    r = np.zeros(d, np.float32); r[1::3] = -0.0; r[::5] = 0.0; rows.append(r)
    r = np.zeros(d, np.float32); r[d // 2] = -0.0; r[d - 1] = 1e-45; rows.append(r)
    # subnormals of assorted magnitudes, both signs
    sub = (rng.integers(1, 1 << 23, size=d).astype(np.uint32)).view(np.float32)
    sign = rng.integers(0, 2, size=d).astype(bool)
    r = np.where(sign, -sub, sub).astype(np.float32); rows.append(r)
    # subnormals mixed with a few normals and zeros
    r = sub.copy(); r[::7] = 0.0; r[3::11] = 1.0; r[5::13] = -np.float32(1.17549435e-38); rows.append(r)
    # few distinct magnitudes -> many ties at every boundary
    for levels in (2, 3, 4, 8):
        mags = rng.integers(0, levels, size=d).astype(np.float32)
        sg = np.where(rng.integers(0, 2, size=d) == 1, -1.0, 1.0).astype(np.float32)
        rows.append((mags * sg).astype(np.float32))
    # powers of two, extreme magnitudes
    r = np.ldexp(np.ones(d, np.float32), rng.integers(-149, 127, size=d)).astype(np.float32)
    r[::3] *= -1; rows.append(r)
    r = np.full(d, np.finfo(np.float32).max, np.float32); r[1::2] *= -1; rows.append(r)
    # magnitudes at and just below powers of two (4, 2, 1.99999988, 1,
    # 0.99999994): the k-th largest lands on an exponent boundary
    for _ in range(2):
        levels = np.array([4.0, 2.0, np.float32(np.nextafter(np.float32(2), np.float32(0))),
                           np.float32(np.nextafter(np.float32(1), np.float32(0)))], np.float32)
        r = np.ones(d, np.float32)
        r[: 4 * (d // 8)] = np.repeat(levels, d // 8)
        r = r[rng.permutation(d)] * np.where(rng.integers(0, 2, size=d) == 1, -1, 1)
        rows.append(r.astype(np.float32))
    # one huge magnitude above ordinary ones
    r = rng.standard_normal(d).astype(np.float32); r[rng.integers(0, d)] = 3e30; rows.append(r)
    # ascending and descending magnitude ramps
    rows.append(np.arange(d, dtype=np.float32))
    rows.append(-np.arange(d, 0, -1, dtype=np.float32))
    # random rows with injected duplicate magnitudes
    for _ in range(16):
        r = rng.standard_normal(d).astype(np.float32)
        j = rng.integers(0, d, size=(d // 4, 2))
        r[j[:, 0]] = np.where(rng.integers(0, 2, size=d // 4) == 1, 1, -1) * np.abs(r[j[:, 1]])
        rows.append(r.astype(np.float32))
    return np.stack(rows).astype(np.float32)


def random_csr(rows: int, d: int, kmax: int, seed: int, *tags, min_len: int = 0):
    """A random CSR sparsity structure with values: row lengths uniform in
    [min_len, kmax] (row 0 empty and the last row full when rows > 1), distinct
    coordinates per row in random order, N(0,1) float32 values.  Returns numpy
    (indptr int32 [rows + 1], indices int64 [nnz], values float32 [nnz])."""
    rng = np.random.default_rng(slice_seed(seed, "csr", *tags))
    lens = rng.integers(min_len, kmax + 1, rows)
    if rows > 1:
        lens[0], lens[-1] = min_len, kmax
    indptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    indices = np.concatenate([rng.permutation(d)[:m] for m in lens] or [np.zeros(0)])
    values = rng.standard_normal(int(indptr[-1])).astype(np.float32)
    return indptr, indices.astype(np.int64), values
