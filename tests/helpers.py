"""Shared helpers for the GPU parity tests (tolerances, dtype plumbing)."""
import math

import numpy as np
import torch

# Tolerances (max-abs), fixed for this method's outputs:
#   float32 V path: O within 1e-5, bf16 V path (float32 output): O within 5e-3,
#   LSE within 1e-4 on every path.  A bf16 output is additionally allowed its
#   own rounding: half a bf16 ulp of the exact value.
TOL_O_F32 = 1e-5
TOL_O_BF16V = 5e-3
TOL_LSE = 1e-4

# Backward (no tolerance is fixed by the method): max |g - g_oracle| as a
# fraction of max |g_oracle| of the same tensor, keyed by (bf16 V, bf16 O and
# dO).  The products themselves carry ~2^-16; the error that dominates enters
# through D_i = dO_i . O_i, computed from the O the caller passes (the
# oracle's D is exact): ~1e-6 relative on the float32 path, ~1e-4 with bf16 V
# (float16 P in the forward), and with O stored in bf16 its rounding, unit
# roundoff 2^-8 (8 significant bits): D_i moves by up to 2^-8 sum_c |dO_ic
# O_ic|, which shifts dS_ij by P_ij times that and dq, dk by about 2^-8 of
# max |g| (measured <= 3.2e-3).  The float32 paths keep a factor of ~10 over
# their error; the bf16-O bound is 1.3 * 2^-8, with either V.
TOL_GRAD = {(False, False): 1e-4, (True, False): 2e-3, (True, True): 5e-3, (False, True): 5e-3}


def np_vals(t: torch.Tensor) -> np.ndarray:
    """float32 tensors -> float32 numpy; bf16 tensors -> uint16 bit patterns."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def np_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().float().double().numpy()


def bf16_half_ulp(x: np.ndarray) -> np.ndarray:
    """Half the spacing of bfloat16 numbers at |x| (8 significant bits)."""
    ax = np.maximum(np.abs(x), np.finfo(np.float32).tiny)
    e = np.floor(np.log2(ax))
    return 0.5 * np.exp2(e - 7)


def check_o(o_gpu: torch.Tensor, o_ref: np.ndarray, tol: float, what: str):
    got = np_f64(o_gpu)
    if o_gpu.dtype == torch.bfloat16:
        bound = tol + bf16_half_ulp(o_ref)
        bad = np.abs(got - o_ref) > bound
        assert not bad.any(), f"{what}: bf16 O off by more than tol+half-ulp at {np.argwhere(bad)[:5]}"
    err = np.abs(got - o_ref).max() if got.size else 0.0
    print(f"[parity] {what}: max|O-O_oracle| = {err:.3e} (tol {tol:.0e}, {o_gpu.dtype})", flush=True)
    if o_gpu.dtype != torch.bfloat16:
        assert err <= tol, f"{what}: max |O - O_oracle| = {err:.3e} > {tol:.1e}"
    return err


def check_lse(lse_gpu: torch.Tensor, lse_ref: np.ndarray, what: str, tol: float = TOL_LSE):
    got = np_f64(lse_gpu)
    err = np.abs(got - lse_ref).max() if got.size else 0.0
    print(f"[parity] {what}: max|LSE-LSE_oracle| = {err:.3e} (tol {tol:.0e})", flush=True)
    assert err <= tol, f"{what}: max |LSE - LSE_oracle| = {err:.3e} > {tol:.1e}"
    return err


def sample_rows(n: int, extra=(), count: int = 24, seed: int = 0, tile: int = 64):
    """Rows 0, 1, n-1, tile boundaries near the start and end, plus random rows."""
    rng = np.random.default_rng(seed)
    rows = {0, 1, n - 1, min(n - 1, tile - 1), min(n - 1, tile), max(0, n - tile), max(0, n - tile - 1)}
    rows |= {r for r in extra if 0 <= r < n}
    rows |= set(rng.integers(0, n, size=count).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def check_grad(g_gpu: torch.Tensor, g_ref: np.ndarray, tol: float, what: str):
    got = np_f64(g_gpu)
    scale = float(np.abs(g_ref).max()) if g_ref.size else 0.0
    err = float(np.abs(got - g_ref).max()) if got.size else 0.0
    rel = err / scale if scale > 0 else err
    print(f"[parity] {what}: max|g-g_oracle| = {err:.3e}, {rel:.2e} of max|g| = {scale:.3e} "
          f"(tol {tol:.0e})", flush=True)
    assert np.isfinite(got).all(), f"{what}: non-finite gradient"
    assert rel <= tol, f"{what}: max |g - g_oracle| / max |g| = {rel:.3e} > {tol:.1e}"
    return rel


# ---------------------------------------------------------------------------
# Running the oracle over many independent rows: the oracle's rows do not
# depend on each other (each query row's softmax is its own), so large
# samples are split across a thread pool.  The arithmetic is the oracle's;
# only the scheduling is here.  numpy's sorts and elementwise kernels release
# the GIL; BLAS is held to one thread per worker to avoid oversubscription.
# ---------------------------------------------------------------------------

import os as _os
from concurrent.futures import ThreadPoolExecutor as _Pool


def pool_size() -> int:
    try:
        n = len(_os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = _os.cpu_count() or 1
    return max(1, min(16, n))


def par_map(fn, items):
    from threadpoolctl import threadpool_limits
    items = list(items)
    with threadpool_limits(1):
        with _Pool(pool_size()) as ex:
            return list(ex.map(fn, items))


def oracle_topk_rows(x: np.ndarray, k: int, chunk: int = 8192):
    """oracle.topk_encode of every row of x [rows, d], in parallel chunks."""
    import oracle
    x = np.ascontiguousarray(x).reshape(-1, x.shape[-1])
    parts = [x[s:s + chunk] for s in range(0, x.shape[0], chunk)]
    res = par_map(lambda c: oracle.topk_encode(c, k), parts)
    if not res:
        return np.zeros((0, k), np.int64), np.zeros((0, k), np.float32)
    return np.concatenate([r[0] for r in res]), np.concatenate([r[1] for r in res])


def oracle_attn_rows(qd: np.ndarray, kd: np.ndarray, vv: np.ndarray, scale: float, causal: bool,
                     pos: np.ndarray, parts: int = 0, **kw):
    """oracle.softmax_attention of the query rows qd [r, d] at positions pos,
    split into interleaved parts that run in parallel; (O [r, dv], LSE [r])."""
    import oracle
    parts = parts or pool_size()
    pos = np.asarray(pos, dtype=np.int64)
    sl = [np.arange(s, len(pos), parts) for s in range(parts)]
    sl = [s for s in sl if s.size]
    res = par_map(lambda s: oracle.softmax_attention(qd[s], kd, vv, scale, causal, pos=pos[s],
                                                     row_chunk=256, **kw), sl)
    O = np.empty((len(pos), vv.shape[1]))
    L = np.empty(len(pos))
    for s, (o_, l_) in zip(sl, res):
        O[s], L[s] = o_, l_
    return O, L


def boundary_tie_rows(x: np.ndarray, k: int) -> np.ndarray:
    """Rows of x whose k-th and (k+1)-th largest magnitudes are equal (the
    Top-k tie rule decides which coordinate is kept)."""
    d = x.shape[-1]
    if k >= d:
        return np.zeros(0, np.int64)
    a = np.abs(x.reshape(-1, d).astype(np.float64))
    part = -np.partition(-a, [k - 1, k], axis=1)
    return np.flatnonzero(part[:, k - 1] == part[:, k])


def full_size_rows(n: int, seed: int, target: int = 4096, tile: int = 64) -> np.ndarray:
    """Query rows for full-size parity: 0, 1, n-1, both sides of every
    tile boundary (64m - 1, 64m), then random rows until `target`."""
    rows = {0, 1, n - 1}
    for m in range(1, (n + tile - 1) // tile):
        rows |= {tile * m - 1, tile * m}
    rng = np.random.default_rng(seed)
    extra = max(1024, target - len(rows)) if n > target else 0
    while extra > 0 and len(rows) < min(n, len(rows) + extra):
        before = len(rows)
        rows |= set(rng.integers(0, n, size=extra).tolist())
        extra -= len(rows) - before
    return np.array(sorted(r for r in rows if 0 <= r < n), dtype=np.int64)
