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
# through D_i = dO_i . O_i, computed from the forward's O: ~1e-6 relative on
# the float32 path, ~1e-4 with bf16 V (float16 P in the forward), 2^-9 when
# O and dO are stored in bf16.  Each bound leaves a factor of ~10 over that.
TOL_GRAD = {(False, False): 1e-4, (True, False): 2e-3, (True, True): 2e-2}


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
