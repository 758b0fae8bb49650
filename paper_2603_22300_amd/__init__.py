"""Python binding of libsfa (Sparse Feature Attention on gfx950).

Argument marshalling only: every function here checks tensor placement,
shapes and dtypes, allocates outputs with torch when the caller passes none,
and calls the C entry point of the same name in libsfa.so on torch's current
stream.  All arithmetic happens in the HIP kernels.  There is no fallback:
if libsfa.so is missing or the device is not a GPU, the call raises.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

__all__ = [
    "SfaError", "lib", "library_path", "sfa_abi_version", "sfa_strerror",
    "sfa_topk_encode", "sfa_attn_fwd_workspace", "sfa_attn_fwd", "sfa_attn_fwd_index",
    "sfa_attn_bwd_workspace", "sfa_attn_bwd",
    "sfa_attn_decode_workspace", "sfa_attn_decode", "sfa_attn_decode_noalloc",
    "sfa_attn_decode_paged", "sfa_kv_append", "sfa_kv_append_q8", "sfa_attn_decode_q8",
    "sfa_csr_to_codes",
    "SFA_OK", "SFA_EINVAL", "SFA_ENOTSUP", "SFA_EHIP", "SFA_ENOSPC",
    "SFA_I32", "SFA_I16", "SFA_F32", "SFA_BF16", "SFA_U8", "SFA_F16",
]

SFA_OK, SFA_EINVAL, SFA_ENOTSUP, SFA_EHIP, SFA_ENOSPC = 0, 1, 2, 3, 4
SFA_I32, SFA_I16, SFA_F32, SFA_BF16, SFA_U8, SFA_F16 = 0, 1, 2, 3, 4, 5

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libsfa.so")

_lib = None


class SfaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {sfa_strerror(status)} (status {status})")


def lib() -> ctypes.CDLL:
    """The loaded libsfa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(library_path):
            raise RuntimeError(
                f"{library_path} is missing: build it with `python -m paper_2603_22300_amd.build`")
        L = ctypes.CDLL(library_path)
        vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
        L.sfa_abi_version.restype = i32
        L.sfa_abi_version.argtypes = []
        L.sfa_strerror.restype = ctypes.c_char_p
        L.sfa_strerror.argtypes = [i32]
        L.sfa_topk_encode.restype = i32
        L.sfa_topk_encode.argtypes = [vp, i64, i32, i32, vp, i32, vp, i32, vp]
        L.sfa_attn_fwd.restype = i32
        L.sfa_attn_fwd.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32,
                                   i32, f32, i32, i32, i32, i32, vp, vp, vp, sz, vp]
        L.sfa_attn_fwd_workspace.restype = sz
        L.sfa_attn_fwd_workspace.argtypes = [i32, i32, i32, i32, i32]
        L.sfa_attn_fwd_index.restype = i32
        L.sfa_attn_fwd_index.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32,
                                         f32, i32, i32, i32, i32, vp, vp, vp]
        L.sfa_attn_bwd.restype = i32
        L.sfa_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                   i32, i32, i32, f32, i32, i32, i32, i32, vp, vp, vp, vp, sz, vp]
        L.sfa_attn_bwd_workspace.restype = sz
        L.sfa_attn_bwd_workspace.argtypes = [i32, i32, i32, i32, i32]
        L.sfa_attn_decode_workspace.restype = sz
        L.sfa_attn_decode_workspace.argtypes = [i32, i32, i32, i32]
        L.sfa_attn_decode.restype = i32
        L.sfa_attn_decode.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, f32,
                                      i32, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, sz, vp]
        L.sfa_attn_decode_noalloc.restype = i32
        L.sfa_attn_decode_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                              f32, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp,
                                              vp]
        L.sfa_attn_decode_paged.restype = i32
        L.sfa_attn_decode_paged.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, vp, i32, i32,
                                            i32, i32, i32, f32, i32, i32, i32, i32, i32, i32,
                                            i32, i32, vp, vp, vp, sz, vp]
        L.sfa_kv_append.restype = i32
        L.sfa_kv_append.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, vp, i32, i32, i32,
                                    vp, vp, vp, i32, i32, i32, i32, vp]
        L.sfa_kv_append_q8.restype = i32
        L.sfa_kv_append_q8.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, vp, i32, i32, i32,
                                       vp, vp, vp, vp, vp, i32, i32, vp]
        L.sfa_attn_decode_q8.restype = i32
        L.sfa_attn_decode_q8.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, vp,
                                         i32, i32, i32, i32, i32, f32, i32, i32, i32, i32, i32,
                                         i32, vp, vp, vp, sz, vp]
        L.sfa_csr_to_codes.restype = i32
        L.sfa_csr_to_codes.argtypes = [vp, vp, i32, vp, i32, i64, i32, i32, vp, i32, vp, vp]
        _lib = L
    return _lib


def sfa_abi_version() -> int:
    return lib().sfa_abi_version()


def sfa_strerror(status: int) -> str:
    return lib().sfa_strerror(status).decode()


# code indices; code values; V and O
_IDX = {torch.int32: SFA_I32, torch.int16: SFA_I16, torch.uint8: SFA_U8}
_CVAL = {torch.float32: SFA_F32, torch.bfloat16: SFA_BF16, torch.float16: SFA_F16}
_VAL = {torch.float32: SFA_F32, torch.bfloat16: SFA_BF16}


def _check(t: torch.Tensor, name: str, table) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype not in table:
        raise TypeError(f"{name}: unsupported dtype {t.dtype}")
    return table[t.dtype]


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _call(status: int, where: str):
    if status != SFA_OK:
        raise SfaError(status, where)


def sfa_topk_encode(x: torch.Tensor, k: int, idx_dtype=torch.int32, val_dtype=torch.float32,
                    idx: torch.Tensor | None = None, val: torch.Tensor | None = None):
    """Row Top-k codes of x [..., d] float32: (idx [..., k], val [..., k])."""
    _check(x, "x", {torch.float32: SFA_F32})
    d = x.shape[-1]
    rows = x.numel() // d if d else 0
    if idx is None:
        idx = torch.empty(x.shape[:-1] + (k,), dtype=idx_dtype, device=x.device)
    if val is None:
        val = torch.empty(x.shape[:-1] + (k,), dtype=val_dtype, device=x.device)
    it = _check(idx, "idx", _IDX)
    vt = _check(val, "val", _CVAL)
    if idx.numel() != rows * k or val.numel() != rows * k:
        raise ValueError("idx/val must hold rows * k elements")
    _call(lib().sfa_topk_encode(x.data_ptr(), rows, d, k, idx.data_ptr(), it, val.data_ptr(), vt,
                                _stream(x)), "sfa_topk_encode")
    return idx, val


def sfa_attn_fwd_workspace(B: int, Hkv: int, n: int, d: int, v_dtype=torch.bfloat16) -> int:
    """Bytes of device workspace sfa_attn_fwd needs (0 for float32 V)."""
    return int(lib().sfa_attn_fwd_workspace(B, Hkv, n, d, _VAL[v_dtype]))


def sfa_attn_fwd(q_idx, q_val, k_idx, k_val, v, causal: bool = True, scale: float | None = None,
                 o_dtype=None, o: torch.Tensor | None = None, lse: torch.Tensor | None = None,
                 want_lse: bool = True, ws: torch.Tensor | None = None, window: int = 0,
                 n_global: int = 0):
    """SFA forward on codes.  q_* [B, Hq, n, k], k_* [B, Hkv, n, k], v [B, Hkv, n, d].
    ws: uint8 device workspace of sfa_attn_fwd_workspace(...) bytes, allocated
    here when None.  window > 0: sliding window |i - j| < window plus n_global
    leading global tokens.  Returns (o [B, Hq, n, d], lse [B, Hq, n] float32 or
    None)."""
    return _fwd("sfa_attn_fwd", q_idx, q_val, k_idx, k_val, v, causal, scale, o_dtype, o, lse,
                want_lse, ws, window, n_global)


def sfa_attn_fwd_index(q_idx, q_val, k_idx, k_val, v, causal: bool = True,
                       scale: float | None = None, o_dtype=None, o: torch.Tensor | None = None,
                       lse: torch.Tensor | None = None, want_lse: bool = True):
    """The inverted-index variant of sfa_attn_fwd (same arguments and results)."""
    return _fwd("sfa_attn_fwd_index", q_idx, q_val, k_idx, k_val, v, causal, scale, o_dtype, o,
                lse, want_lse, None, 0, 0)


def _fwd(name, q_idx, q_val, k_idx, k_val, v, causal, scale, o_dtype, o, lse, want_lse, ws,
         window, n_global):
    B, Hq, n, k = q_idx.shape
    Hkv, d = k_idx.shape[1], v.shape[-1]
    if tuple(q_val.shape) != (B, Hq, n, k) or tuple(k_idx.shape) != (B, Hkv, n, k) \
            or tuple(k_val.shape) != (B, Hkv, n, k) or tuple(v.shape) != (B, Hkv, n, d):
        raise ValueError("inconsistent shapes")
    if q_idx.dtype != k_idx.dtype or q_val.dtype != k_val.dtype:
        raise TypeError("query and key codes must share index and value dtypes")
    it = _check(q_idx, "q_idx", _IDX); _check(k_idx, "k_idx", _IDX)
    qt = _check(q_val, "q_val", _CVAL); _check(k_val, "k_val", _CVAL)
    vt = _check(v, "v", _VAL)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if o is None:
        o = torch.empty((B, Hq, n, d), dtype=o_dtype or v.dtype, device=v.device)
    ot = _check(o, "o", _VAL)
    if tuple(o.shape) != (B, Hq, n, d):
        raise ValueError("o has the wrong shape")
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, n), dtype=torch.float32, device=v.device)
    lp = 0
    if lse is not None:
        _check(lse, "lse", {torch.float32: SFA_F32})
        lp = lse.data_ptr()
    mask = [int(bool(causal))]
    if name == "sfa_attn_fwd":
        mask += [int(window), int(n_global)]
    args = [q_idx.data_ptr(), q_val.data_ptr(), k_idx.data_ptr(), k_val.data_ptr(), v.data_ptr(),
            B, Hq, Hkv, n, d, k] + mask + [float(scale), it, qt, vt, ot, o.data_ptr(), lp]
    if name == "sfa_attn_fwd":
        need = int(lib().sfa_attn_fwd_workspace(B, Hkv, n, d, vt))
        if ws is None and need > 0:
            ws = torch.empty(need, dtype=torch.uint8, device=v.device)
        if ws is not None:
            if ws.device.type != "cuda" or not ws.is_contiguous():
                raise ValueError("ws must be a contiguous GPU tensor")
            args += [ws.data_ptr(), ws.numel() * ws.element_size()]
        else:
            args += [0, 0]
    _call(getattr(lib(), name)(*args, _stream(v)), name)
    return o, lse


def sfa_attn_bwd_workspace(B: int, Hq: int, Hkv: int, n: int, d: int) -> int:
    """Bytes of device workspace sfa_attn_bwd needs."""
    return int(lib().sfa_attn_bwd_workspace(B, Hq, Hkv, n, d))


def sfa_attn_bwd(q_idx, q_val, k_idx, k_val, v, o, lse, dout, causal: bool = True,
                 scale: float | None = None, dq: torch.Tensor | None = None,
                 dk: torch.Tensor | None = None, dv: torch.Tensor | None = None,
                 ws: torch.Tensor | None = None, window: int = 0, n_global: int = 0):
    """SFA backward (straight-through estimator).  Shapes as sfa_attn_fwd, and
    the same causal / window / n_global as the forward that gave o and lse;
    o, dout [B, Hq, n, d] (same dtype), lse [B, Hq, n] float32.  Returns
    (dq_val [B, Hq, n, k], dk_val [B, Hkv, n, k], dv [B, Hkv, n, d]), float32:
    the gradients of the code values (Eq. (6): zero off the supports)."""
    B, Hq, n, k = q_idx.shape
    Hkv, d = k_idx.shape[1], v.shape[-1]
    if tuple(q_val.shape) != (B, Hq, n, k) or tuple(k_idx.shape) != (B, Hkv, n, k) \
            or tuple(k_val.shape) != (B, Hkv, n, k) or tuple(v.shape) != (B, Hkv, n, d) \
            or tuple(o.shape) != (B, Hq, n, d) or tuple(dout.shape) != (B, Hq, n, d) \
            or tuple(lse.shape) != (B, Hq, n):
        raise ValueError("inconsistent shapes")
    if q_idx.dtype != k_idx.dtype or q_val.dtype != k_val.dtype or o.dtype != dout.dtype:
        raise TypeError("query/key codes, and o/dout, must share dtypes")
    it = _check(q_idx, "q_idx", _IDX); _check(k_idx, "k_idx", _IDX)
    qt = _check(q_val, "q_val", _CVAL); _check(k_val, "k_val", _CVAL)
    vt = _check(v, "v", _VAL)
    ot = _check(o, "o", _VAL); _check(dout, "dout", _VAL)
    _check(lse, "lse", {torch.float32: SFA_F32})
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    f32 = dict(dtype=torch.float32, device=v.device)
    dq = torch.empty((B, Hq, n, k), **f32) if dq is None else dq
    dk = torch.empty((B, Hkv, n, k), **f32) if dk is None else dk
    dv = torch.empty((B, Hkv, n, d), **f32) if dv is None else dv
    for t, name, shape in ((dq, "dq", (B, Hq, n, k)), (dk, "dk", (B, Hkv, n, k)),
                           (dv, "dv", (B, Hkv, n, d))):
        _check(t, name, {torch.float32: SFA_F32})
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has the wrong shape")
    if ws is None:
        ws = torch.empty(sfa_attn_bwd_workspace(B, Hq, Hkv, n, d), dtype=torch.uint8,
                         device=v.device)
    if ws.device.type != "cuda" or not ws.is_contiguous():
        raise ValueError("ws must be a contiguous GPU tensor")
    _call(lib().sfa_attn_bwd(q_idx.data_ptr(), q_val.data_ptr(), k_idx.data_ptr(),
                             k_val.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                             dout.data_ptr(), B, Hq, Hkv, n, d, k, int(bool(causal)),
                             int(window), int(n_global), float(scale), it, qt, vt, ot,
                             dq.data_ptr(), dk.data_ptr(),
                             dv.data_ptr(), ws.data_ptr(), ws.numel() * ws.element_size(),
                             _stream(v)), "sfa_attn_bwd")
    return dq, dk, dv


def sfa_attn_decode_workspace(B: int, Hq: int, Lmax: int, d: int) -> int:
    return int(lib().sfa_attn_decode_workspace(B, Hq, Lmax, d))


def sfa_attn_decode(q_idx, q_val, kc_idx, kc_val, v_cache, seq_len=None, scale: float | None = None,
                    o_dtype=None, o=None, lse=None, want_lse: bool = True, ws=None,
                    window: int = 0, n_global: int = 0):
    """SFA decode step.  q_* [B, Hq, k], kc_* [B, Hkv, Lmax, k], v_cache [B, Hkv, Lmax, d],
    seq_len int32 [B] on the GPU or None.  Returns (o [B, Hq, d], lse [B, Hq] or None)."""
    B, Hq, k = q_idx.shape
    Hkv, Lmax, d = kc_idx.shape[1], kc_idx.shape[2], v_cache.shape[-1]
    if tuple(q_val.shape) != (B, Hq, k) or tuple(kc_idx.shape) != (B, Hkv, Lmax, k) \
            or tuple(kc_val.shape) != (B, Hkv, Lmax, k) or tuple(v_cache.shape) != (B, Hkv, Lmax, d):
        raise ValueError("inconsistent shapes")
    qit = _check(q_idx, "q_idx", _IDX); qvt = _check(q_val, "q_val", _CVAL)
    cit = _check(kc_idx, "kc_idx", _IDX); cvt = _check(kc_val, "kc_val", _CVAL)
    vt = _check(v_cache, "v_cache", _VAL)
    sp = 0
    if seq_len is not None:
        _check(seq_len, "seq_len", {torch.int32: SFA_I32})
        if seq_len.numel() != B:
            raise ValueError("seq_len must hold B entries")
        sp = seq_len.data_ptr()
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if o is None:
        o = torch.empty((B, Hq, d), dtype=o_dtype or v_cache.dtype, device=v_cache.device)
    ot = _check(o, "o", _VAL)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=v_cache.device)
    lp = 0
    if lse is not None:
        _check(lse, "lse", {torch.float32: SFA_F32})
        lp = lse.data_ptr()
    need = sfa_attn_decode_workspace(B, Hq, Lmax, d)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=v_cache.device)
    _call(lib().sfa_attn_decode(q_idx.data_ptr(), q_val.data_ptr(), kc_idx.data_ptr(),
                                kc_val.data_ptr(), v_cache.data_ptr(), sp, B, Hq, Hkv, Lmax, d, k,
                                float(scale), int(window), int(n_global), qit, qvt, cit, cvt, vt,
                                ot, o.data_ptr(), lp,
                                ws.data_ptr(), ws.numel() * ws.element_size(), _stream(v_cache)),
          "sfa_attn_decode")
    return o, lse


def sfa_attn_decode_noalloc(q_idx, q_val, kc_idx, kc_val, v_cache, o, lse=None, seq_len=None,
                            scale: float | None = None, window: int = 0, n_global: int = 0):
    """sfa_attn_decode on the library's static device scratch: no workspace and
    no allocation, so the outputs o [B, Hq, d] (and lse [B, Hq] float32, or
    None) are the caller's.  Calls that overlap in time on one GPU race on the
    scratch."""
    B, Hq, k = q_idx.shape
    Hkv, Lmax, d = kc_idx.shape[1], kc_idx.shape[2], v_cache.shape[-1]
    if tuple(q_val.shape) != (B, Hq, k) or tuple(kc_idx.shape) != (B, Hkv, Lmax, k) \
            or tuple(kc_val.shape) != (B, Hkv, Lmax, k) or tuple(v_cache.shape) != (B, Hkv, Lmax, d) \
            or tuple(o.shape) != (B, Hq, d):
        raise ValueError("inconsistent shapes")
    qit = _check(q_idx, "q_idx", _IDX); qvt = _check(q_val, "q_val", _CVAL)
    cit = _check(kc_idx, "kc_idx", _IDX); cvt = _check(kc_val, "kc_val", _CVAL)
    vt = _check(v_cache, "v_cache", _VAL); ot = _check(o, "o", _VAL)
    sp = 0
    if seq_len is not None:
        _check(seq_len, "seq_len", {torch.int32: SFA_I32})
        if seq_len.numel() != B:
            raise ValueError("seq_len must hold B entries")
        sp = seq_len.data_ptr()
    lp = 0
    if lse is not None:
        _check(lse, "lse", {torch.float32: SFA_F32})
        if lse.numel() != B * Hq:
            raise ValueError("lse must hold B * Hq entries")
        lp = lse.data_ptr()
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    _call(lib().sfa_attn_decode_noalloc(q_idx.data_ptr(), q_val.data_ptr(), kc_idx.data_ptr(),
                                        kc_val.data_ptr(), v_cache.data_ptr(), sp, B, Hq, Hkv,
                                        Lmax, d, k, float(scale), int(window), int(n_global), qit,
                                        qvt, cit, cvt, vt, ot, o.data_ptr(), lp, _stream(v_cache)),
          "sfa_attn_decode_noalloc")
    return o, lse


def _i32_vec(t, name: str, n: int) -> int:
    _check(t, name, {torch.int32: SFA_I32})
    if t.numel() != n:
        raise ValueError(f"{name} must hold {n} entries")
    return t.data_ptr()


def sfa_kv_append(k_new, v_new, seq_len, kc_idx, kc_val, v_cache, k: int, block_table=None,
                  n_new=None):
    """Append coded keys and values to a KV cache, in place, and advance seq_len.

    k_new float32 [B, Hkv, T, d]; v_new [B, Hkv, T, d] (float32 or bf16);
    seq_len int32 [B] (in/out).  Contiguous cache (block_table None):
    kc_* [B, Hkv, Lmax, k], v_cache [B, Hkv, Lmax, d].  Paged cache:
    kc_* [num_pages, Hkv, page_size, k], v_cache [num_pages, Hkv, page_size, d],
    block_table int32 [B, max_pages].  n_new int32 [B] or None (= T)."""
    B, Hkv, T, d = k_new.shape
    _check(k_new, "k_new", {torch.float32: SFA_F32})
    vnt = _check(v_new, "v_new", _VAL)
    if tuple(v_new.shape) != (B, Hkv, T, d):
        raise ValueError("v_new must match k_new")
    cit = _check(kc_idx, "kc_idx", _IDX); cvt = _check(kc_val, "kc_val", _CVAL)
    vt = _check(v_cache, "v_cache", _VAL)
    npg, P = kc_idx.shape[0], kc_idx.shape[2]
    if tuple(kc_idx.shape) != (npg, Hkv, P, k) or tuple(kc_val.shape) != (npg, Hkv, P, k) \
            or tuple(v_cache.shape) != (npg, Hkv, P, d):
        raise ValueError("inconsistent cache shapes")
    sp = _i32_vec(seq_len, "seq_len", B)
    tp, maxp = 0, 1
    if block_table is not None:
        _check(block_table, "block_table", {torch.int32: SFA_I32})
        if block_table.dim() != 2 or block_table.shape[0] != B:
            raise ValueError("block_table must be [B, max_pages]")
        tp, maxp = block_table.data_ptr(), block_table.shape[1]
    elif npg != B:
        raise ValueError("a contiguous cache holds B sequences")
    npp = 0 if n_new is None else _i32_vec(n_new, "n_new", B)
    _call(lib().sfa_kv_append(k_new.data_ptr(), v_new.data_ptr(), npp, sp, B, Hkv, T, d, k, tp,
                              maxp, P, npg, kc_idx.data_ptr(), kc_val.data_ptr(),
                              v_cache.data_ptr(), cit, cvt, vnt, vt, _stream(k_new)),
          "sfa_kv_append")
    return seq_len


def sfa_attn_decode_paged(kc_idx, kc_val, v_cache, block_table, seq_len=None, q=None, q_idx=None,
                          q_val=None, scale: float | None = None, o_dtype=None, o=None, lse=None,
                          want_lse: bool = True, ws=None, window: int = 0, n_global: int = 0):
    """SFA decode step over a paged cache.  Give either the dense query q
    (float32 [B, Hq, d], coded inside the kernel) or its codes q_idx, q_val
    [B, Hq, k].  kc_* [num_pages, Hkv, page_size, k], v_cache
    [num_pages, Hkv, page_size, d], block_table int32 [B, max_pages],
    seq_len int32 [B] or None.  Returns (o [B, Hq, d], lse [B, Hq] or None)."""
    npg, Hkv, P, k = kc_idx.shape
    d = v_cache.shape[-1]
    if tuple(kc_val.shape) != (npg, Hkv, P, k) or tuple(v_cache.shape) != (npg, Hkv, P, d):
        raise ValueError("inconsistent cache shapes")
    cit = _check(kc_idx, "kc_idx", _IDX); cvt = _check(kc_val, "kc_val", _CVAL)
    vt = _check(v_cache, "v_cache", _VAL)
    _check(block_table, "block_table", {torch.int32: SFA_I32})
    if block_table.dim() != 2:
        raise ValueError("block_table must be [B, max_pages]")
    B, maxp = block_table.shape
    qp = qip = qvp = 0
    qit = qvt = 0
    if q is not None:
        if q_idx is not None or q_val is not None:
            raise ValueError("give either q or (q_idx, q_val)")
        _check(q, "q", {torch.float32: SFA_F32})
        if q.dim() != 3 or q.shape[0] != B or q.shape[2] != d:
            raise ValueError("q must be [B, Hq, d]")
        Hq = q.shape[1]
        qp = q.data_ptr()
    else:
        qit = _check(q_idx, "q_idx", _IDX); qvt = _check(q_val, "q_val", _CVAL)
        if q_idx.dim() != 3 or tuple(q_idx.shape) != (B, q_idx.shape[1], k) \
                or tuple(q_val.shape) != tuple(q_idx.shape):
            raise ValueError("q codes must be [B, Hq, k]")
        Hq = q_idx.shape[1]
        qip, qvp = q_idx.data_ptr(), q_val.data_ptr()
    sp = 0 if seq_len is None else _i32_vec(seq_len, "seq_len", B)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if o is None:
        o = torch.empty((B, Hq, d), dtype=o_dtype or v_cache.dtype, device=v_cache.device)
    ot = _check(o, "o", _VAL)
    if tuple(o.shape) != (B, Hq, d):
        raise ValueError("o has the wrong shape")
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=v_cache.device)
    lp = 0
    if lse is not None:
        _check(lse, "lse", {torch.float32: SFA_F32})
        lp = lse.data_ptr()
    if ws is None:
        ws = torch.empty(sfa_attn_decode_workspace(B, Hq, maxp * P, d), dtype=torch.uint8,
                         device=v_cache.device)
    _call(lib().sfa_attn_decode_paged(qp, qip, qvp, kc_idx.data_ptr(), kc_val.data_ptr(),
                                      v_cache.data_ptr(), block_table.data_ptr(), maxp, P, npg,
                                      sp, B, Hq, Hkv, d, k, float(scale), int(window),
                                      int(n_global), qit, qvt, cit, cvt, vt,
                                      ot, o.data_ptr(), lp, ws.data_ptr(),
                                      ws.numel() * ws.element_size(), _stream(v_cache)),
          "sfa_attn_decode_paged")
    return o, lse


def sfa_kv_append_q8(k_new, v_new, seq_len, kc_idx, kc_val, kc_scale, v_cache, v_scale, k: int,
                     block_table=None, n_new=None):
    """Append to an 8-bit cache (int8 code values and value rows, a float32
    scale per row).  k_new [B, Hkv, T, d] float32, v_new [B, Hkv, T, d] float32
    or bf16; contiguous cache kc_idx [B, Hkv, Lmax, k], kc_val int8 [B, Hkv,
    Lmax, k], kc_scale [B, Hkv, Lmax], v_cache int8 [B, Hkv, Lmax, d], v_scale
    [B, Hkv, Lmax]; or paged [num_pages, Hkv, P, ...] with block_table [B,
    max_pages].  seq_len int32 [B] on the GPU is advanced in place."""
    B, Hkv, T, d = k_new.shape
    _check(k_new, "k_new", {torch.float32: SFA_F32})
    vt = _check(v_new, "v_new", _VAL)
    cit = _check(kc_idx, "kc_idx", _IDX)
    _check(kc_val, "kc_val", {torch.int8: 0}); _check(v_cache, "v_cache", {torch.int8: 0})
    _check(kc_scale, "kc_scale", {torch.float32: SFA_F32})
    _check(v_scale, "v_scale", {torch.float32: SFA_F32})
    P = kc_idx.shape[2]
    if tuple(kc_val.shape) != tuple(kc_idx.shape) or kc_idx.shape[3] != k \
            or tuple(v_cache.shape) != tuple(kc_idx.shape[:3]) + (d,) \
            or tuple(kc_scale.shape) != tuple(kc_idx.shape[:3]) \
            or tuple(v_scale.shape) != tuple(kc_idx.shape[:3]):
        raise ValueError("inconsistent cache shapes")
    sp = _i32_vec(seq_len, "seq_len", B)
    np_ = _i32_vec(n_new, "n_new", B) if n_new is not None else 0
    tp, max_pages, num_pages = 0, 0, 0
    if block_table is not None:
        _check(block_table, "block_table", {torch.int32: SFA_I32})
        tp, max_pages, num_pages = block_table.data_ptr(), block_table.shape[1], kc_idx.shape[0]
    elif kc_idx.shape[0] != B:
        raise ValueError("contiguous cache: first dimension must be B")
    _call(lib().sfa_kv_append_q8(k_new.data_ptr(), v_new.data_ptr(), np_, sp, B, Hkv, T, d, k, tp,
                                 max_pages, P, num_pages, kc_idx.data_ptr(), kc_val.data_ptr(),
                                 kc_scale.data_ptr(), v_cache.data_ptr(), v_scale.data_ptr(), cit,
                                 vt, _stream(k_new)), "sfa_kv_append_q8")


def sfa_attn_decode_q8(kc_idx, kc_val, kc_scale, v_cache, v_scale, block_table=None, seq_len=None,
                       q=None, q_idx=None, q_val=None, Hq=None, scale: float | None = None,
                       o_dtype=torch.float32, o=None, lse=None, want_lse: bool = True, ws=None,
                       window: int = 0, n_global: int = 0):
    """Decode over an 8-bit cache (contiguous, or paged with block_table), with
    query codes q_idx / q_val [B, Hq, k] or a dense float32 query q [B, Hq, d]
    coded in the kernel.  Returns (o [B, Hq, d], lse [B, Hq] or None)."""
    Hkv, P, k = kc_idx.shape[1], kc_idx.shape[2], kc_idx.shape[3]
    d = v_cache.shape[-1]
    if q is not None:
        B, Hq, _ = q.shape
        _check(q, "q", {torch.float32: SFA_F32})
        qp, qip, qvp, qit, qvt = q.data_ptr(), 0, 0, 0, 0
    else:
        B, Hq, _ = q_idx.shape
        qit = _check(q_idx, "q_idx", _IDX); qvt = _check(q_val, "q_val", _CVAL)
        qp, qip, qvp = 0, q_idx.data_ptr(), q_val.data_ptr()
    cit = _check(kc_idx, "kc_idx", _IDX)
    _check(kc_val, "kc_val", {torch.int8: 0}); _check(v_cache, "v_cache", {torch.int8: 0})
    _check(kc_scale, "kc_scale", {torch.float32: SFA_F32})
    _check(v_scale, "v_scale", {torch.float32: SFA_F32})
    tp, max_pages, num_pages = 0, 0, 0
    if block_table is not None:
        _check(block_table, "block_table", {torch.int32: SFA_I32})
        tp, max_pages, num_pages = block_table.data_ptr(), block_table.shape[1], kc_idx.shape[0]
        cap = max_pages * P
    else:
        if kc_idx.shape[0] != B:
            raise ValueError("contiguous cache: first dimension must be B")
        cap = P
    sp = _i32_vec(seq_len, "seq_len", B) if seq_len is not None else 0
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if o is None:
        o = torch.empty((B, Hq, d), dtype=o_dtype, device=v_cache.device)
    ot = _check(o, "o", _VAL)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=v_cache.device)
    lp = lse.data_ptr() if lse is not None else 0
    if ws is None:
        ws = torch.empty(sfa_attn_decode_workspace(B, Hq, cap, d), dtype=torch.uint8,
                         device=v_cache.device)
    _call(lib().sfa_attn_decode_q8(qp, qip, qvp, kc_idx.data_ptr(), kc_val.data_ptr(),
                                   kc_scale.data_ptr(), v_cache.data_ptr(), v_scale.data_ptr(), tp,
                                   max_pages, P, num_pages, sp, B, Hq, Hkv, d, k, float(scale),
                                   int(window), int(n_global), qit, qvt, cit, ot, o.data_ptr(), lp,
                                   ws.data_ptr(), ws.numel() * ws.element_size(), _stream(v_cache)),
          "sfa_attn_decode_q8")
    return o, lse


def sfa_csr_to_codes(indptr, indices, values, d: int, kmax: int, idx_dtype=None, idx=None,
                     val=None):
    """CSR codes (indptr int32 [rows + 1], indices [nnz], values [nnz]) to fixed
    rows (idx [rows, kmax] of idx_dtype, default the indices' dtype; val
    [rows, kmax] of the values' dtype), padded with zeros at the lowest free
    coordinates.  Returns (idx, val)."""
    _check(indptr, "indptr", {torch.int32: SFA_I32})
    if indptr.dim() != 1 or indptr.numel() < 1:
        raise ValueError("indptr must be 1-D with rows + 1 entries")
    rows = indptr.numel() - 1
    iit = _check(indices, "indices", _IDX)
    vit = _check(values, "values", _CVAL)
    if idx is None:
        idx = torch.empty((rows, kmax), dtype=idx_dtype or indices.dtype, device=indptr.device)
    if val is None:
        val = torch.empty((rows, kmax), dtype=values.dtype, device=indptr.device)
    it = _check(idx, "idx", _IDX)
    if _check(val, "val", _CVAL) != vit:
        raise TypeError("val must have the values' dtype")
    if idx.numel() != rows * kmax or val.numel() != rows * kmax:
        raise ValueError("idx and val must hold rows * kmax entries")
    _call(lib().sfa_csr_to_codes(indptr.data_ptr(), indices.data_ptr(), iit, values.data_ptr(),
                                 vit, rows, d, kmax, idx.data_ptr(), it, val.data_ptr(),
                                 _stream(indptr)), "sfa_csr_to_codes")
    return idx, val
