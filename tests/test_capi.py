"""The C-ABI library: loads, exports every entry point include/sfa.h declares,
and rejects bad arguments on the host, before anything is launched (so these
run without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sfa.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sfa_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    import paper_2603_22300_amd as sfa
    if not os.path.exists(sfa.library_path):
        from paper_2603_22300_amd.build import build
        build()
    return sfa.lib()


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert {"sfa_topk_encode", "sfa_attn_fwd", "sfa_attn_fwd_workspace", "sfa_attn_fwd_index",
            "sfa_attn_bwd", "sfa_attn_bwd_workspace",
            "sfa_attn_decode", "sfa_attn_decode_workspace", "sfa_abi_version",
            "sfa_strerror"} <= set(names)
    for nm in names:
        assert hasattr(L, nm), nm


def test_version_and_strerror(L):
    assert L.sfa_abi_version() == 4
    for s in range(5):
        assert L.sfa_strerror(s)


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation


def _fwd(L, fn="sfa_attn_fwd", **kw):
    a = dict(q_idx=FAKE, q_val=FAKE, k_idx=FAKE, k_val=FAKE, v=FAKE, B=1, Hq=4, Hkv=2, n=16, d=64,
             k=8, causal=1)
    if fn == "sfa_attn_fwd":
        a.update(window=0, n_global=0)
    a.update(scale=0.125, idx_t=0, qk_val_t=2, v_t=3, o_t=2, o=FAKE, lse=None)
    if fn == "sfa_attn_fwd":
        a.update(ws=FAKE, ws_bytes=ctypes.c_size_t(1 << 40))
    a["stream"] = None
    a.update(kw)
    return getattr(L, fn)(*a.values())


@pytest.mark.parametrize("fn", ["sfa_attn_fwd", "sfa_attn_fwd_index"])
def test_fwd_validation(L, fn):
    assert _fwd(L, fn, q_idx=None) == 1
    assert _fwd(L, fn, o=None) == 1
    assert _fwd(L, fn, k=0) == 1
    assert _fwd(L, fn, k=65, d=64) == 1
    assert _fwd(L, fn, Hq=3, Hkv=2) == 1
    assert _fwd(L, fn, n=0) == 1
    assert _fwd(L, fn, idx_t=2) == 1            # a value dtype as index dtype
    assert _fwd(L, fn, v_t=0) == 1
    assert _fwd(L, fn, scale=float("nan")) == 1
    assert _fwd(L, fn, d=300, k=8) == 2          # beyond the largest head dim, 256
    if fn == "sfa_attn_fwd_index":
        assert _fwd(L, fn, d=96, k=8) == 2       # the index variant: d in {64, 128}
    else:
        # other head dims take the float32 vector kernel, one query head per
        # grid row: B * Hq is bounded by the grid
        assert _fwd(L, fn, d=96, k=8, B=40000, Hq=2, Hkv=1) == 2
    if fn == "sfa_attn_fwd_index":
        assert _fwd(L, fn, Hq=12, Hkv=4) == 2    # group of 3 heads: the index tables need 2^m
    else:
        # a group of 3 heads at d = 64 runs the float32 kernel: its grid bound
        # on B * Hq applies (and rejects before any launch)
        assert _fwd(L, fn, B=6000, Hq=12, Hkv=4) == 2
    assert _fwd(L, fn, B=70000, Hkv=1, Hq=1) == 2  # grid limit
    assert _fwd(L, fn, n=(1 << 22) + 1, d=128, k=16) == 2  # 32-bit per-head offsets


def test_window_validation(L):
    assert _fwd(L, window=-1) == 1
    assert _fwd(L, window=4, n_global=-2) == 1
    assert _dec(L, window=-3) == 1
    assert _bwd(L, window=-1) == 1
    assert _paged(L, n_global=-1, ws_bytes=ctypes.c_size_t(1 << 30)) == 1


def test_fwd_workspace(L):
    need = L.sfa_attn_fwd_workspace(1, 2, 16, 64, 3)
    assert need > 0                                          # bf16 V: float16 V tiles + flags
    assert L.sfa_attn_fwd_workspace(1, 2, 16, 64, 2) == 0    # float32 V needs none
    assert L.sfa_attn_fwd_workspace(1, 2, 16, 96, 3) == 0    # unsupported head dim
    assert L.sfa_attn_fwd_workspace(0, 2, 16, 64, 3) == 0
    big = L.sfa_attn_fwd_workspace(2, 8, 32768, 128, 3)
    assert big >= 2 * 8 * 512 * 128 * 68 * 2                # one float16 V^T tile per key tile
    assert _fwd(L, ws_bytes=ctypes.c_size_t(need - 1)) == 4
    assert _fwd(L, ws=None) == 4


def test_fwd_index_limits(L):
    assert _fwd(L, "sfa_attn_fwd_index", d=128, k=128) == 2   # index tables exceed LDS


def test_encode_validation(L):
    enc = L.sfa_topk_encode
    assert enc(FAKE, 10, 64, 0, FAKE, 0, FAKE, 2, None) == 1
    assert enc(FAKE, 10, 64, 65, FAKE, 0, FAKE, 2, None) == 1
    assert enc(None, 10, 64, 8, FAKE, 0, FAKE, 2, None) == 1
    assert enc(FAKE, -1, 64, 8, FAKE, 0, FAKE, 2, None) == 1
    assert enc(FAKE, 10, 64, 8, FAKE, 3, FAKE, 2, None) == 1
    assert enc(FAKE, 10, 300, 8, FAKE, 0, FAKE, 2, None) == 2
    assert enc(None, 0, 64, 8, None, 0, None, 2, None) == 0     # empty: no-op


def _dec(L, **kw):
    a = dict(q_idx=FAKE, q_val=FAKE, kc_idx=FAKE, kc_val=FAKE, v=FAKE, seq_len=None, B=2, Hq=8,
             Hkv=2, Lmax=100, d=128, k=16, scale=0.088, window=0, n_global=0, q_idx_t=0,
             q_val_t=2, kc_idx_t=1,
             kc_val_t=3, v_t=3, o_t=2, o=FAKE, lse=None, ws=FAKE, ws_bytes=1 << 30, stream=None)
    a.update(kw)
    return L.sfa_attn_decode(*a.values())


def test_decode_validation_and_workspace(L):
    need = L.sfa_attn_decode_workspace(2, 8, 100, 128)
    assert need > 0
    assert L.sfa_attn_decode_workspace(0, 8, 100, 128) == 0
    assert _dec(L, ws_bytes=need - 1) == 4
    assert _dec(L, ws=None) == 1
    assert _dec(L, Hq=6, Hkv=4) == 1
    assert _dec(L, Hq=32, Hkv=2) == 2       # group of 16 heads: unsupported
    assert _dec(L, d=300, k=8) == 2          # beyond the largest head dim, 256
    # other head dims run the float32 decode: group size up to 8, any value
    assert _dec(L, d=80, k=8, Hq=18, Hkv=2) == 2
    assert _dec(L, d=80, k=8, ws_bytes=L.sfa_attn_decode_workspace(2, 8, 100, 80) - 1) == 4
    assert _dec(L, kc_idx_t=3) == 1


def _bwd(L, **kw):
    a = dict(q_idx=FAKE, q_val=FAKE, k_idx=FAKE, k_val=FAKE, v=FAKE, o=FAKE, lse=FAKE, dout=FAKE,
             B=1, Hq=4, Hkv=2, n=16, d=64, k=8, causal=1, window=0, n_global=0, scale=0.125,
             idx_t=0, qk_val_t=2,
             v_t=3, o_t=3, dq=FAKE, dk=FAKE, dv=FAKE, ws=FAKE, ws_bytes=ctypes.c_size_t(1 << 40),
             stream=None)
    a.update(kw)
    return L.sfa_attn_bwd(*a.values())


def test_bwd_validation_and_workspace(L):
    need = L.sfa_attn_bwd_workspace(1, 4, 2, 16, 64)
    assert need > 0
    assert L.sfa_attn_bwd_workspace(1, 4, 2, 16, 96) == 0
    assert _bwd(L, ws_bytes=ctypes.c_size_t(need - 1)) == 4
    assert _bwd(L, ws=None) == 4
    assert _bwd(L, lse=None) == 1
    assert _bwd(L, dout=None) == 1
    assert _bwd(L, dq=None) == 1
    assert _bwd(L, k=0) == 1
    assert _bwd(L, Hq=3, Hkv=2) == 1
    # a group of 16 heads runs the float32 backward: its grid bound on B * Hq
    assert _bwd(L, B=4000, Hq=32, Hkv=2) == 2
    assert _bwd(L, d=300, k=8) == 2                 # beyond the largest head dim, 256
    assert _bwd(L, d=96, k=8, B=40000, Hq=2, Hkv=1) == 2  # float32 backward: grid bound on B * Hq


def _paged(L, **kw):
    a = dict(q=None, q_idx=FAKE, q_val=FAKE, kc_idx=FAKE, kc_val=FAKE, v_cache=FAKE,
             block_table=FAKE, max_pages=4, page_size=64, num_pages=16, seq_len=None, B=2, Hq=8,
             Hkv=2, d=128, k=16, scale=0.1, window=0, n_global=0, q_idx_t=0, q_val_t=2,
             kc_idx_t=1, kc_val_t=3, v_t=3,
             o_t=2, o=FAKE, lse=None, ws=FAKE, ws_bytes=ctypes.c_size_t(1), stream=None)
    a.update(kw)
    return L.sfa_attn_decode_paged(*a.values())


def test_decode_paged_validation(L):
    need = L.sfa_attn_decode_workspace(2, 8, 4 * 64, 128)
    assert _paged(L) == 4                            # workspace too small, checked last
    assert _paged(L, ws_bytes=ctypes.c_size_t(need - 1)) == 4
    ok = dict(ws_bytes=ctypes.c_size_t(need))
    assert _paged(L, q=FAKE, **ok) == 1              # dense query and codes both given
    assert _paged(L, q_idx=None, **ok) == 1          # neither complete
    assert _paged(L, block_table=None, **ok) == 1
    assert _paged(L, page_size=48, **ok) == 1        # not a power of two
    assert _paged(L, page_size=8, **ok) == 1         # below 16
    assert _paged(L, max_pages=0, **ok) == 1
    assert _paged(L, num_pages=0, **ok) == 1
    assert _paged(L, max_pages=1 << 25, page_size=64, **ok) == 1  # capacity beyond 2^30
    assert _paged(L, Hq=6, Hkv=4, **ok) == 1
    assert _paged(L, Hq=32, Hkv=2, **ok) == 2
    assert _paged(L, d=300, k=8, **ok) == 2
    assert _paged(L, d=96, k=8, Hq=18, Hkv=2, **ok) == 2   # float32 decode: group <= 8
    assert _paged(L, kc_val_t=1, **ok) == 1
    assert _paged(L, q=FAKE, q_idx=None, q_val=None, q_idx_t=7, o=None, **ok) == 1  # o missing


def _append(L, **kw):
    a = dict(k_new=FAKE, v_new=FAKE, n_new=None, seq_len=FAKE, B=2, Hkv=2, T=3, d=128, k=16,
             block_table=None, max_pages=0, page_size=100, num_pages=0, kc_idx=FAKE, kc_val=FAKE,
             v_cache=FAKE, kc_idx_t=1, kc_val_t=3, v_new_t=3, v_t=3, stream=None)
    a.update(kw)
    return L.sfa_kv_append(*a.values())


def test_kv_append_validation(L):
    assert _append(L, seq_len=None) == 1
    assert _append(L, k_new=None) == 1
    assert _append(L, kc_idx=None) == 1
    assert _append(L, k=0) == 1
    assert _append(L, k=129) == 1
    assert _append(L, T=-1) == 1
    assert _append(L, page_size=0) == 1
    assert _append(L, block_table=FAKE, max_pages=0, num_pages=4) == 1
    assert _append(L, block_table=FAKE, max_pages=1 << 21, num_pages=4, page_size=1024) == 1
    assert _append(L, block_table=FAKE, max_pages=4, num_pages=4, page_size=48) == 1  # paged: power of two
    assert _append(L, kc_idx_t=2) == 1
    assert _append(L, v_new_t=0) == 1
    assert _append(L, d=300, k=8) == 2


def _csr(L, **kw):
    a = dict(indptr=FAKE, indices=FAKE, indices_t=4, values=FAKE, values_t=5, rows=10, d=128,
             kmax=16, idx=FAKE, idx_t=4, val=FAKE, stream=None)
    a.update(kw)
    return L.sfa_csr_to_codes(*a.values())


def test_csr_to_codes_validation(L):
    assert _csr(L, rows=0, indptr=None) == 0      # empty: no-op before pointer checks
    assert _csr(L, indptr=None) == 1
    assert _csr(L, kmax=0) == 1
    assert _csr(L, kmax=129) == 1                 # kmax > d
    assert _csr(L, rows=-1) == 1
    assert _csr(L, indices_t=2) == 1              # a value dtype as index dtype
    assert _csr(L, values_t=0) == 1               # an index dtype as value dtype
    assert _csr(L, idx_t=5) == 1
    assert _csr(L, d=300, kmax=8) == 2


def test_compact_dtypes_accepted_for_codes_only(L):
    # U8 indices / F16 code values pass validation of the forward up to the
    # workspace check; F16 is not a V or O dtype
    assert _fwd(L, idx_t=4, qk_val_t=5, ws_bytes=ctypes.c_size_t(0)) == 4
    assert _fwd(L, idx_t=4, qk_val_t=5, v_t=5) == 1
    assert _fwd(L, o_t=5) == 1
    assert _dec(L, kc_idx_t=4, kc_val_t=5, ws_bytes=1) == 4
    assert _dec(L, v_t=5) == 1


def test_decode_noalloc_host_checks(L):
    # the allocation-free decode rejects, before any HIP call: partials beyond
    # its static scratch (SFA_ENOSPC) and null pointers (SFA_EINVAL)
    B, Hq, Hkv, Lmax, d, k = 64, 32, 8, 1 << 17, 128, 16
    assert L.sfa_attn_decode_workspace(B, Hq, Lmax, d) > 32 << 20
    args = [FAKE, FAKE, FAKE, FAKE, FAKE, None, B, Hq, Hkv, Lmax, d, k, ctypes.c_float(0.088), 0,
            0, 0, 2, 1, 3, 3, 2, FAKE, None, None]
    assert L.sfa_attn_decode_noalloc(*args) == 4
    args[6], args[9] = 1, 4096
    args[0] = None
    assert L.sfa_attn_decode_noalloc(*args) == 1


def test_q8_cache_host_checks(L):
    # 8-bit cache entry points: rejections before any launch
    app = [FAKE, FAKE, None, FAKE, 2, 2, 3, 128, 16, None, 0, 100, 0, FAKE, FAKE, FAKE, FAKE, FAKE,
           1, 3, None]
    a = list(app); a[13] = None                    # kc_idx missing
    assert L.sfa_kv_append_q8(*a) == 1
    a = list(app); a[8] = 129                      # k > d
    assert L.sfa_kv_append_q8(*a) == 1
    a = list(app); a[7], a[8] = 300, 8             # d beyond 256
    assert L.sfa_kv_append_q8(*a) == 2
    dec = [None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0, 4096, 0, None, 2, 8, 2, 128, 16,
           ctypes.c_float(0.088), 0, 0, 0, 2, 1, 2, FAKE, None, FAKE, ctypes.c_size_t(1 << 40), None]
    a = list(dec); a[0] = FAKE                     # dense query and codes together
    assert L.sfa_attn_decode_q8(*a) == 1
    a = list(dec); a[17] = 12                      # k without the vector path
    assert L.sfa_attn_decode_q8(*a) == 2
    a = list(dec); a[16], a[17] = 96, 8            # head dim without the tuned kernel
    assert L.sfa_attn_decode_q8(*a) == 2
    a = list(dec); a[23] = 0                       # int32 cache indices
    assert L.sfa_attn_decode_q8(*a) == 2
    a = list(dec); a[14] = 12                      # group of 6
    assert L.sfa_attn_decode_q8(*a) == 2
    a = list(dec); a[28] = ctypes.c_size_t(16)     # workspace too small
    assert L.sfa_attn_decode_q8(*a) == 4
