// C ABI of libsfa: argument validation, dtype dispatch, launch, error codes.
// Every check runs on the host before anything is enqueued.
#include <hip/hip_runtime.h>
#include <math.h>

#include "../../include/sfa.h"
#include "sfa_device.h"
#include "sfa_launch.h"

namespace {

constexpr int kAbiVersion = 4;
constexpr int kMaxLds = 160 * 1024;  // LDS per workgroup on gfx950

// index arrays of codes; values of codes; V and O
bool is_idx(int t) { return t == SFA_I32 || t == SFA_I16 || t == SFA_U8; }
bool is_cval(int t) { return t == SFA_F32 || t == SFA_BF16 || t == SFA_F16; }
bool is_val(int t) { return t == SFA_F32 || t == SFA_BF16; }
// kernel-side format codes (sfa_device.h)
int ifmt_of(int t) { return t == SFA_I16 ? sfa::kIdxI16 : (t == SFA_U8 ? sfa::kIdxU8 : sfa::kIdxI32); }
int vfmt_of(int t) { return t == SFA_BF16 ? sfa::kValBF16 : (t == SFA_F16 ? sfa::kValF16 : sfa::kValF32); }
bool pow2_le(int g, int maxg) { return g >= 1 && g <= maxg && (g & (g - 1)) == 0; }

sfa_status from_hip(hipError_t e) { return e == hipSuccess ? SFA_OK : SFA_EHIP; }

}  // namespace

extern "C" {

int sfa_abi_version(void) { return kAbiVersion; }

const char* sfa_strerror(int status) {
  switch (status) {
    case SFA_OK: return "ok";
    case SFA_EINVAL: return "invalid argument";
    case SFA_ENOTSUP: return "unsupported shape or dtype";
    case SFA_EHIP: return "HIP runtime error";
    case SFA_ENOSPC: return "workspace too small";
    default: return "unknown status";
  }
}

sfa_status sfa_topk_encode(const float* x, int64_t rows, int d, int k, void* idx, int idx_t,
                           void* val, int val_t, void* stream) {
  if (rows < 0 || d < 1 || k < 1 || k > d) return SFA_EINVAL;
  if (!is_idx(idx_t) || !is_cval(val_t)) return SFA_EINVAL;
  if (d > 256) return SFA_ENOTSUP;
  if (rows == 0) return SFA_OK;
  if (!x || !idx || !val) return SFA_EINVAL;
  if ((rows + 3) / 4 > 0x7fffffffLL) return SFA_ENOTSUP;
  return from_hip(sfa::launch_topk_encode(x, rows, d, k, idx, ifmt_of(idx_t), val,
                                          vfmt_of(val_t), (hipStream_t)stream));
}

namespace {

sfa_status check_fwd(const void* q_idx, const void* q_val, const void* k_idx, const void* k_val,
                     const void* v, int B, int Hq, int Hkv, int n, int d, int k, float scale,
                     int idx_t, int qk_val_t, int v_t, int o_t, const void* o) {
  if (!q_idx || !q_val || !k_idx || !k_val || !v || !o) return SFA_EINVAL;
  if (B < 1 || Hq < 1 || Hkv < 1 || n < 1 || d < 1 || k < 1 || k > d) return SFA_EINVAL;
  if (Hq % Hkv != 0) return SFA_EINVAL;
  if (!is_idx(idx_t) || !is_cval(qk_val_t) || !is_val(v_t) || !is_val(o_t)) return SFA_EINVAL;
  if (!isfinite(scale)) return SFA_EINVAL;
  if (d > 256) return SFA_ENOTSUP;  // callers with matrix-core kernels only also require 64 or 128
  if ((long long)B * Hkv > 65535) return SFA_ENOTSUP;
  // per-head code and value offsets are 32-bit byte offsets in the kernels
  if ((long long)n * d > (1LL << 29) || (long long)n * k > (1LL << 29)) return SFA_ENOTSUP;
  return SFA_OK;
}

}  // namespace

size_t sfa_attn_fwd_workspace(int B, int Hkv, int n, int d, int v_t) {
  if (B < 1 || Hkv < 1 || n < 1 || (d != 64 && d != 128) || !is_val(v_t)) return 0;
  return sfa::fwd_workspace_bytes(B, Hkv, n, d, v_t == SFA_BF16);
}

sfa_status sfa_attn_fwd(const void* q_idx, const void* q_val, const void* k_idx,
                        const void* k_val, const void* v, int B, int Hq, int Hkv, int n, int d,
                        int k, int causal, int window, int n_global, float scale, int idx_t,
                        int qk_val_t, int v_t, int o_t, void* o, float* lse, void* ws,
                        size_t ws_bytes, void* stream) {
  sfa_status st = check_fwd(q_idx, q_val, k_idx, k_val, v, B, Hq, Hkv, n, d, k, scale, idx_t,
                            qk_val_t, v_t, o_t, o);
  if (st != SFA_OK) return st;
  if (window < 0 || n_global < 0) return SFA_EINVAL;
  if ((d != 64 && d != 128) || !pow2_le(Hq / Hkv, sfa::fwd_max_group())) {
    // head dimensions or group sizes without a matrix-core kernel: the
    // float32 vector-unit forward (any group size, no workspace)
    if (!sfa::fwd_generic_supported(d, k) || (long long)B * Hq > 65535) return SFA_ENOTSUP;
    return from_hip(sfa::launch_attn_fwd_generic(q_idx, q_val, k_idx, k_val, v, B, Hq, Hkv, n, d,
                                                 k, causal != 0, window,
                                                 window > 0 ? n_global : 0, scale,
                                                 ifmt_of(idx_t), vfmt_of(qk_val_t),
                                                 v_t == SFA_BF16, o_t == SFA_BF16, o, lse,
                                                 (hipStream_t)stream));
  }
  const size_t need = sfa::fwd_workspace_bytes(B, Hkv, n, d, v_t == SFA_BF16);
  if (need > 0 && (ws == nullptr || ws_bytes < need)) return SFA_ENOSPC;
  return from_hip(sfa::launch_attn_fwd(q_idx, q_val, k_idx, k_val, v, B, Hq, Hkv, n, d, k,
                                       causal != 0, window, window > 0 ? n_global : 0, scale,
                                       ifmt_of(idx_t),
                                       vfmt_of(qk_val_t), v_t == SFA_BF16, o_t == SFA_BF16,
                                       o, lse, ws, (hipStream_t)stream));
}

size_t sfa_attn_bwd_workspace(int B, int Hq, int Hkv, int n, int d) {
  if (B < 1 || Hq < 1 || Hkv < 1 || n < 1 || (d != 64 && d != 128)) return 0;
  return sfa::bwd_workspace_bytes(B, Hq, Hkv, n, d);
}

sfa_status sfa_attn_bwd(const void* q_idx, const void* q_val, const void* k_idx,
                        const void* k_val, const void* v, const void* o, const float* lse,
                        const void* dout, int B, int Hq, int Hkv, int n, int d, int k, int causal,
                        int window, int n_global, float scale, int idx_t, int qk_val_t, int v_t,
                        int o_t, float* dq_val,
                        float* dk_val, float* dv, void* ws, size_t ws_bytes, void* stream) {
  sfa_status st = check_fwd(q_idx, q_val, k_idx, k_val, v, B, Hq, Hkv, n, d, k, scale, idx_t,
                            qk_val_t, v_t, o_t, o);
  if (st != SFA_OK) return st;
  if (!lse || !dout || !dq_val || !dk_val || !dv) return SFA_EINVAL;
  if (window < 0 || n_global < 0) return SFA_EINVAL;
  if ((d != 64 && d != 128) || !pow2_le(Hq / Hkv, sfa::bwd_max_group())) {
    // head dimensions or group sizes without the matrix-core kernels: the
    // float32 backward (any group size, no workspace)
    if (!sfa::bwd_generic_supported(d, k) || (long long)B * Hq > 65535) return SFA_ENOTSUP;
    return from_hip(sfa::launch_attn_bwd_generic(
        q_idx, q_val, k_idx, k_val, v, o, lse, dout, B, Hq, Hkv, n, d, k, causal != 0, window,
        window > 0 ? n_global : 0, scale, ifmt_of(idx_t), vfmt_of(qk_val_t), v_t == SFA_BF16,
        o_t == SFA_BF16, dq_val, dk_val, dv, (hipStream_t)stream));
  }
  if (ws == nullptr || ws_bytes < sfa::bwd_workspace_bytes(B, Hq, Hkv, n, d)) return SFA_ENOSPC;
  return from_hip(sfa::launch_attn_bwd(q_idx, q_val, k_idx, k_val, v, o, lse, dout, B, Hq, Hkv, n,
                                       d, k, causal != 0, window, window > 0 ? n_global : 0,
                                       scale, ifmt_of(idx_t),
                                       vfmt_of(qk_val_t), v_t == SFA_BF16, o_t == SFA_BF16,
                                       dq_val, dk_val, dv, ws, (hipStream_t)stream));
}

sfa_status sfa_attn_fwd_index(const void* q_idx, const void* q_val, const void* k_idx,
                              const void* k_val, const void* v, int B, int Hq, int Hkv, int n,
                              int d, int k, int causal, float scale, int idx_t, int qk_val_t,
                              int v_t, int o_t, void* o, float* lse, void* stream) {
  sfa_status st = check_fwd(q_idx, q_val, k_idx, k_val, v, B, Hq, Hkv, n, d, k, scale, idx_t,
                            qk_val_t, v_t, o_t, o);
  if (st != SFA_OK) return st;
  if (d != 64 && d != 128) return SFA_ENOTSUP;
  if (!pow2_le(Hq / Hkv, sfa::fwd_index_rows_per_block())) return SFA_ENOTSUP;
  if (k > sfa::fwd_index_max_k()) return SFA_ENOTSUP;
  if (sfa::fwd_index_lds_bytes(d, k, v_t == SFA_BF16) > kMaxLds) return SFA_ENOTSUP;
  return from_hip(sfa::launch_attn_fwd_index(q_idx, q_val, k_idx, k_val, v, B, Hq, Hkv, n, d, k,
                                             causal != 0, scale, ifmt_of(idx_t),
                                             vfmt_of(qk_val_t), v_t == SFA_BF16,
                                             o_t == SFA_BF16, o, lse, (hipStream_t)stream));
}

size_t sfa_attn_decode_workspace(int B, int Hq, int Lmax, int d) {
  if (B < 1 || Hq < 1 || Lmax < 1 || d < 1) return 0;
  return sfa::decode_workspace_bytes(B, Hq, Lmax, d);
}

}  // extern "C"

namespace {

// Contiguous-cache decode behind sfa_attn_decode and sfa_attn_decode_noalloc.
// ws == nullptr selects the library's static device scratch (after every
// argument check, and only if the partials fit it).
sfa_status decode_contiguous(const void* q_idx, const void* q_val, const void* kc_idx,
                             const void* kc_val, const void* v_cache, const int32_t* seq_len,
                             int B, int Hq, int Hkv, int Lmax, int d, int k, float scale,
                             int window, int n_global, int q_idx_t, int q_val_t, int kc_idx_t,
                             int kc_val_t, int v_t, int o_t, void* o, float* lse, void* ws,
                             size_t ws_bytes, bool use_scratch, void* stream) {
  if (!q_idx || !q_val || !kc_idx || !kc_val || !v_cache || !o) return SFA_EINVAL;
  if (!use_scratch && !ws) return SFA_EINVAL;
  if (B < 1 || Hq < 1 || Hkv < 1 || Lmax < 1 || d < 1 || k < 1 || k > d) return SFA_EINVAL;
  if (window < 0 || n_global < 0) return SFA_EINVAL;
  if (Lmax > (1 << 30)) return SFA_ENOTSUP;
  if (Hq % Hkv != 0) return SFA_EINVAL;
  if (!is_idx(q_idx_t) || !is_cval(q_val_t) || !is_idx(kc_idx_t) || !is_cval(kc_val_t) ||
      !is_val(v_t) || !is_val(o_t))
    return SFA_EINVAL;
  if (!isfinite(scale)) return SFA_EINVAL;
  if ((long long)B * Hkv > 65535) return SFA_ENOTSUP;
  // head dims or group sizes without the tuned kernel: the float32 decode
  // (no alignment needs)
  const bool generic = (d != 64 && d != 128) || !pow2_le(Hq / Hkv, sfa::decode_max_group());
  if (generic && (d > 256 || Hq / Hkv > sfa::decode_generic_max_group())) return SFA_ENOTSUP;
  if (!generic && ((uintptr_t)v_cache | (uintptr_t)kc_idx | (uintptr_t)kc_val) % 16 != 0)
    return SFA_EINVAL;
  const size_t need = sfa::decode_workspace_bytes(B, Hq, Lmax, d);
  if (use_scratch) {
    if (need > sfa::noalloc_scratch_bytes()) return SFA_ENOSPC;
    if (sfa::noalloc_scratch(&ws) != hipSuccess) return SFA_EHIP;
  } else if (ws_bytes < need) {
    return SFA_ENOSPC;
  }
  sfa::DecodeArgs a = {};
  a.q_idx = q_idx; a.q_val = q_val; a.kc_idx = kc_idx; a.kc_val = kc_val; a.v = v_cache;
  a.seq_len = seq_len;
  a.B = B; a.Hq = Hq; a.Hkv = Hkv; a.Lmax = Lmax; a.d = d; a.k = k; a.scale = scale;
  a.window = window; a.n_global = window > 0 ? n_global : 0;
  a.qifmt = ifmt_of(q_idx_t); a.qvfmt = vfmt_of(q_val_t);
  a.kifmt = ifmt_of(kc_idx_t); a.kvfmt = vfmt_of(kc_val_t);
  a.vbf16 = v_t == SFA_BF16; a.obf16 = o_t == SFA_BF16;
  a.o = o; a.lse = lse; a.ws = ws;
  return from_hip(generic ? sfa::launch_attn_decode_generic(a, (hipStream_t)stream)
                          : sfa::launch_attn_decode(a, (hipStream_t)stream));
}

}  // namespace

extern "C" {

sfa_status sfa_attn_decode(const void* q_idx, const void* q_val, const void* kc_idx,
                           const void* kc_val, const void* v_cache, const int32_t* seq_len,
                           int B, int Hq, int Hkv, int Lmax, int d, int k, float scale,
                           int window, int n_global,
                           int q_idx_t, int q_val_t, int kc_idx_t, int kc_val_t, int v_t,
                           int o_t, void* o, float* lse, void* ws, size_t ws_bytes,
                           void* stream) {
  return decode_contiguous(q_idx, q_val, kc_idx, kc_val, v_cache, seq_len, B, Hq, Hkv, Lmax, d,
                           k, scale, window, n_global, q_idx_t, q_val_t, kc_idx_t, kc_val_t, v_t,
                           o_t, o, lse, ws, ws_bytes, false, stream);
}

sfa_status sfa_attn_decode_noalloc(const void* q_idx, const void* q_val, const void* kc_idx,
                                   const void* kc_val, const void* v_cache,
                                   const int32_t* seq_len, int B, int Hq, int Hkv, int Lmax,
                                   int d, int k, float scale, int window, int n_global,
                                   int q_idx_t, int q_val_t, int kc_idx_t, int kc_val_t, int v_t,
                                   int o_t, void* o, float* lse, void* stream) {
  return decode_contiguous(q_idx, q_val, kc_idx, kc_val, v_cache, seq_len, B, Hq, Hkv, Lmax, d,
                           k, scale, window, n_global, q_idx_t, q_val_t, kc_idx_t, kc_val_t, v_t,
                           o_t, o, lse, nullptr, 0, true, stream);
}

sfa_status sfa_attn_decode_paged(const float* q, const void* q_idx, const void* q_val,
                                 const void* kc_idx, const void* kc_val, const void* v_cache,
                                 const int32_t* block_table, int max_pages, int page_size,
                                 int num_pages, const int32_t* seq_len, int B, int Hq, int Hkv,
                                 int d, int k, float scale, int window, int n_global,
                                 int q_idx_t, int q_val_t,
                                 int kc_idx_t, int kc_val_t, int v_t, int o_t, void* o,
                                 float* lse, void* ws, size_t ws_bytes, void* stream) {
  const bool dense_q = q != nullptr;
  if (dense_q ? (q_idx || q_val) : (!q_idx || !q_val)) return SFA_EINVAL;
  if (!kc_idx || !kc_val || !v_cache || !block_table || !o || !ws) return SFA_EINVAL;
  if (B < 1 || Hq < 1 || Hkv < 1 || d < 1 || k < 1 || k > d) return SFA_EINVAL;
  if (max_pages < 1 || num_pages < 1) return SFA_EINVAL;
  if (window < 0 || n_global < 0) return SFA_EINVAL;
  if (page_size < 16 || (page_size & (page_size - 1)) != 0) return SFA_EINVAL;
  if ((long long)max_pages * page_size > (1LL << 30)) return SFA_EINVAL;
  if (Hq % Hkv != 0) return SFA_EINVAL;
  if ((!dense_q && (!is_idx(q_idx_t) || !is_cval(q_val_t))) || !is_idx(kc_idx_t) ||
      !is_cval(kc_val_t) || !is_val(v_t) || !is_val(o_t))
    return SFA_EINVAL;
  if (!isfinite(scale)) return SFA_EINVAL;
  if ((long long)B * Hkv > 65535) return SFA_ENOTSUP;
  const bool generic = (d != 64 && d != 128) || !pow2_le(Hq / Hkv, sfa::decode_max_group());
  if (generic && (d > 256 || Hq / Hkv > sfa::decode_generic_max_group())) return SFA_ENOTSUP;
  const int Lmax = max_pages * page_size;
  if (!generic && ((uintptr_t)v_cache | (uintptr_t)kc_idx | (uintptr_t)kc_val) % 16 != 0)
    return SFA_EINVAL;
  if (ws_bytes < sfa::decode_workspace_bytes(B, Hq, Lmax, d)) return SFA_ENOSPC;
  int log2P = 0;
  while ((1 << log2P) < page_size) ++log2P;
  sfa::DecodeArgs a = {};
  a.q_dense = q; a.q_idx = q_idx; a.q_val = q_val;
  a.kc_idx = kc_idx; a.kc_val = kc_val; a.v = v_cache;
  a.seq_len = seq_len; a.table = block_table;
  a.B = B; a.Hq = Hq; a.Hkv = Hkv; a.Lmax = Lmax; a.d = d; a.k = k; a.scale = scale;
  a.max_pages = max_pages; a.log2P = log2P; a.num_pages = num_pages;
  a.window = window; a.n_global = window > 0 ? n_global : 0;
  a.qifmt = dense_q ? 0 : ifmt_of(q_idx_t); a.qvfmt = dense_q ? 0 : vfmt_of(q_val_t);
  a.kifmt = ifmt_of(kc_idx_t); a.kvfmt = vfmt_of(kc_val_t);
  a.vbf16 = v_t == SFA_BF16; a.obf16 = o_t == SFA_BF16;
  a.o = o; a.lse = lse; a.ws = ws;
  return from_hip(generic ? sfa::launch_attn_decode_generic(a, (hipStream_t)stream)
                          : sfa::launch_attn_decode(a, (hipStream_t)stream));
}

sfa_status sfa_kv_append(const float* k_new, const void* v_new, const int32_t* n_new,
                         int32_t* seq_len, int B, int Hkv, int T, int d, int k,
                         const int32_t* block_table, int max_pages, int page_size,
                         int num_pages, void* kc_idx, void* kc_val, void* v_cache,
                         int kc_idx_t, int kc_val_t, int v_new_t, int v_t, void* stream) {
  if (!seq_len || !kc_idx || !kc_val || !v_cache) return SFA_EINVAL;
  if (B < 1 || Hkv < 1 || T < 0 || d < 1 || k < 1 || k > d || page_size < 1) return SFA_EINVAL;
  if (T > 0 && (!k_new || !v_new)) return SFA_EINVAL;
  if (block_table && (max_pages < 1 || num_pages < 1)) return SFA_EINVAL;
  if (block_table && (long long)max_pages * page_size > (1LL << 30)) return SFA_EINVAL;
  if (block_table && (page_size & (page_size - 1)) != 0) return SFA_EINVAL;
  if (!is_idx(kc_idx_t) || !is_cval(kc_val_t) || !is_val(v_new_t) || !is_val(v_t))
    return SFA_EINVAL;
  if (kc_idx_t == SFA_I16 && d > 32767) return SFA_EINVAL;
  if (d > 256) return SFA_ENOTSUP;
  if ((long long)B * Hkv * T > (1LL << 31)) return SFA_ENOTSUP;
  sfa::AppendArgs a = {};
  a.k_new = k_new; a.v_new = v_new; a.n_new = n_new; a.seq_len = seq_len;
  a.table = block_table; a.kc_idx = kc_idx; a.kc_val = kc_val; a.v_cache = v_cache;
  a.B = B; a.Hkv = Hkv; a.T = T; a.d = d; a.k = k;
  a.page_size = page_size; a.max_pages = max_pages; a.num_pages = num_pages;
  while ((1 << a.log2P) < page_size) ++a.log2P;
  a.ifmt = ifmt_of(kc_idx_t); a.vfmt = vfmt_of(kc_val_t);
  a.vin_bf16 = v_new_t == SFA_BF16; a.vc_bf16 = v_t == SFA_BF16;
  return from_hip(sfa::launch_kv_append(a, (hipStream_t)stream));
}

sfa_status sfa_csr_to_codes(const int32_t* indptr, const void* indices, int indices_t,
                            const void* values, int values_t, int64_t rows, int d, int kmax,
                            void* idx, int idx_t, void* val, void* stream) {
  if (rows < 0 || d < 1 || kmax < 1 || kmax > d) return SFA_EINVAL;
  if (!is_idx(indices_t) || !is_idx(idx_t) || !is_cval(values_t)) return SFA_EINVAL;
  if (d > 256) return SFA_ENOTSUP;
  if (rows == 0) return SFA_OK;
  if (!indptr || !indices || !values || !idx || !val) return SFA_EINVAL;
  if ((rows + 3) / 4 > 0x7fffffffLL) return SFA_ENOTSUP;
  sfa::CsrArgs a = {};
  a.indptr = indptr; a.indices = indices; a.values = values; a.rows = rows; a.d = d;
  a.kmax = kmax; a.ifmt_in = ifmt_of(indices_t); a.vbytes = values_t == SFA_F32 ? 4 : 2;
  a.idx_out = idx; a.ifmt_out = ifmt_of(idx_t); a.val_out = val;
  return from_hip(sfa::launch_csr_to_codes(a, (hipStream_t)stream));
}

sfa_status sfa_kv_append_q8(const float* k_new, const void* v_new, const int32_t* n_new,
                            int32_t* seq_len, int B, int Hkv, int T, int d, int k,
                            const int32_t* block_table, int max_pages, int page_size,
                            int num_pages, void* kc_idx, int8_t* kc_val, float* kc_scale,
                            int8_t* v_cache, float* v_scale, int kc_idx_t, int v_new_t,
                            void* stream) {
  if (!seq_len || !kc_idx || !kc_val || !kc_scale || !v_cache || !v_scale) return SFA_EINVAL;
  if (B < 1 || Hkv < 1 || T < 0 || d < 1 || k < 1 || k > d || page_size < 1) return SFA_EINVAL;
  if (T > 0 && (!k_new || !v_new)) return SFA_EINVAL;
  if (block_table && (max_pages < 1 || num_pages < 1)) return SFA_EINVAL;
  if (block_table && (long long)max_pages * page_size > (1LL << 30)) return SFA_EINVAL;
  if (block_table && (page_size & (page_size - 1)) != 0) return SFA_EINVAL;
  if (!is_idx(kc_idx_t) || !is_val(v_new_t)) return SFA_EINVAL;
  if (d > 256) return SFA_ENOTSUP;
  if ((long long)B * Hkv * T > (1LL << 31)) return SFA_ENOTSUP;
  sfa::AppendArgs a = {};
  a.k_new = k_new; a.v_new = v_new; a.n_new = n_new; a.seq_len = seq_len;
  a.table = block_table; a.kc_idx = kc_idx; a.kc_val = kc_val; a.v_cache = v_cache;
  a.B = B; a.Hkv = Hkv; a.T = T; a.d = d; a.k = k;
  a.page_size = page_size; a.max_pages = max_pages; a.num_pages = num_pages;
  while ((1 << a.log2P) < page_size) ++a.log2P;
  a.ifmt = ifmt_of(kc_idx_t); a.vfmt = sfa::kValF32;
  a.vin_bf16 = v_new_t == SFA_BF16; a.vc_bf16 = 0;
  a.q8 = 1; a.kc_scale = kc_scale; a.v_scale = v_scale;
  return from_hip(sfa::launch_kv_append(a, (hipStream_t)stream));
}

sfa_status sfa_attn_decode_q8(const float* q, const void* q_idx, const void* q_val,
                              const void* kc_idx, const int8_t* kc_val, const float* kc_scale,
                              const int8_t* v_cache, const float* v_scale,
                              const int32_t* block_table, int max_pages, int page_size,
                              int num_pages, const int32_t* seq_len, int B, int Hq, int Hkv,
                              int d, int k, float scale, int window, int n_global, int q_idx_t,
                              int q_val_t, int kc_idx_t, int o_t, void* o, float* lse, void* ws,
                              size_t ws_bytes, void* stream) {
  const bool dense_q = q != nullptr;
  if (dense_q ? (q_idx || q_val) : (!q_idx || !q_val)) return SFA_EINVAL;
  if (!kc_idx || !kc_val || !kc_scale || !v_cache || !v_scale || !o || !ws) return SFA_EINVAL;
  if (B < 1 || Hq < 1 || Hkv < 1 || d < 1 || k < 1 || k > d || page_size < 1) return SFA_EINVAL;
  if (block_table && (max_pages < 1 || num_pages < 1)) return SFA_EINVAL;
  if (block_table && (page_size < 16 || (page_size & (page_size - 1)) != 0)) return SFA_EINVAL;
  if (window < 0 || n_global < 0) return SFA_EINVAL;
  if (Hq % Hkv != 0) return SFA_EINVAL;
  if ((!dense_q && (!is_idx(q_idx_t) || !is_cval(q_val_t))) || !is_idx(kc_idx_t) || !is_val(o_t))
    return SFA_EINVAL;
  if (!isfinite(scale)) return SFA_EINVAL;
  const long long cap = block_table ? (long long)max_pages * page_size : page_size;
  if (cap > (1LL << 30)) return SFA_ENOTSUP;
  if ((long long)B * Hkv > 65535) return SFA_ENOTSUP;
  // the 8-bit cache runs the vector decode: int16 indices, k in {8, 16, 32},
  // d in {64, 128}, a power-of-two group <= 8
  if (kc_idx_t != SFA_I16 || !sfa::decode_q8_supported(d, k, Hq / Hkv)) return SFA_ENOTSUP;
  if (((uintptr_t)v_cache | (uintptr_t)kc_idx | (uintptr_t)kc_val) % 16 != 0) return SFA_EINVAL;
  const int Lmax = (int)cap;
  if (ws_bytes < sfa::decode_workspace_bytes(B, Hq, Lmax, d)) return SFA_ENOSPC;
  int log2P = 0;
  if (block_table)
    while ((1 << log2P) < page_size) ++log2P;
  sfa::DecodeArgs a = {};
  a.q_dense = q; a.q_idx = q_idx; a.q_val = q_val;
  a.kc_idx = kc_idx; a.kc_val = kc_val; a.v = v_cache;
  a.kc_scale = kc_scale; a.v_scale = v_scale;
  a.seq_len = seq_len; a.table = block_table;
  a.B = B; a.Hq = Hq; a.Hkv = Hkv; a.Lmax = Lmax; a.d = d; a.k = k; a.scale = scale;
  a.max_pages = max_pages; a.log2P = log2P; a.num_pages = num_pages;
  a.window = window; a.n_global = window > 0 ? n_global : 0;
  a.qifmt = dense_q ? 0 : ifmt_of(q_idx_t); a.qvfmt = dense_q ? 0 : vfmt_of(q_val_t);
  a.kifmt = sfa::kIdxI16; a.kvfmt = sfa::kValF32;
  a.vbf16 = 0; a.obf16 = o_t == SFA_BF16;
  a.o = o; a.lse = lse; a.ws = ws;
  return from_hip(sfa::launch_attn_decode_q8(a, (hipStream_t)stream));
}

}  // extern "C"
