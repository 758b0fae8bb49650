// Internal launchers behind the C ABI (host side).  Arguments are validated
// by the ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sfa {

hipError_t launch_topk_encode(const float* x, int64_t rows, int d, int k, void* idx, int ifmt,
                              void* val, int vfmt, hipStream_t stream);

hipError_t launch_attn_fwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, int B, int Hq, int Hkv, int n, int d,
                           int k, int causal, int window, int n_global, float scale, int ifmt,
                           int vfmt, int vbf16, int obf16, void* o, float* lse, void* ws,
                           hipStream_t stream);
int fwd_max_group();
size_t fwd_workspace_bytes(int B, int Hkv, int n, int d, int vbf16);

// float32 vector-unit forward for head dimensions without a matrix-core
// kernel (d <= 256); no workspace, any group size
hipError_t launch_attn_fwd_generic(const void* q_idx, const void* q_val, const void* k_idx,
                                   const void* k_val, const void* v, int B, int Hq, int Hkv,
                                   int n, int d, int k, int causal, int window, int n_global,
                                   float scale, int ifmt, int vfmt, int vbf16, int obf16, void* o,
                                   float* lse, hipStream_t stream);
bool fwd_generic_supported(int d, int k);

hipError_t launch_attn_bwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, const void* o, const float* lse,
                           const void* dout, int B, int Hq, int Hkv, int n, int d, int k,
                           int causal, int window, int n_global, float scale, int ifmt,
                           int vfmt, int vbf16, int obf16, float* dq, float* dk, float* dv,
                           void* ws, hipStream_t stream);
size_t bwd_workspace_bytes(int B, int Hq, int Hkv, int n, int d);
int bwd_max_group();

// float32 backward for head dimensions without the matrix-core kernels
// (d <= 256); no workspace, any group size
hipError_t launch_attn_bwd_generic(const void* q_idx, const void* q_val, const void* k_idx,
                                   const void* k_val, const void* v, const void* o,
                                   const float* lse, const void* dout, int B, int Hq, int Hkv,
                                   int n, int d, int k, int causal, int window, int n_global,
                                   float scale, int ifmt, int vfmt, int vbf16, int obf16,
                                   float* dq, float* dk, float* dv, hipStream_t stream);
bool bwd_generic_supported(int d, int k);

hipError_t launch_attn_fwd_index(const void* q_idx, const void* q_val, const void* k_idx,
                                 const void* k_val, const void* v, int B, int Hq, int Hkv, int n,
                                 int d, int k, int causal, float scale, int ifmt, int vfmt,
                                 int vbf16, int obf16, void* o, float* lse, hipStream_t stream);
int fwd_index_lds_bytes(int d, int k, int vbf16);
int fwd_index_max_k();
int fwd_index_rows_per_block();

// Decode over a contiguous (table == nullptr: [B, Hkv, Lmax, ...]) or paged
// (pages [num_pages, Hkv, 1 << log2P, ...], table [B, max_pages],
// Lmax = max_pages << log2P) cache; query codes, or q_dense coded in-kernel.
struct DecodeArgs {
  const float* q_dense;
  const void *q_idx, *q_val, *kc_idx, *kc_val, *v;
  const int32_t* seq_len;
  const int32_t* table;
  int B, Hq, Hkv, Lmax, d, k;
  int max_pages, log2P, num_pages;
  int window, n_global;  // token pattern (window 0: none)
  float scale;
  int qifmt, qvfmt, kifmt, kvfmt, vbf16, obf16;
  void* o;
  float* lse;
  void* ws;
  // 8-bit cache (launch_attn_decode_q8): float32 scale per key row / value row
  const float* kc_scale;
  const float* v_scale;
};
// Keys per decode workgroup (one context chunk); the workspace holds one
// partial (m, l, o) per chunk, query head and sequence.
constexpr int kDecodeChunk = 4096;
hipError_t launch_attn_decode(const DecodeArgs& a, hipStream_t stream);
size_t decode_workspace_bytes(int B, int Hq, int Lmax, int d);
int decode_max_group();
// float32 decode for head dimensions without the tuned kernel (d <= 256);
// same workspace and partial layout, Hq / Hkv <= decode_generic_max_group()
hipError_t launch_attn_decode_generic(const DecodeArgs& a, hipStream_t stream);
int decode_generic_max_group();

// Static device scratch of the allocation-free decode (one copy per GPU):
// its size, and its device address on the current device (looked up once per
// device).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void** out);

// Decode over the 8-bit cache: int8 code values (int16 indices, k in
// {8, 16, 32}) and int8 value rows with their scales; d in {64, 128}, Hq /
// Hkv a power of two <= 8.
hipError_t launch_attn_decode_q8(const DecodeArgs& a, hipStream_t stream);
bool decode_q8_supported(int d, int k, int G);

// KV-cache append: Top-k coding of new keys and copy of their values into a
// contiguous (table == nullptr: [B, Hkv, P, ...]) or paged cache, then
// seq_len[b] += the appended count (clamped to the capacity).
struct AppendArgs {
  const float* k_new;
  const void* v_new;
  const int32_t* n_new;
  int32_t* seq_len;
  const int32_t* table;
  void *kc_idx, *kc_val, *v_cache;
  int B, Hkv, T, d, k;
  int page_size, max_pages, num_pages;
  int log2P;  // paged: page_size == 1 << log2P
  int ifmt, vfmt, vin_bf16, vc_bf16;
  // 8-bit cache: kc_val and v_cache hold int8, with one float32 scale per
  // key row (kc_scale) and value row (v_scale)
  int q8;
  float* kc_scale;
  float* v_scale;
};
hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream);

// CSR codes (row r: entries indptr[r] .. indptr[r+1]-1) to fixed rows of kmax
// entries, padded with zero values at the lowest free coordinates.
struct CsrArgs {
  const int32_t* indptr;
  const void* indices;
  const void* values;
  int64_t rows;
  int d, kmax;
  int ifmt_in, vbytes;  // index format; value storage bytes (copied bitwise)
  void* idx_out;
  int ifmt_out;
  void* val_out;
};
hipError_t launch_csr_to_codes(const CsrArgs& a, hipStream_t stream);

}  // namespace sfa
