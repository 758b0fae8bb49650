// Internal launchers behind the C ABI (host side).  Arguments are validated
// by the ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sfa {

hipError_t launch_topk_encode(const float* x, int64_t rows, int d, int k, void* idx, int idx16,
                              void* val, int valbf16, hipStream_t stream);

hipError_t launch_attn_fwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, int B, int Hq, int Hkv, int n, int d,
                           int k, int causal, float scale, int idx16, int valbf16, int vbf16,
                           int obf16, void* o, float* lse, void* ws, hipStream_t stream);
int fwd_max_group();
size_t fwd_workspace_bytes(int B, int Hkv, int n, int d, int vbf16);

hipError_t launch_attn_bwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, const void* o, const float* lse,
                           const void* dout, int B, int Hq, int Hkv, int n, int d, int k,
                           int causal, float scale, int idx16, int valbf16, int vbf16, int obf16,
                           float* dq, float* dk, float* dv, void* ws, hipStream_t stream);
size_t bwd_workspace_bytes(int B, int Hq, int Hkv, int n, int d);
int bwd_max_group();

hipError_t launch_attn_fwd_index(const void* q_idx, const void* q_val, const void* k_idx,
                                 const void* k_val, const void* v, int B, int Hq, int Hkv, int n,
                                 int d, int k, int causal, float scale, int idx16, int valbf16,
                                 int vbf16, int obf16, void* o, float* lse, hipStream_t stream);
int fwd_index_lds_bytes(int d, int k, int vbf16);
int fwd_index_max_k();
int fwd_index_rows_per_block();

hipError_t launch_attn_decode(const void* q_idx, const void* q_val, const void* kc_idx,
                              const void* kc_val, const void* v, const int32_t* seq_len, int B,
                              int Hq, int Hkv, int Lmax, int d, int k, float scale, int qidx16,
                              int qvalbf16, int kidx16, int kvalbf16, int vbf16, int obf16,
                              void* o, float* lse, void* ws, hipStream_t stream);
size_t decode_workspace_bytes(int B, int Hq, int Lmax, int d);
int decode_max_group();

}  // namespace sfa
