/*
 * sfa.h -- C ABI of libsfa, a gfx950 (AMD Instinct MI355X) implementation of
 * Sparse Feature Attention (SFA): attention in which every query and key is a
 * k-sparse code, the Top-k of its d-dimensional projection.
 *
 * Paper: "Scaling Attention via Feature Sparsity" (arXiv 2603.22300).
 *   - Top-k coding: Sec. 3.1, Eqs. (3)-(4).
 *   - Overlap scores s_ij = scale * sum_{u in S_i cap S_j} q_iu k_ju: Sec. 3.1, Eq. (5).
 *   - Masked softmax and value aggregation: Sec. 2, Eqs. (1)-(2);
 *     the tiled kernel's result equals softmax(Q~ K~^T / sqrt(d)) V: Sec. 3.2.
 *   - Decode against a cache of sparse key codes and dense V: App. B
 *     ("KV-cache latency") and App. J (code storage); appending coded keys
 *     to a contiguous or paged cache, and decode through its block table.
 *
 * Conventions shared by every entry point
 *   - All array pointers are DEVICE pointers to dense, row-major, contiguous
 *     arrays owned by the caller.  The library never allocates device memory
 *     and keeps no state across calls apart from cached device properties.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Every call only enqueues work on `stream` and returns; results are
 *     ready when the stream reaches that point.
 *   - Arguments are validated on the host before anything is launched.  On
 *     any error nothing is launched and no output is touched.  No exception
 *     crosses the ABI.
 *   - Codes: a code row is k (index, value) pairs.  Indices lie in [0, d) and
 *     are distinct within a row; sfa_topk_encode writes them in ascending
 *     order (the attention entry points accept any order).  Values and V must
 *     be finite.  Violating these device-side preconditions gives undefined
 *     results (no fault: indices are masked into range before any access).
 *   - Grouped heads: query head h reads KV head h / (Hq / Hkv).
 *   - dtype codes below: code index arrays are SFA_I32, SFA_I16 or SFA_U8;
 *     code value arrays are SFA_F32, SFA_BF16 (bfloat16 bit patterns) or
 *     SFA_F16 (binary16); V and O are SFA_F32 or SFA_BF16.  Narrow formats
 *     are written with round-to-nearest-even.
 *   - Device pointers are at least 16-byte aligned (any torch allocation is);
 *     the decode entry points check this for the cache arrays.
 */
#ifndef SFA_H
#define SFA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SFA_OK = 0,
  SFA_EINVAL = 1,  /* bad argument: null pointer, size out of range, k > d,
                      Hq not a multiple of Hkv, bad dtype code             */
  SFA_ENOTSUP = 2, /* valid but unsupported: head dim or dtype combination
                      without a kernel, or a shape whose tiles exceed LDS  */
  SFA_EHIP = 3,    /* the HIP runtime reported an error at launch          */
  SFA_ENOSPC = 4   /* the caller's workspace is smaller than required      */
} sfa_status;

/* SFA_U8 (8-bit unsigned indices) and SFA_F16 (IEEE binary16 values) are the
 * compact code storage of App. J (int8 indices, fp16 values): for code arrays
 * only, not for V or O. */
typedef enum {
  SFA_I32 = 0, SFA_I16 = 1, SFA_F32 = 2, SFA_BF16 = 3, SFA_U8 = 4, SFA_F16 = 5
} sfa_dtype;

/* Version of this ABI (incremented on any incompatible change). */
int sfa_abi_version(void);

/* Static, human-readable text for a status code. */
const char* sfa_strerror(int status);

/*
 * Row-wise Top-k coding (Sec. 3.1, Eqs. (3)-(4)).
 *
 * x    [rows, d] float32.  For each row, keeps the k coordinates of largest
 *      |x_u|; ties go to the lower index (the paper leaves ties open).
 *      Magnitudes are compared as exact float32 values: subnormals are
 *      ordered, never flushed; +0 and -0 tie.
 * idx  [rows, k] of idx_t (SFA_I32, SFA_I16 or SFA_U8; d <= 256 fits all):
 *      the kept coordinates in ascending order.
 * val  [rows, k] of val_t: SFA_F32 copies x_u bit for bit; SFA_BF16 and
 *      SFA_F16 store x_u rounded to nearest-even bfloat16 / binary16
 *      (selection still uses the float32 magnitudes; binary16 overflows to
 *      +-inf beyond 65504 and keeps subnormals).
 * Limits: 1 <= d <= 256, 1 <= k <= d, rows >= 0 (rows == 0 is a no-op).
 * Errors: SFA_EINVAL (null pointer with rows > 0, k or d out of range,
 *         bad dtype), SFA_ENOTSUP (d > 256), SFA_EHIP.
 */
sfa_status sfa_topk_encode(const float* x, int64_t rows, int d, int k,
                           void* idx, int idx_t, void* val, int val_t,
                           void* stream);

/*
 * SFA forward (Sec. 3.1-3.2): for every batch b, query head h and position i
 *   s_ij  = scale * sum_{u in S_i cap S_j} q_iu k_ju            (allowed j)
 *   O_i   = sum_j exp(s_ij - m_i) v_j / l_i,  l_i = sum_j exp(s_ij - m_i)
 *   LSE_i = m_i + ln(l_i),  m_i = max_j s_ij
 * where the allowed keys are j <= i if `causal`, else all j < n.  An allowed
 * key whose support does not overlap the query's enters with s_ij = 0.
 * No n x n matrix is ever stored.
 * Token sparsity (App. E: SFA composed with Longformer-style patterns): with
 * window > 0 the allowed keys are further limited to |i - j| < window, plus
 * the n_global leading tokens, which every query sees and which see every
 * key; key tiles outside every row's window are skipped, not masked.
 * window 0 (n_global ignored) is plain causal / full attention.
 *
 * q_idx, q_val  [B, Hq, n, k]   query codes (idx_t, qk_val_t)
 * k_idx, k_val  [B, Hkv, n, k]  key codes   (idx_t, qk_val_t)
 * v             [B, Hkv, n, d]  values (v_t: SFA_BF16 or SFA_F32)
 * o             [B, Hq, n, d]   output (o_t: SFA_F32 or SFA_BF16, the latter
 *                               rounded to nearest-even from float32)
 * lse           [B, Hq, n] float32 natural-log LSE, or NULL to skip it.
 * ws, ws_bytes  caller-owned device workspace of at least
 *               sfa_attn_fwd_workspace(B, Hkv, n, d, v_t) bytes (0 for float32
 *               V and for head dims other than 64 and 128, where ws may be
 *               NULL).  With bf16 V it receives, on the
 *               stream, V converted once to float16 and laid out as the
 *               kernel's key tiles, and a range flag per tile (at d = 128
 *               also the per-tile inverted indexes below).  Calls that
 *               overlap in time need separate workspaces.
 * Arithmetic: the scores are the product of the densified codes on the
 * matrix cores, each value split into 16-bit pieces whose products are
 * exact in float32: with bf16 V two float16 pieces x0 = f16(x),
 * x1 = f16(x - x0) and three piece products (relative error ~3 * 2^-22 of
 * sum |q_u k_u|); with float32 V, and for code values of magnitude >= 65504
 * (query values after the scale), three bfloat16 pieces and six products
 * (~2^-24); softmax and accumulation in float32.  16-bit code values (SFA_BF16 or SFA_F16) with bf16 V and a
 * nonzero scale: the raw query and key values are the matrix-core
 * operands (bf16 or float16 products, exact in float32, one per coordinate
 * block), the sign of scale is folded into the query values and |scale| is
 * applied to the float32 scores.  With bf16 V, V is converted to float16
 * (exact for normal values up to 65504) and the probabilities (below 2^15)
 * enter P.V as float16,
 * relative rounding 2^-11 per weight (MFMA, float32 accumulate).  Workgroups
 * whose keys reach a V value of magnitude >= 65536 (or inf / NaN), or a
 * code value too large for the float16 pieces, are recomputed by a second
 * kernel launched on the same stream, with bf16 V and the probabilities
 * split into two bfloat16 terms (~2^-17); it returns at once when no
 * workgroup was handed back.  With float32 V
 * the P.V product is float32.
 * Inverted-index scores (Sec. 3.2: intersect the supports through the keys'
 * active features): at d = 128, k <= 2, bf16 V, each key tile's codes are
 * bucketed once per call by (coordinate, key parity), and each query
 * nonzero (u, q_u) adds q_u * k_u into the scores of exactly the keys of the
 * tile that hold u (float32 products and sums).  This is chosen on the device
 * from the data: if the tiles' longest buckets average at most 6 entries
 * (near-uniform supports); skewed supports (long buckets) take the matrix-core
 * product instead.  The results agree with the matrix-core path up to float32
 * summation order.
 * Other head dims (d <= 256 except 64 and 128), and group sizes Hq / Hkv
 * that are not a power of two <= 128, run on a float32 vector-unit kernel:
 * overlap sums by code lookups, exact running maximum, float32 probabilities
 * and P.V; any group size, no workspace (ws is then unused).
 * Limits: B, Hq, Hkv, n >= 1; Hq % Hkv == 0; 1 <= k <= d <= 256;
 *         B * Hkv <= 65535; n * d <= 2^29 and n * k <= 2^29;
 *         on the float32 kernel: B * Hq <= 65535 (SFA_ENOTSUP otherwise);
 *         window, n_global >= 0.
 * Errors: SFA_EINVAL, SFA_ENOTSUP, SFA_ENOSPC (workspace missing or too
 *         small), SFA_EHIP.
 */
sfa_status sfa_attn_fwd(const void* q_idx, const void* q_val,
                        const void* k_idx, const void* k_val,
                        const void* v,
                        int B, int Hq, int Hkv, int n, int d, int k,
                        int causal, int window, int n_global, float scale,
                        int idx_t, int qk_val_t, int v_t, int o_t,
                        void* o, float* lse, void* ws, size_t ws_bytes,
                        void* stream);

/*
 * Bytes of device workspace sfa_attn_fwd needs for these sizes: 0 for
 * float32 V (v_t == SFA_F32), for head dims other than 64 and 128 (no
 * workspace), and for invalid sizes.
 */
size_t sfa_attn_fwd_workspace(int B, int Hkv, int n, int d, int v_t);

/*
 * The same forward with the overlap scores accumulated through a per-key-tile
 * inverted index in LDS (Sec. 3.2's feature-intersection formulation): the
 * tile's key codes are counting-sorted by (coordinate, key parity), and for
 * each nonzero (u, q_u) of a query row the row's two owner threads add
 * q_u * k_u into the score tile for exactly the keys holding u.  Same
 * arguments (without the workspace) and definitions as sfa_attn_fwd; the
 * scores agree up to float32 summation order, and with bf16 V the
 * probabilities enter P.V as two bfloat16 pieces, hi + lo (relative rounding
 * ~2^-17 per weight).  Results are bitwise repeatable.  Slower on this hardware than
 * sfa_attn_fwd; kept as the direct realisation of the overlap formulation.
 * Limits: as sfa_attn_fwd with d in {64, 128}, plus k <= 64, Hq / Hkv <= 128,
 * and the per-tile tables must fit LDS (SFA_ENOTSUP otherwise).
 */
sfa_status sfa_attn_fwd_index(const void* q_idx, const void* q_val,
                              const void* k_idx, const void* k_val,
                              const void* v,
                              int B, int Hq, int Hkv, int n, int d, int k,
                              int causal, float scale,
                              int idx_t, int qk_val_t, int v_t, int o_t,
                              void* o, float* lse, void* stream);

/*
 * SFA backward with the straight-through estimator (Sec. 3.1, Eq. (6)).
 * With the forward's weights P_ij = exp(s_ij - LSE_i) over the allowed keys
 * (s_ij as in sfa_attn_fwd) and D_i = dO_i . O_i:
 *   dV_j  = sum_i P_ij dO_i
 *   dS_ij = P_ij (dO_i . v_j - D_i)
 *   dQ~_i = scale sum_j dS_ij k~_j,   dK~_j = scale sum_i dS_ij q~_i
 * and, by Eq. (6), the gradient of a query coordinate u is dQ~_iu on the
 * query's support and 0 elsewhere (likewise for keys).  The results come in
 * code form, aligned with the codes: dq_val[..., t] is the gradient at
 * q_idx[..., t].  A KV head's dk_val and dv sum over the query heads that
 * read it.
 *
 * q_*, k_*, v, B ... o_t   as sfa_attn_fwd (o and dout share o_t), including
 *               the token window: the allowed keys must be those of the
 *               forward that produced o and lse; tiles outside every
 *               row's (key's) window are skipped in each kernel.
 * o             [B, Hq, n, d]   the forward's output
 * lse           [B, Hq, n] float32, the forward's LSE (natural log)
 * dout          [B, Hq, n, d]   dL/dO
 * dq_val        [B, Hq, n, k]  float32 out
 * dk_val        [B, Hkv, n, k] float32 out
 * dv            [B, Hkv, n, d] float32 out
 * ws, ws_bytes  caller-owned device workspace of at least
 *               sfa_attn_bwd_workspace(B, Hq, Hkv, n, d) bytes: tile images of
 *               the codes, V and dO, and partial gradients of the keys that
 *               global tokens make every query see, written and read on the
 *               stream (0 bytes and ws unused for head dims other than 64
 *               and 128).  Calls that overlap in time need separate
 *               workspaces.
 * Arithmetic: every product on the matrix cores with both operands split
 * into two bfloat16 pieces and three piece products kept (relative error
 * ~2^-16 of the sum of |terms|), float32 accumulation; P recomputed as
 * exp2(s log2(e) - LSE log2(e)) in float32.
 * Other head dims (d <= 256 except 64 and 128), and group sizes Hq / Hkv
 * that are not a power of two <= 8, run a float32 vector-unit backward: the
 * same formulas, scores and P recomputed in float32, no workspace (ws may be
 * NULL), any group size.
 * Limits: as sfa_attn_fwd; on the float32 backward: B * Hq <= 65535.
 * Errors: SFA_EINVAL, SFA_ENOTSUP, SFA_ENOSPC, SFA_EHIP.
 */
sfa_status sfa_attn_bwd(const void* q_idx, const void* q_val,
                        const void* k_idx, const void* k_val,
                        const void* v, const void* o, const float* lse,
                        const void* dout,
                        int B, int Hq, int Hkv, int n, int d, int k,
                        int causal, int window, int n_global, float scale,
                        int idx_t, int qk_val_t, int v_t, int o_t,
                        float* dq_val, float* dk_val, float* dv,
                        void* ws, size_t ws_bytes, void* stream);

/* Bytes of device workspace sfa_attn_bwd needs (0 for invalid sizes or d). */
size_t sfa_attn_bwd_workspace(int B, int Hq, int Hkv, int n, int d);

/*
 * Bytes of device workspace sfa_attn_decode needs for these sizes.
 */
size_t sfa_attn_decode_workspace(int B, int Hq, int Lmax, int d);

/*
 * SFA decode step (App. B, KV-cache attention with one new query per
 * sequence): each query code attends to the first seq_len[b] cached keys
 * (all of them allowed), with the same s, O and LSE definitions as
 * sfa_attn_fwd.  The context is split into chunks processed in parallel and
 * the partial (max, sum, output) triples are merged by their LSE.
 * With window > 0 the query, the token at position L - 1 (L = seq_len[b]),
 * sees only keys j > L - 1 - window and the n_global leading tokens (all
 * keys if it is itself one of them), as row L - 1 of sfa_attn_fwd with the
 * same window; context outside is skipped.
 *
 * q_idx, q_val    [B, Hq, k]          query codes (q_idx_t, q_val_t)
 * kc_idx, kc_val  [B, Hkv, Lmax, k]   cached key codes (kc_idx_t, kc_val_t)
 * v_cache         [B, Hkv, Lmax, d]   cached values (v_t)
 * seq_len         [B] int32 on the device, each in [1, Lmax]; NULL means
 *                 every sequence holds Lmax keys.  Values outside the range
 *                 are clamped into [0, Lmax]; a sequence with 0 keys gets
 *                 O = 0 and LSE = -inf.
 * o               [B, Hq, d] (o_t);  lse [B, Hq] float32 or NULL.
 * ws, ws_bytes    caller-owned device workspace of at least
 *                 sfa_attn_decode_workspace(B, Hq, Lmax, d) bytes; its
 *                 contents need no initialisation and are scratch after the
 *                 call.  Concurrent calls must use distinct workspaces.
 * d in {64, 128} with Hq / Hkv a power of two runs the tuned kernel (16-byte
 * aligned cache arrays); other d <= 256 and other group sizes run a float32
 * kernel with the same chunks and merge (any Hq / Hkv <= 8, no alignment
 * needs).
 * Limits: B, Hq, Hkv, Lmax >= 1; Lmax <= 2^30; Hq % Hkv == 0; Hq / Hkv <= 8;
 *         B * Hkv <= 65535; 1 <= k <= d <= 256; window, n_global >= 0.
 * Errors: SFA_EINVAL, SFA_ENOTSUP, SFA_ENOSPC (ws_bytes too small), SFA_EHIP.
 */
sfa_status sfa_attn_decode(const void* q_idx, const void* q_val,
                           const void* kc_idx, const void* kc_val,
                           const void* v_cache, const int32_t* seq_len,
                           int B, int Hq, int Hkv, int Lmax, int d, int k,
                           float scale, int window, int n_global,
                           int q_idx_t, int q_val_t, int kc_idx_t, int kc_val_t,
                           int v_t, int o_t,
                           void* o, float* lse,
                           void* ws, size_t ws_bytes, void* stream);

/*
 * sfa_attn_decode without a caller workspace and without any allocation, for
 * callers that cannot allocate device memory around the call (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc).
 *
 * Same arguments, definitions, kernels and results (bit for bit) as
 * sfa_attn_decode, minus ws / ws_bytes.  The partial (max, sum, output)
 * triples of the context chunks go to a static device scratch array of the
 * library, SFA_DECODE_NOALLOC_MAX_BYTES per GPU, which each GPU the library
 * runs on holds until the process ends; its device address is looked up
 * once per device, on the first call with that device current.  The call
 * allocates nothing and calls no allocating routine.  Every call on one GPU
 * shares that GPU's scratch: calls that overlap in time on one GPU (other
 * streams, other threads) race on it and must not be issued.  No part of the
 * scratch needs to start at zero: each partial is written before it is read.
 * Errors: as sfa_attn_decode; SFA_ENOSPC when the partials,
 * sfa_attn_decode_workspace(B, Hq, Lmax, d) bytes, exceed
 * SFA_DECODE_NOALLOC_MAX_BYTES (at d = 128 and 4096-key chunks: B * Hq *
 * ceil(Lmax / 4096) <= 64,527 query-head chunks, e.g. 64 sequences x 32
 * heads x 64K keys); SFA_EHIP if the scratch address cannot be looked up.
 */
#define SFA_DECODE_NOALLOC_MAX_BYTES ((size_t)32 << 20)
sfa_status sfa_attn_decode_noalloc(const void* q_idx, const void* q_val,
                                   const void* kc_idx, const void* kc_val,
                                   const void* v_cache, const int32_t* seq_len,
                                   int B, int Hq, int Hkv, int Lmax, int d, int k,
                                   float scale, int window, int n_global,
                                   int q_idx_t, int q_val_t, int kc_idx_t, int kc_val_t,
                                   int v_t, int o_t,
                                   void* o, float* lse, void* stream);

/*
 * CSR code storage to fixed-width codes (Sec. 2, sparse formats; App. J: the
 * paper stores codes as CSR with int32 indptr, int8 indices, fp16 values).
 *
 * indptr   [rows + 1] int32 on the device: row r holds entries
 *          indptr[r] .. indptr[r+1]-1 of indices / values, at most kmax of
 *          them, with distinct indices in [0, d) (any order).
 * indices  [nnz] of indices_t (SFA_I32 | SFA_I16 | SFA_U8).
 * values   [nnz] of values_t (SFA_F32 | SFA_BF16 | SFA_F16).
 * idx, val [rows, kmax] of idx_t / values_t: each row's own entries plus
 *          zero-valued entries at the lowest coordinates it does not hold,
 *          kmax in all, in ascending index order.  Values are copied bit for
 *          bit.  The result is the same matrix as the CSR input, in the form
 *          every attention entry point takes (with k = kmax); rows shorter
 *          than kmax are padded the way Top-k coding treats rows with fewer
 *          than k nonzeros.
 * Rows longer than kmax keep their first kmax entries; indices outside
 * [0, d) are ignored (violated preconditions: undefined results, no fault).
 * Limits: 1 <= kmax <= d <= 256; rows >= 0 (0 is a no-op).
 * Errors: SFA_EINVAL, SFA_ENOTSUP (d > 256), SFA_EHIP.
 */
sfa_status sfa_csr_to_codes(const int32_t* indptr, const void* indices, int indices_t,
                            const void* values, int values_t, int64_t rows, int d, int kmax,
                            void* idx, int idx_t, void* val, void* stream);

/*
 * KV-cache maintenance for decode (App. B: generation extends the cache by
 * one coded key and its value per token; App. J: keys are stored as codes).
 *
 * Paged cache.  A pool of num_pages pages, each holding page_size
 * consecutive positions of one sequence for all Hkv heads:
 *     kc_idx, kc_val  [num_pages, Hkv, page_size, k]
 *     v_cache         [num_pages, Hkv, page_size, d]
 * block_table [B, max_pages] int32 on the device: position j of sequence b
 * lives in page block_table[b * max_pages + j / page_size] at slot
 * j % page_size.  A sequence holds at most max_pages * page_size positions.
 * The caller owns the pool and the table and decides which pages a sequence
 * gets; pages shared by two sequences must not be appended to by both.
 */

/*
 * Append new tokens to a contiguous or paged cache (Top-k coding of the keys,
 * Sec. 3.1, Eqs. (3)-(4), fused with the cache write).
 *
 * k_new    [B, Hkv, T, d] float32 dense keys; coded like sfa_topk_encode
 *          (k coordinates of largest |x|, ties to the lower index, ascending)
 *          into kc_idx_t (SFA_I16 | SFA_I32) / kc_val_t (SFA_BF16: round to
 *          nearest even | SFA_F32: bit copy).
 * v_new    [B, Hkv, T, d] values (v_new_t), stored as v_t (float32 to bf16
 *          rounds to nearest even; bf16 to float32 is exact).
 * n_new    [B] int32 on the device, tokens of sequence b to append (clamped
 *          into [0, T]); NULL means T for every sequence.
 * seq_len  [B] int32 on the device, in/out: on entry each sequence's length,
 *          which is the position of its first new token; on return (in
 *          stream order) min(length + appended, capacity).
 * block_table, max_pages, page_size, num_pages: the paged layout above
 *          (page_size a power of two); with block_table NULL the cache is
 *          contiguous [B, Hkv, page_size, ...] (page_size = Lmax, any value;
 *          max_pages and num_pages ignored).
 * Tokens whose position reaches the capacity, or whose page id lies outside
 * [0, num_pages), are not written.  With T == 0 only the clamping of seq_len
 * into [0, capacity] happens.
 * Limits: 1 <= d <= 256; 1 <= k <= d; B * Hkv * T <= 2^31;
 *         max_pages * page_size <= 2^30.
 * Errors: SFA_EINVAL, SFA_ENOTSUP (d > 256), SFA_EHIP.
 */
sfa_status sfa_kv_append(const float* k_new, const void* v_new, const int32_t* n_new,
                         int32_t* seq_len, int B, int Hkv, int T, int d, int k,
                         const int32_t* block_table, int max_pages, int page_size,
                         int num_pages, void* kc_idx, void* kc_val, void* v_cache,
                         int kc_idx_t, int kc_val_t, int v_new_t, int v_t, void* stream);

/*
 * SFA decode step over a paged cache (App. B), optionally coding the query
 * inside the decode kernel.
 *
 * q               [B, Hq, d] float32 dense query, coded in the kernel exactly
 *                 as sfa_topk_encode codes it (float32 values); q_idx and
 *                 q_val must then be NULL.  Or q NULL and q_idx, q_val
 *                 [B, Hq, k] query codes (q_idx_t, q_val_t), as in
 *                 sfa_attn_decode.
 * kc_idx, kc_val, v_cache, block_table, max_pages, page_size, num_pages:
 *                 the paged layout above; page_size a power of two >= 16.
 *                 Page ids outside [0, num_pages) are clamped into range
 *                 (undefined results, no fault).
 * seq_len         [B] int32 on the device (clamped into
 *                 [0, max_pages * page_size]) or NULL for full sequences.
 * o, lse, ws, ws_bytes, scale, window, n_global, dtypes: as
 *                 sfa_attn_decode, with the
 *                 workspace sized by
 *                 sfa_attn_decode_workspace(B, Hq, max_pages * page_size, d).
 * The result equals sfa_attn_decode on the gathered contiguous cache (same
 * chunking and summation order, hence the same bits).
 * Limits: as sfa_attn_decode; max_pages * page_size <= 2^30.
 * Errors: SFA_EINVAL, SFA_ENOTSUP, SFA_ENOSPC, SFA_EHIP.
 */
sfa_status sfa_attn_decode_paged(const float* q, const void* q_idx, const void* q_val,
                                 const void* kc_idx, const void* kc_val, const void* v_cache,
                                 const int32_t* block_table, int max_pages, int page_size,
                                 int num_pages, const int32_t* seq_len, int B, int Hq, int Hkv,
                                 int d, int k, float scale, int window, int n_global,
                                 int q_idx_t, int q_val_t,
                                 int kc_idx_t, int kc_val_t, int v_t, int o_t, void* o,
                                 float* lse, void* ws, size_t ws_bytes, void* stream);

/*
 * 8-bit KV cache ("SFA (quant)", App. E comparison table: SFA combined with
 * 8-bit quantisation of the activations; with a KV cache, the cached keys
 * and values are those activations).  Every cached key code and every value
 * row is one int8 row with its float32 scale (symmetric, per row):
 *     s = max_u |x_u| / 127,   q_u = round-half-even(x_u / s) in [-127, 127]
 * (both float32 divisions correctly rounded; a zero row has s = 0, q = 0).
 * The cache then stands for the values q_u * s, and the attention computed
 * over it is the plain SFA decode of those values.
 *
 * Layout (contiguous: rows (b, h, j) of [B, Hkv, Lmax]; paged: rows
 * (page, h, slot) of [num_pages, Hkv, page_size], as for sfa_kv_append):
 *     kc_idx   [rows, k] indices (kc_idx_t)      kc_val [rows, k] int8
 *     kc_scale [rows] float32                    v_cache [rows, d] int8
 *     v_scale  [rows] float32
 * 184 bytes per cached key and KV head at d = 128, k = 16 with int16
 * indices, against 320 with int16 / bf16 codes and bf16 V.
 */

/*
 * Append to an 8-bit cache: as sfa_kv_append (Top-k coding of k_new, the
 * same positions, capacity and page rules, seq_len advanced), with the kept
 * code values quantised as one row (its scale to kc_scale) and the value
 * row v_new (v_new_t SFA_F32 or SFA_BF16, widened exactly) quantised as one
 * row (its scale to v_scale).  Indices are stored as kc_idx_t (SFA_I32,
 * SFA_I16 or SFA_U8).
 * Limits and errors: as sfa_kv_append.
 */
sfa_status sfa_kv_append_q8(const float* k_new, const void* v_new, const int32_t* n_new,
                            int32_t* seq_len, int B, int Hkv, int T, int d, int k,
                            const int32_t* block_table, int max_pages, int page_size,
                            int num_pages, void* kc_idx, int8_t* kc_val, float* kc_scale,
                            int8_t* v_cache, float* v_scale, int kc_idx_t, int v_new_t,
                            void* stream);

/*
 * Decode step over an 8-bit cache: sfa_attn_decode (or, with block_table
 * non-NULL, sfa_attn_decode_paged, including the dense query q coded in the
 * kernel) with key j's code values q_ju * ks_j and value row v_j = qv_j * vs_j.
 * The score is the integer-coded overlap sum times scale * ks_j (float32);
 * the probability enters P.V times vs_j, the int8 values widened exactly.
 * block_table NULL: contiguous cache [B, Hkv, page_size, ...] (page_size =
 * Lmax; max_pages and num_pages ignored).  seq_len, window, n_global, o,
 * lse, ws (sized by sfa_attn_decode_workspace(B, Hq, capacity, d)) as
 * sfa_attn_decode.
 * Limits: kc_idx_t SFA_I16, k in {8, 16, 32}, d in {64, 128}, Hq / Hkv a
 * power of two <= 8 (SFA_ENOTSUP otherwise); 16-byte aligned cache arrays;
 * paged: page_size a power of two >= 16.
 * Errors: SFA_EINVAL, SFA_ENOTSUP, SFA_ENOSPC, SFA_EHIP.
 */
sfa_status sfa_attn_decode_q8(const float* q, const void* q_idx, const void* q_val,
                              const void* kc_idx, const int8_t* kc_val, const float* kc_scale,
                              const int8_t* v_cache, const float* v_scale,
                              const int32_t* block_table, int max_pages, int page_size,
                              int num_pages, const int32_t* seq_len, int B, int Hq, int Hkv,
                              int d, int k, float scale, int window, int n_global, int q_idx_t,
                              int q_val_t, int kc_idx_t, int o_t, void* o, float* lse, void* ws,
                              size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SFA_H */
