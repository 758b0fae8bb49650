// SFA decode step (App. B, KV-cache attention) on gfx950.
//
// The cache holds sparse key codes (k index/value pairs per key) and dense V.
// Grid = (context chunks, B * Hkv): a workgroup streams one chunk of one KV
// head and serves all G query heads of the group from each load.
//   scores: lane = key.  The G query codes are densified once into an LDS
//           table qd[u][h]; a key's score for head h is
//           scale * sum_t kval_t * qd[kidx_t][h] -- zero-cost for coordinates
//           the query does not hold, which is exactly the overlap sum.
//   softmax: online, base 2, the running max kept wave-uniform per head.
//   P.V:    lanes over (8 dims, key subset); float32 FMAs.
// Each workgroup writes one partial (max, sum, unnormalised output) per query
// head; a second kernel merges the chunks by their LSE.
//
// Cache layouts: contiguous [B, Hkv, Lmax, ...], or paged -- a pool of pages
// [num_pages, Hkv, P, ...] with a block table mapping each run of P
// positions of a sequence to a page (P a power of two >= 16).  A wave's
// 1024-position range spans at most 64 pages; their ids are loaded once into
// one register (lane l: the range's l-th page) and read back by lane shuffle
// for the codes (lane = key) and by readlane for V, whose keys within one
// wide load always share a page.
// Query: codes, or the dense float32 query coded in the prologue with the
// same Top-k selection as the coding kernel (one wavefront per head).
#pragma once

#include "sfa_device.h"
#include "sfa_launch.h"
#include "sfa_topk.h"

namespace sfa {

constexpr int kDecWaves = 4;
constexpr int kDecThreads = 64 * kDecWaves;
constexpr int kDecChunk = kDecodeChunk;  // keys per workgroup
constexpr int kDecMaxG = 8;

struct DecParams {
  const void* q_idx;
  const void* q_val;
  const void* kc_idx;
  const void* kc_val;
  const void* v;
  const int32_t* seq_len;
  float* ws_m;  // [B*Hq, nch]
  float* ws_l;  // [B*Hq, nch]
  float* ws_o;  // [B*Hq, nch, D]
  int Hq, Hkv, Lmax, k, nch;  // nch: partial slots per (b, h)
  float scale_log2;
  int qifmt, qvfmt, kifmt, kvfmt;
  const float* q_dense;   // [B, Hq, D] or null (then q_idx / q_val)
  const int32_t* table;   // paged: [B, max_pages]
  int max_pages, log2P, num_pages;
  int window, n_global;   // token pattern (window 0: all cached keys)
  int nvc;                // window: workgroups per (b, KV head) (0: nch)
  // 8-bit cache: int8 code values and value rows, one float32 scale per row
  const float* kc_scale;  // [cache rows]
  const float* v_scale;   // [cache rows]
};

// Kernel parameters of a decode call (sfa_decode.hip), and the merge of its
// chunk partials, shared by the bf16 / float32 and the 8-bit cache launchers.
DecParams make_dec_params(const DecodeArgs& a);
hipError_t launch_decode_combine(const DecParams& p, const DecodeArgs& a, hipStream_t stream);

__device__ __forceinline__ int seq_len_of(const int32_t* seq_len, int b, int Lmax) {
  if (!seq_len) return Lmax;
  int L = seq_len[b];
  return L < 0 ? 0 : (L > Lmax ? Lmax : L);
}

namespace {

// KC8 > 0: cache codes with k = 8 * KC8 in one of two compact formats --
// int16 indices with bf16 values, or (C8) uint8 indices with float16 values --
// loaded as 16-byte vectors and prefetched one 64-key sub-block ahead, with
// the sub-block's V (bf16) in flight during its score phase.  KC8 = 0: any
// format and k, element loads issued as a batch per sub-block.
// Q8 (with KC8 > 0, int16 indices): the 8-bit cache -- int8 code values and
// int8 value rows, each key row and value row with its float32 scale.  A
// key's score is its integer-coded overlap sum times its scale (folded into
// the softmax's base-2 factor); its probability enters P.V times the value
// row's scale, so the value rows stay integers until the float32 FMAs.
template <int D, int G, bool VBF16, int KC8, bool C8, bool PAGED, bool Q8 = false>
__global__ __launch_bounds__(kDecThreads) void sfa_decode_kernel(DecParams p) {
  static_assert(!Q8 || (KC8 > 0 && !C8), "8-bit cache: the vector path, int16 indices");
  constexpr int DL = D / 8;     // lanes covering one key's D values (8 each)
  constexpr int KPL = 64 / DL;  // keys per wave-wide V load
  constexpr int NR = 64 / KPL;  // V loads per lane per 64-key sub-block
  __shared__ float qd[D][G];
  // P of the wave's 64 keys, [key][head] in float32; the 8-bit cache keeps
  // them as float16 pairs instead, in the order its P.V loop reads them:
  // slot (r / 2) * KPL + ksub holds keys r * KPL + ksub (low half) and
  // (r + 1) * KPL + ksub (high half), r even, one pair per head.
  __shared__ float pbuf[kDecWaves][64][G];
  uint32_t* pb2 = (uint32_t*)&pbuf[0][0][0];  // 8-bit cache: [wave][32 slots][G]
  __shared__ float red_m[kDecWaves][G], red_l[kDecWaves][G];
  __shared__ float red_o[kDecWaves][G][D];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: per-wave values stay scalar
  const int bh = blockIdx.y;
  const int b = bh / p.Hkv, hkv = bh - b * p.Hkv;
  const int L = seq_len_of(p.seq_len, b, p.Lmax);
  // Token window: the query (position L - 1) sees keys [0, wg) and [wlo, L)
  // only.  The grid then covers only the chunks holding them: workgroup x
  // takes the x-th of the global chunks followed by the window's chunks, and
  // writes its partial to slot x (past the last such chunk: an empty one).
  const bool winq = p.window > 0 && L - 1 >= p.n_global;
  const int wlo = winq ? max(0, L - p.window) : 0;
  const int wg = winq ? min(p.n_global, L) : 0;
  int chunk = blockIdx.x;
  if (winq) {
    const int ngc = (wg + kDecChunk - 1) / kDecChunk;
    const int wc0 = max(ngc, wlo / kDecChunk);
    chunk = chunk < ngc ? chunk : wc0 + (chunk - ngc);
  }
  const int c0 = chunk * kDecChunk;  // at most Lmax + 2 chunks: no overflow
  const int c1 = min(L, c0 + kDecChunk);
  const int k = p.k;
  const int dmask = D - 1;

  // densify the G query codes: qd[u][h]
  if (p.q_dense) {
    // code each dense query row here: one wavefront per head, kept
    // coordinates keep their float32 value, the rest are zero
    constexpr int E = D / 64;
    for (int h = __builtin_amdgcn_readfirstlane(wave); h < G; h += kDecWaves) {
      const float* qr = p.q_dense + ((int64_t)b * p.Hq + hkv * G + h) * D;
      uint32_t bits[E], key[E];
      bool sel[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        bits[e] = __float_as_uint(qr[lane + 64 * e]);
        key[e] = topk_key(bits[e], true);
      }
      topk_select<E>(key, k, sel);
#pragma unroll
      for (int e = 0; e < E; ++e) qd[lane + 64 * e][h] = sel[e] ? __uint_as_float(bits[e]) : 0.f;
    }
  } else {
    for (int x = tid; x < D * G; x += kDecThreads) (&qd[0][0])[x] = 0.f;
    __syncthreads();
    for (int x = tid; x < G * k; x += kDecThreads) {
      const int h = x / k, t = x - h * k;
      const int64_t qi = ((int64_t)b * p.Hq + hkv * G + h) * k + t;
      const int u = load_idx(p.q_idx, qi, p.qifmt, dmask);
      qd[u][h] = load_val(p.q_val, qi, p.qvfmt);
    }
  }
  __syncthreads();

  float m_run[G], l_lane[G], o[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m_run[h] = -INFINITY;
    l_lane[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
  }

  const int64_t kv_row0 = ((int64_t)b * p.Hkv + hkv) * p.Lmax;
  const int dsub = lane % DL;  // 8-dim group of this lane in the P.V phase
  const int ksub = lane / DL;  // key offset within a wave-wide V load
  const int per_wave = kDecChunk / kDecWaves;
  int w0 = c0 + wave * per_wave;
  int w1 = min(c1, w0 + per_wave);
  // A wave range inside the window's gap does nothing; one that starts in it
  // starts at the window (64-aligned; the keys before wlo are masked).
  if (winq && w0 >= wg) {
    if (w1 <= wlo) w1 = w0;
    else w0 = max(w0, wlo & ~63);
  }
  auto key_ok = [&](int j) { return j >= wlo || j < wg; };

  // Row of key j in the cache arrays.  Paged: lane l of `tblv` holds the
  // page of the wave's l-th page-sized run (ids clamped into the pool).
  int tblv = 0;
  const int pg0 = PAGED ? (w0 >> p.log2P) : 0;
  if constexpr (PAGED) {
    if (w0 < w1) {
      // <= 64 (P >= 16; w0 is 1024-aligned, or 64-aligned at a window start)
      const int npg = ((w1 - 1) >> p.log2P) - pg0 + 1;
      if (lane < npg) {
        const int pg = p.table[(int64_t)b * p.max_pages + pg0 + lane];
        tblv = min(max(pg, 0), p.num_pages - 1);
      }
    }
  }
  const int pmask = (1 << (PAGED ? p.log2P : 0)) - 1;
  auto paged_row = [&](int pg, int j) -> int64_t {
    return (((int64_t)pg * p.Hkv + hkv) << p.log2P) + (j & pmask);
  };
  // j may differ across lanes (w0 <= j < w1)
  auto row_of = [&](int j) -> int64_t {
    if constexpr (PAGED) return paged_row(__shfl(tblv, (j >> p.log2P) - pg0, 64), j);
    else return kv_row0 + j;
  };
  // jb wave-uniform (w0 <= jb < w1), j on the same page as jb
  auto row_near = [&](int jb, int j) -> int64_t {
    if constexpr (PAGED) return paged_row(__builtin_amdgcn_readlane(tblv, (jb >> p.log2P) - pg0), j);
    else return kv_row0 + j;
  };

  // ---- per-sub-block pieces ----
  // online softmax of the lane's key scores s[h] (valid: ok), in base-2
  // exponents s * kfac; writes P (times pfac) to pbuf
  auto softmax_block = [&](float (&s)[G], bool ok, float kfac, float pfac) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float tt = ok ? s[h] * kfac : -INFINITY;
      const float mb = wave_max_dpp(tt);
      const float m_new = fmaxf(m_run[h], mb);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run[h] - m_use);
      const float pj = __builtin_amdgcn_exp2f(tt - m_use);
      l_lane[h] = l_lane[h] * alpha + pj;
      m_run[h] = m_new;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] *= alpha;
      if constexpr (Q8) {
        const int r = lane / KPL;
        _Float16* dst = (_Float16*)&pb2[(wave * 32 + (r >> 1) * KPL + lane % KPL) * G + h];
        dst[r & 1] = (_Float16)(pj * pfac);
      } else {
        pbuf[wave][lane][h] = pj * pfac;
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  };
  auto pv_accum = [&](int jj, const float (&vv)[8]) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float ph = pbuf[wave][jj][h];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] = fmaf(ph, vv[e], o[h][e]);
    }
  };

  if constexpr (KC8 > 0) {
    // ---------------- vectorized, prefetched path ----------------
    // a key's codes as 32-bit words: indices (2 or 4 per word), values (2 per word)
    constexpr int NIW = C8 ? 2 * KC8 : 4 * KC8, NVW = Q8 ? 2 * KC8 : 4 * KC8;
    uint32_t cidx[NIW], cval[NVW];
    float ksc = 1.f, vsc = 1.f;  // 8-bit cache: the key's code and value-row scales
    auto load_codes = [&](int sb) {
      // contiguous cache: a wave-uniform base row and 32-bit lane offsets
      const int64_t row = PAGED ? row_of(min(sb + lane, w1 - 1)) : kv_row0 + sb;
      const int lo = PAGED ? 0 : min(lane, w1 - 1 - sb);
      if constexpr (Q8) {
        ksc = (p.kc_scale + row)[lo];
        vsc = (p.v_scale + row)[lo];
      }
      const uint32_t* pi = (const uint32_t*)((const unsigned char*)p.kc_idx + row * (4 * NIW) +
                                             (uint32_t)lo * (4 * NIW));
      const uint32_t* pv = (const uint32_t*)((const unsigned char*)p.kc_val + row * (4 * NVW) +
                                             (uint32_t)lo * (4 * NVW));
      if constexpr (NIW % 4 == 0) {
#pragma unroll
        for (int c = 0; c < NIW / 4; ++c) {
          const uint4 w = ((const uint4*)pi)[c];
          cidx[4 * c] = w.x; cidx[4 * c + 1] = w.y; cidx[4 * c + 2] = w.z; cidx[4 * c + 3] = w.w;
        }
      } else {
        const uint2 w = *(const uint2*)pi;
        cidx[0] = w.x; cidx[1] = w.y;
      }
      if constexpr (NVW % 4 == 0) {
#pragma unroll
        for (int c = 0; c < NVW / 4; ++c) {
          const uint4 w = ((const uint4*)pv)[c];
          cval[4 * c] = w.x; cval[4 * c + 1] = w.y; cval[4 * c + 2] = w.z; cval[4 * c + 3] = w.w;
        }
      } else {
        const uint2 w = *(const uint2*)pv;
        cval[0] = w.x; cval[1] = w.y;
      }
    };
    if (w0 < w1) load_codes(w0);
    for (int sb = w0; sb < w1; sb += 64) {
      // V of this sub-block: in flight during the score phase (8 dims of a
      // key per lane: 16 bytes of bf16, or 8 bytes of int8)
      uint4 vraw[Q8 ? 1 : NR];
      uint2 vraw8[Q8 ? NR : 1];
      constexpr int VB = Q8 ? 1 : 2;  // bytes per V value
      if constexpr (!PAGED) {
        // a wave-uniform base row and 32-bit lane offsets (keys clamped
        // into the range)
        const unsigned char* vb = (const unsigned char*)p.v + (kv_row0 + sb) * (int64_t)(D * VB);
        const int jlast = w1 - 1 - sb;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const int jj = min(r * KPL + ksub, jlast);
          const unsigned char* src = vb + (uint32_t)((jj * D + dsub * 8) * VB);
          if constexpr (Q8) vraw8[r] = *(const uint2*)src;
          else vraw[r] = *(const uint4*)src;
        }
      } else {
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const int jg = min(sb + r * KPL + ksub, w1 - 1);
          const int64_t row = row_near(min(sb + r * KPL, w1 - 1), jg);
          if constexpr (Q8)
            vraw8[r] = *(const uint2*)((const int8_t*)p.v + row * D + dsub * 8);
          else
            vraw[r] = *(const uint4*)((const uint16_t*)p.v + row * D + dsub * 8);
        }
      }
      // scores, lane = key
      float s[G];
#pragma unroll
      for (int h = 0; h < G; ++h) s[h] = 0.f;
#pragma unroll
      for (int e = 0; e < 8 * KC8; ++e) {
        const int u = (C8 ? (int)((cidx[e >> 2] >> (8 * (e & 3))) & 0xffu)
                          : (int)((cidx[e >> 1] >> (16 * (e & 1))) & 0xffffu)) & dmask;
        float kv;
        if constexpr (Q8) {
          kv = (float)(int)(int8_t)((cval[e >> 2] >> (8 * (e & 3))) & 0xffu);
        } else {
          const uint32_t h16 = (e & 1) ? (cval[e >> 1] >> 16) : (cval[e >> 1] & 0xffffu);
          kv = C8 ? f16_bits_to_f32(h16) : __uint_as_float(h16 << 16);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) s[h] = fmaf(kv, qd[u][h], s[h]);
      }
      softmax_block(s, sb + lane < w1 && key_ok(sb + lane), Q8 ? p.scale_log2 * ksc : p.scale_log2,
                    vsc);
      if (sb + 64 < w1) load_codes(sb + 64);  // next sub-block's codes during P.V
      // P.V: lanes over (8 dims, key subset)
      if constexpr (Q8) {
        // Two keys per step: their int8 values of a dimension as a float16
        // pair, their probabilities (times the value rows' scales) rounded
        // to a float16 pair, and one float32 two-term dot product per head
        // and dimension.  The pair is built by byte placement: with
        // u = q + 128 (q xor 0x80), the float16 bits 0x64uu are 1024 + u
        // exactly, and one packed float16 add of -1152 leaves q exactly.
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
        const h2 off = {(_Float16)-1152.f, (_Float16)-1152.f};
#pragma unroll
        for (int r = 0; r < NR; r += 2) {
          const int j0 = r * KPL + ksub, j1 = j0 + KPL;
          (void)j1;
          h2 pp[G];
          const uint32_t* ps = &pb2[(wave * 32 + (r >> 1) * KPL + ksub) * G];
#pragma unroll
          for (int h = 0; h < G; ++h) pp[h] = __builtin_bit_cast(h2, ps[h]);
#pragma unroll
          for (int half = 0; half < 2; ++half) {  // dims 4 half .. 4 half + 3
            const uint32_t x0 = (half ? vraw8[r].y : vraw8[r].x) ^ 0x80808080u;
            const uint32_t x1 = (half ? vraw8[r + 1].y : vraw8[r + 1].x) ^ 0x80808080u;
            // bytes (x0.b0, x1.b0, x0.b1, x1.b1) and (x0.b2, x1.b2, x0.b3, x1.b3)
            const uint32_t il[2] = {__builtin_amdgcn_perm(x1, x0, 0x05010400u),
                                    __builtin_amdgcn_perm(x1, x0, 0x07030602u)};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              // (x0.b_e, 0x64, x1.b_e, 0x64): the float16 pair (1024 + u0, 1024 + u1)
              const uint32_t bits = __builtin_amdgcn_perm(0x64646464u, il[e >> 1],
                                                          (e & 1) ? 0x04030402u : 0x04010400u);
              const h2 vp = __builtin_bit_cast(h2, bits) + off;
#pragma unroll
              for (int h = 0; h < G; ++h)
                o[h][4 * half + e] = __builtin_amdgcn_fdot2(vp, pp[h], o[h][4 * half + e], false);
            }
          }
        }
      }
#pragma unroll
      for (int r = 0; r < (Q8 ? 0 : NR); ++r) {
        float vv[8];
        {
          vv[0] = __uint_as_float(vraw[r].x << 16); vv[1] = __uint_as_float(vraw[r].x & 0xffff0000u);
          vv[2] = __uint_as_float(vraw[r].y << 16); vv[3] = __uint_as_float(vraw[r].y & 0xffff0000u);
          vv[4] = __uint_as_float(vraw[r].z << 16); vv[5] = __uint_as_float(vraw[r].z & 0xffff0000u);
          vv[6] = __uint_as_float(vraw[r].w << 16); vv[7] = __uint_as_float(vraw[r].w & 0xffff0000u);
        }
        pv_accum(r * KPL + ksub, vv);
      }
      __builtin_amdgcn_wave_barrier();
    }
  } else {
    // ---------------- generic path: any code format and k ----------------
    for (int sb = w0; sb < w1; sb += 64) {
      const int j = min(sb + lane, w1 - 1);
      const bool ok = sb + lane < w1 && key_ok(sb + lane);
      float s[G];
#pragma unroll
      for (int h = 0; h < G; ++h) s[h] = 0.f;
      const int64_t cbase = row_of(j) * k;
      for (int t = 0; t < k; ++t) {
        const int u = load_idx(p.kc_idx, cbase + t, p.kifmt, dmask);
        const float kv = load_val(p.kc_val, cbase + t, p.kvfmt);
#pragma unroll
        for (int h = 0; h < G; ++h) s[h] = fmaf(kv, qd[u][h], s[h]);
      }
      softmax_block(s, ok, p.scale_log2, 1.f);
      for (int r = 0; r < 64; r += KPL) {
        const int jj = r + ksub;
        const int jg = min(sb + jj, w1 - 1);
        const int64_t row = row_near(min(sb + r, w1 - 1), jg);
        float vv[8];
        if constexpr (VBF16) {
          const uint4 raw = *(const uint4*)((const uint16_t*)p.v + row * D + dsub * 8);
          vv[0] = __uint_as_float(raw.x << 16); vv[1] = __uint_as_float(raw.x & 0xffff0000u);
          vv[2] = __uint_as_float(raw.y << 16); vv[3] = __uint_as_float(raw.y & 0xffff0000u);
          vv[4] = __uint_as_float(raw.z << 16); vv[5] = __uint_as_float(raw.z & 0xffff0000u);
          vv[6] = __uint_as_float(raw.w << 16); vv[7] = __uint_as_float(raw.w & 0xffff0000u);
        } else {
          const float4* src = (const float4*)((const float*)p.v + row * D + dsub * 8);
          const float4 a = src[0], c = src[1];
          vv[0] = a.x; vv[1] = a.y; vv[2] = a.z; vv[3] = a.w;
          vv[4] = c.x; vv[5] = c.y; vv[6] = c.z; vv[7] = c.w;
        }
        pv_accum(jj, vv);
      }
      __builtin_amdgcn_wave_barrier();
    }
  }

  // ---- reduce within the wave: sums over lanes, outputs over key subsets ----
#pragma unroll
  for (int h = 0; h < G; ++h) {
    l_lane[h] = wave_sum(l_lane[h]);
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int off = DL; off < 64; off <<= 1) o[h][e] += __shfl_xor(o[h][e], off, 64);
  }
  if (lane < DL) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) red_o[wave][h][lane * 8 + e] = o[h][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) { red_m[wave][h] = m_run[h]; red_l[wave][h] = l_lane[h]; }
  }
  __syncthreads();
  // ---- merge the waves and write this chunk's partial ----
  for (int x = tid; x < G * D; x += kDecThreads) {
    const int h = x / D, dd = x - h * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, red_m[w][h]);
    const float Mu = (M == -INFINITY) ? 0.f : M;
    float lsum = 0.f, osum = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float sc = exp2f(red_m[w][h] - Mu);
      lsum += sc * red_l[w][h];
      osum += sc * red_o[w][h][dd];
    }
    const int64_t slot = ((int64_t)b * p.Hq + hkv * G + h) * p.nch + blockIdx.x;
    p.ws_o[slot * D + dd] = osum;
    if (dd == 0) { p.ws_m[slot] = M; p.ws_l[slot] = lsum; }
  }
}

}  // namespace
}  // namespace sfa
