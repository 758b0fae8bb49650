// SFA forward (Sec. 3.1-3.2) on gfx950, inverted-index variant.
//
// This variant follows the sparse-overlap formulation literally; the default
// forward (sfa_fwd.hip) computes the same scores on the matrix cores.
//
// Workgroup = 4 wavefronts = 128 query rows: the G query heads of one KV
// head times BR = 128 / G positions, so all G heads share every key tile.
// Per key tile of BC = 64 keys:
//   1. the tile's BC*k key codes are counting-sorted into an LDS inverted
//      index by (coordinate u, key parity): bucket 2u + p lists the keys of
//      parity p that hold u;
//   2. thread (row r, parity p) walks, for each nonzero (u, q_u) of row r,
//      bucket 2u + p and adds q_u * k_u into the score tile's entry
//      (key, r), so only overlapping coordinates cost work.  Each score entry
//      has one owner thread: the adds are plain LDS read-modify-writes, in
//      program order, with no atomics (LDS float atomics run at a fraction
//      of a lane per clock);
//   3. each wavefront reads its 32 rows of the score tile in the register
//      layout of the MFMA B operand, applies scale and the causal mask, runs
//      the online-softmax update (base-2 exponent, scale * log2(e) folded),
//      and clears the tile for the next key tile;
//   4. O^T += V^T P^T on the matrix cores: bf16 V (transposed into LDS while
//      staging) x P split into two bf16 pieces (hi + lo, ~2^-17 relative) with
//      float32 accumulation, or float32 x float32.
// Keys that share no coordinate with a query keep score 0 and still enter
// the softmax, so the result is exactly softmax(Q~ K~^T * scale) V.
#include <mutex>

#include "sfa_device.h"
#include "sfa_launch.h"

namespace sfa {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 32 * kWaves;  // query rows per workgroup
constexpr int kBC = 64;             // keys per tile
constexpr int kSP = kRows + 4;      // score tile [key][row]: key pitch (floats)
constexpr int kVP = kBC + 8;        // transposed-V row pitch (bf16)
constexpr int kMaxK = 64;           // largest supported k

struct FwdParams {
  const void* q_idx;
  const void* q_val;
  const void* k_idx;
  const void* k_val;
  const void* v;
  void* o;
  float* lse;
  int Hq, Hkv, n, k, causal;
  float scale_log2;  // scale * log2(e)
  int ifmt, vfmt, obf16;
  int G, BR, nqb;
  float inv_k;
};

struct FwdLds {
  int s_off, qent_off, kent_off, cnt_off, koff_off, v_off, total;
};

template <int D, bool VBF16>
__host__ __device__ inline FwdLds fwd_lds_layout(int k) {
  FwdLds L;
  int off = 0;
  L.s_off = off;    off += kBC * kSP * 4;
  L.qent_off = off; off += kRows * k * 8;
  L.kent_off = off; off += kBC * k * 8;
  L.cnt_off = off;  off += (2 * D + 1) * 4;
  L.koff_off = off; off += (2 * D + 1) * 4;
  off = (off + 15) & ~15;
  L.v_off = off;    off += VBF16 ? D * kVP * 2 : kBC * D * 4;
  L.total = off;
  return L;
}

// Exclusive scan of cnt[0..D) into off[0..D] by wavefront 0 (off[D] = total).
template <int D>
__device__ __forceinline__ void bucket_offsets(const uint32_t* cnt, uint32_t* off, int lane) {
  constexpr int F = D / 64;  // coordinates per lane, consecutive
  uint32_t c[F];
  uint32_t local = 0;
#pragma unroll
  for (int f = 0; f < F; ++f) { c[f] = cnt[lane * F + f]; local += c[f]; }
  uint32_t incl = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  uint32_t run = incl - local;
#pragma unroll
  for (int f = 0; f < F; ++f) { off[lane * F + f] = run; run += c[f]; }
  if (lane == 63) off[D] = incl;
}

// KM: compile-time bound on k (16 or 64) sizing the per-thread code registers.
template <int D, bool VBF16, int KM>
__global__ __launch_bounds__(kThreads, 2) void sfa_fwd_index_kernel(FwdParams p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const FwdLds L = fwd_lds_layout<D, VBF16>(p.k);
  float* S = (float*)(smem + L.s_off);
  uint2* qent = (uint2*)(smem + L.qent_off);
  uint2* kent = (uint2*)(smem + L.kent_off);
  uint32_t* cnt = (uint32_t*)(smem + L.cnt_off);
  uint32_t* koff = (uint32_t*)(smem + L.koff_off);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int k = p.k;
  const int dmask = D - 1;

  const int qb = p.nqb - 1 - (int)blockIdx.x;  // longest causal blocks first
  const int bh = blockIdx.y;                    // b * Hkv + kv head
  const int b = bh / p.Hkv;
  const int hkv = bh - b * p.Hkv;
  const int i0 = qb * p.BR;
  const int n = p.n;

  // ---------------- the workgroup's query codes, per row -------------------
  // row rho in [0, kRows): query head hkv*G + rho / BR, position i0 + rho % BR;
  // qent[rho * k + t] = (coordinate, value) of its t-th nonzero (rows past n:
  // value 0)
  const int nqe = kRows * k;
  for (int e = tid; e < nqe; e += kThreads) {
    const int rho = (int)(((float)e + 0.5f) * p.inv_k);
    const int t = e - rho * k;
    const int hq = hkv * p.G + rho / p.BR;
    const int i = i0 + rho % p.BR;
    uint2 qe = make_uint2(0u, 0u);
    if (i < n) {
      const int64_t gi = (((int64_t)b * p.Hq + hq) * n + i) * k + t;
      qe = make_uint2((uint32_t)load_idx(p.q_idx, gi, p.ifmt, dmask),
                      __float_as_uint(load_val(p.q_val, gi, p.vfmt)));
    }
    qent[e] = qe;
  }
  // zero the score tile
  for (int x = tid; x < kBC * kSP; x += kThreads) S[x] = 0.f;
  __syncthreads();
  static_assert(kThreads == 2 * kRows, "two threads (key parities) per row");
  constexpr int kKE = kBC * KM / kThreads;  // key code entries per thread and tile
  // score-phase ownership: row sr, key parity spar
  const int sr = tid & (kRows - 1);
  const int spar = tid / kRows;
  float* Scol = S + sr;  // entry (key c, row sr) at Scol[c * kSP]

  // ---------------- per-wave row state (MFMA B-operand layout) ------------
  const int hh = lane >> 5;               // which 8-key half of each 16-key block
  const int rho = wave * 32 + (lane & 31);  // this lane's row
  const int my_i = i0 + rho % p.BR;
  const int my_hq = hkv * p.G + rho / p.BR;
  const bool row_ok = my_i < n;
  float m_run = -INFINITY, l_run = 0.f;
  constexpr int NDB = D / 32;  // 32-wide output dim blocks
  floatx16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  // wave's largest position (rows of one wave share a head when BR >= 32)
  const int wave_i_max = i0 + (wave * 32 + 31) % p.BR;
  const int blk_last = min(n, i0 + p.BR) - 1;
  const int n_keys = p.causal ? blk_last + 1 : n;
  const int ntiles = (n_keys + kBC - 1) / kBC;

  const int64_t kv_base = ((int64_t)b * p.Hkv + hkv) * n;  // row index of key 0

  for (int jt = 0; jt < ntiles; ++jt) {
    const int j0 = jt * kBC;

    // ---- stage V tile into LDS (zero beyond n) ----
    if constexpr (VBF16) {
      uint16_t* Vt = (uint16_t*)(smem + L.v_off);
      const uint16_t* Vg = (const uint16_t*)p.v;
      constexpr int NDP = D / 2;                 // dim pairs
      constexpr int ITEMS = NDP * (kBC / 8);     // (dim pair, 8-key group)
#pragma unroll
      for (int it = tid; it < ITEMS; it += kThreads) {
        const int dp = it % NDP;
        const int kg = it / NDP;
        uint32_t w[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = j0 + kg * 8 + e;
          w[e] = (j < n) ? *(const uint32_t*)(Vg + (kv_base + j) * D + 2 * dp) : 0u;
        }
        uint4 lo, hi;
        lo.x = (w[0] & 0xffffu) | (w[1] << 16); hi.x = (w[0] >> 16) | (w[1] & 0xffff0000u);
        lo.y = (w[2] & 0xffffu) | (w[3] << 16); hi.y = (w[2] >> 16) | (w[3] & 0xffff0000u);
        lo.z = (w[4] & 0xffffu) | (w[5] << 16); hi.z = (w[4] >> 16) | (w[5] & 0xffff0000u);
        lo.w = (w[6] & 0xffffu) | (w[7] << 16); hi.w = (w[6] >> 16) | (w[7] & 0xffff0000u);
        *(uint4*)(Vt + (2 * dp) * kVP + kg * 8) = lo;
        *(uint4*)(Vt + (2 * dp + 1) * kVP + kg * 8) = hi;
      }
    } else {
      float* Vs = (float*)(smem + L.v_off);
      const float* Vg = (const float*)p.v;
      constexpr int N4 = kBC * D / 4;
      for (int it = tid; it < N4; it += kThreads) {
        const int j = it / (D / 4);
        const int c4 = it % (D / 4);
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (j0 + j < n) val = *(const float4*)(Vg + (kv_base + j0 + j) * D + 4 * c4);
        *(float4*)(Vs + j * D + 4 * c4) = val;
      }
    }

    // ---- inverted index of the key tile by (coordinate, key parity): count ----
    for (int f = tid; f <= 2 * D; f += kThreads) cnt[f] = 0;
    __syncthreads();
    int k_slot[kKE], k_f[kKE];
    float k_v[kKE];
    const int nke = kBC * k;
#pragma unroll
    for (int r = 0; r < kKE; ++r) {
      const int e = tid + r * kThreads;
      k_slot[r] = -1;
      k_f[r] = 0;
      k_v[r] = 0.f;
      if (e < nke) {
        const int c = (int)(((float)e + 0.5f) * p.inv_k);
        const int t = e - c * k;
        const int j = j0 + c;
        if (j < n) {
          const int64_t gi = (kv_base + j) * k + t;
          k_f[r] = 2 * load_idx(p.k_idx, gi, p.ifmt, dmask) + (c & 1);
          k_v[r] = load_val(p.k_val, gi, p.vfmt);
          k_slot[r] = (int)atomicAdd(&cnt[k_f[r]], 1u);
        }
      }
    }
    __syncthreads();
    if (wave == 0) bucket_offsets<2 * D>(cnt, koff, lane);
    __syncthreads();
    // ---- place entries: (column byte offset, value) ----
#pragma unroll
    for (int r = 0; r < kKE; ++r) {
      const int e = tid + r * kThreads;
      if (k_slot[r] >= 0) {
        const int c = (int)(((float)e + 0.5f) * p.inv_k);
        kent[koff[k_f[r]] + k_slot[r]] = make_uint2((uint32_t)(c * kSP), __float_as_uint(k_v[r]));
      }
    }
    __syncthreads();

    // ---- overlap scores: each (row, parity) thread walks its row's buckets ----
    // A bucket holds a key at most once, so its four reads and four writes
    // touch distinct entries; a key met again under a later coordinate is
    // read after the earlier write (LDS operations of a wave run in order).
    for (int t = 0; t < k; ++t) {
      const uint2 qe = qent[sr * k + t];
      const float qv = __uint_as_float(qe.y);
      const int bk = 2 * (int)qe.x + spar;
      const int p0 = (int)koff[bk], p1 = (int)koff[bk + 1];
      for (int q = p0; q < p1; q += 4) {
        uint2 ke[4];
        float sv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) ke[u] = kent[min(q + u, p1 - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) sv[u] = Scol[ke[u].x];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (q + u < p1) Scol[ke[u].x] = fmaf(qv, __uint_as_float(ke[u].y), sv[u]);
      }
    }
    __syncthreads();

    // ---- online softmax on this wave's 32 rows, then P.V ----
    float* Srow = S + rho;  // entry (key c, row rho) at Srow[c * kSP]
    const bool wave_active = !p.causal || wave_i_max >= j0;
    if (wave_active) {
      float t[4][8];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 8; ++e) t[kb][e] = Srow[(kb * 16 + 8 * hh + e) * kSP];
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int j = j0 + kb * 16 + 8 * hh + e;
          const bool ok = row_ok && j < n && (!p.causal || j <= my_i);
          t[kb][e] = ok ? t[kb][e] * p.scale_log2 : -INFINITY;
          mt = fmaxf(mt, t[kb][e]);
        }
      mt = fmaxf(mt, swap_halves(mt));
      const float m_new = fmaxf(m_run, mt);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = exp2f(m_run - m_use);
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          t[kb][e] = exp2f(t[kb][e] - m_use);
          rs += t[kb][e];
        }
      rs += swap_halves(rs);
      l_run = l_run * alpha + rs;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;

      if constexpr (VBF16) {
        const uint16_t* Vt = (const uint16_t*)(smem + L.v_off);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          // P as two bfloat16 pieces, hi = bf16(p) and lo = bf16(p - hi): the
          // pair carries p to ~2^-17 relative (a single bf16 P would carry
          // 2^-8, which can exceed the output tolerance by itself)
          bf16x8 ph, pl;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            ph[e] = (__bf16)t[kb][e];
            pl[e] = (__bf16)(t[kb][e] - (float)ph[e]);
          }
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const bf16x8 va = *(const bf16x8*)(Vt + (db * 32 + (lane & 31)) * kVP + kb * 16 + 8 * hh);
            acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, ph, acc[db], 0, 0, 0);
            acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pl, acc[db], 0, 0, 0);
          }
        }
      } else {
        const float* Vs = (const float*)(smem + L.v_off);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int jj = kb * 16 + 8 * hh + e;
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
              const float va = Vs[jj * D + db * 32 + (lane & 31)];
              acc[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(va, t[kb][e], acc[db], 0, 0, 0);
            }
          }
      }
    }
    // clear this wave's rows of the score tile for the next key tile
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 8; ++e) Srow[(kb * 16 + 8 * hh + e) * kSP] = 0.f;
    __syncthreads();  // V tile and score tile are reused by the next key tile
  }

  // ---------------- epilogue: O = acc / l, LSE = ln(l) + m ln 2 -------------
  if (row_ok) {
    const float inv = 1.f / l_run;
    const int64_t orow = ((int64_t)b * p.Hq + my_hq) * n + my_i;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dim = db * 32 + 8 * g + 4 * hh;
        const float o0 = acc[db][4 * g + 0] * inv, o1 = acc[db][4 * g + 1] * inv;
        const float o2 = acc[db][4 * g + 2] * inv, o3 = acc[db][4 * g + 3] * inv;
        if (p.obf16) {
          uint2 w;
          w.x = f32_to_bf16_rne(o0) | (f32_to_bf16_rne(o1) << 16);
          w.y = f32_to_bf16_rne(o2) | (f32_to_bf16_rne(o3) << 16);
          *(uint2*)((uint16_t*)p.o + orow * D + dim) = w;
        } else {
          *(float4*)((float*)p.o + orow * D + dim) = make_float4(o0, o1, o2, o3);
        }
      }
    if (p.lse && hh == 0) p.lse[orow] = (m_run + __log2f(l_run)) * kLn2;
  }
}

template <int D, bool VBF16, int KM>
static hipError_t launch_fwd_km(const FwdParams& p, int B, hipStream_t stream) {
  const FwdLds L = fwd_lds_layout<D, VBF16>(p.k);
  // the largest dynamic LDS size set so far, per instantiation (it grows with k)
  static std::mutex mu;
  static int configured_bytes = 0;
  if (L.total > 65536) {
    std::lock_guard<std::mutex> lock(mu);
    if (L.total > configured_bytes) {
      hipError_t e = hipFuncSetAttribute((const void*)sfa_fwd_index_kernel<D, VBF16, KM>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, L.total);
      if (e != hipSuccess) return e;
      configured_bytes = L.total;
    }
  }
  dim3 grid(p.nqb, B * p.Hkv), block(kThreads);
  hipLaunchKernelGGL((sfa_fwd_index_kernel<D, VBF16, KM>), grid, block, L.total, stream, p);
  return hipGetLastError();
}

template <int D, bool VBF16>
static hipError_t launch_fwd_t(const FwdParams& p, int B, hipStream_t stream) {
  return p.k <= 16 ? launch_fwd_km<D, VBF16, 16>(p, B, stream)
                   : launch_fwd_km<D, VBF16, 64>(p, B, stream);
}

}  // namespace

int fwd_index_lds_bytes(int d, int k, int vbf16) {
  if (d == 64) return vbf16 ? fwd_lds_layout<64, true>(k).total : fwd_lds_layout<64, false>(k).total;
  return vbf16 ? fwd_lds_layout<128, true>(k).total : fwd_lds_layout<128, false>(k).total;
}

int fwd_index_max_k() { return kMaxK; }

hipError_t launch_attn_fwd_index(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, int B, int Hq, int Hkv, int n,
                           int d, int k, int causal, float scale, int ifmt, int vfmt,
                           int vbf16, int obf16, void* o, float* lse, hipStream_t stream) {
  FwdParams p;
  p.q_idx = q_idx; p.q_val = q_val; p.k_idx = k_idx; p.k_val = k_val; p.v = v;
  p.o = o; p.lse = lse;
  p.Hq = Hq; p.Hkv = Hkv; p.n = n; p.k = k; p.causal = causal;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);
  p.ifmt = ifmt; p.vfmt = vfmt; p.obf16 = obf16;
  p.G = Hq / Hkv;
  p.BR = kRows / p.G;
  p.nqb = (n + p.BR - 1) / p.BR;
  p.inv_k = 1.0f / (float)k;
  if (d == 64) return vbf16 ? launch_fwd_t<64, true>(p, B, stream) : launch_fwd_t<64, false>(p, B, stream);
  return vbf16 ? launch_fwd_t<128, true>(p, B, stream) : launch_fwd_t<128, false>(p, B, stream);
}

int fwd_index_rows_per_block() { return kRows; }

}  // namespace sfa
