// SFA forward (Sec. 3.1-3.2) on gfx950: overlap scores on the matrix cores.
//
// The overlap score s_ij = scale * sum_{u in S_i cap S_j} q_iu k_ju is the
// product of the densified codes (Sec. 3.1: S = Q~ K~^T): coordinates outside
// either support contribute exact zeros.  On a wave64 machine at k/d = 1/8 the
// data-dependent scatter of the overlap formulation is bound by LDS
// read-modify-write traffic (LDS float atomics run far below a lane per
// clock), while the matrix cores take the densified product at 2.5 PFLOP/s;
// so the codes are densified tile by tile into LDS and contracted there.
//
// Precision: each code value x is split into bfloat16 pieces x = x0 + x1 (+ x2),
// x0 = bf16(x), x1 = bf16(x - x0), x2 = bf16(x - x0 - x1).  Products of
// bf16 pieces are exact in float32 and accumulate in float32.  With bf16 V the
// score keeps the terms q0k0 + q0k1 + q1k0 (relative error ~2^-16 of
// sum|q_u k_u|); with float32 V it keeps every term of order <= 2
// (q0k0 + q0k1 + q1k0 + q0k2 + q1k1 + q2k0, ~2^-24).
//
// Workgroup = NW wavefronts = 32*NW query rows: the G query heads of one KV
// head times BR = 32*NW/G positions, so all G heads share each key tile.
// Per tile of 64 keys:
//   [A] scatter the tile's key codes (bf16 pieces) into a zeroed dense LDS
//       tile Kd[piece][key][coordinate]; stage V, transposed, into LDS;
//   [B] per wavefront, two 32-key sub-tiles: S^T = K~ Q~^T on
//       v_mfma_f32_32x32x16_bf16 (the query pieces live in registers for the
//       whole kernel), leaving each lane with one query row and 16 keys;
//       scale, causal mask and the online-softmax update (base 2) run on those
//       registers; the bf16 probabilities are already in the B-operand layout
//       of O^T += V^T P^T, the second MFMA;
//   [C] clear the scattered entries.
// Keys whose support does not overlap a query keep score 0 and still enter
// the softmax: the result is exactly softmax(Q~ K~^T * scale) V.
#include "sfa_device.h"
#include "sfa_launch.h"

namespace sfa {
namespace {

constexpr int kBC = 64;  // keys per tile

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
  int idx16, valbf16, obf16;
  int G, BR, nqb;
  float inv_k;
};

template <int D>
struct Geo {
  static constexpr int KP = D + 8;    // bf16 pitch of a densified row
  static constexpr int VP = kBC + 8;  // bf16 pitch of a transposed V row
  static constexpr int NKB = D / 16;  // 16-coordinate blocks of the score MFMA
  static constexpr int NDB = D / 32;  // 32-wide output blocks
};

template <int D, bool VBF16, int NW>
__host__ __device__ constexpr int lds_bytes() {
  constexpr int NP = VBF16 ? 2 : 3;
  constexpr int kd = NP * kBC * Geo<D>::KP * 2;
  constexpr int vt = VBF16 ? D * Geo<D>::VP * 2 : kBC * D * 4;
  constexpr int qs = NW * 32 * Geo<D>::KP * 2;
  return (kd + vt) > qs ? (kd + vt) : qs;
}

// bf16 piece `pc` of x (0: nearest bf16; 1, 2: bf16 of the remaining error).
__device__ __forceinline__ uint16_t bf16_piece(float x, int pc) {
  uint32_t h = f32_to_bf16_rne(x);
  if (pc == 0) return (uint16_t)h;
  const float r1 = x - bf16_bits_to_f32(h);
  const uint32_t m = f32_to_bf16_rne(r1);
  if (pc == 1) return (uint16_t)m;
  return (uint16_t)f32_to_bf16_rne(r1 - bf16_bits_to_f32(m));
}

template <int D, bool VBF16, int NW, int KM>
__global__ __launch_bounds__(NW * 64) void sfa_fwd_kernel(FwdParams p) {
  constexpr int NT = NW * 64;
  constexpr int R = NW * 32;
  constexpr int NP = VBF16 ? 2 : 3;
  constexpr int KP = Geo<D>::KP, VP = Geo<D>::VP, NKB = Geo<D>::NKB, NDB = Geo<D>::NDB;
  constexpr int KE = (kBC * KM + NT - 1) / NT;  // key-code entries per thread and tile
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* Kd = (uint16_t*)smem;                    // [NP][kBC][KP]
  unsigned char* vt = smem + NP * kBC * KP * 2;      // V tile
  uint16_t* Qs = (uint16_t*)smem;                    // setup only: [R][KP]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int hh = lane >> 5;
  const int l32 = lane & 31;
  const int k = p.k;
  const int n = p.n;
  const int dmask = D - 1;

  const int qb = p.nqb - 1 - (int)blockIdx.x;  // longest causal blocks first
  const int bh = blockIdx.y;
  const int b = bh / p.Hkv;
  const int hkv = bh - b * p.Hkv;
  const int i0 = qb * p.BR;

  // row of this lane: query head hkv*G + rho / BR at position i0 + rho % BR
  const int rho = wave * 32 + l32;
  const int my_i = i0 + rho % p.BR;
  const int my_hq = hkv * p.G + rho / p.BR;
  const bool row_ok = my_i < n;

  // ---------------- query operand: NP bf16 pieces of the densified rows ----
  bf16x8 qB[NP][NKB];
#pragma unroll
  for (int pc = 0; pc < NP; ++pc) {
    for (int x = tid; x < R * KP / 8; x += NT) ((uint4*)Qs)[x] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    for (int e = tid; e < R * k; e += NT) {
      const int r = (int)(((float)e + 0.5f) * p.inv_k);
      const int t = e - r * k;
      const int i = i0 + r % p.BR;
      if (i < n) {
        const int hq = hkv * p.G + r / p.BR;
        const int64_t gi = (((int64_t)b * p.Hq + hq) * n + i) * k + t;
        const int f = load_idx(p.q_idx, gi, p.idx16, dmask);
        Qs[r * KP + f] = bf16_piece(load_val(p.q_val, gi, p.valbf16), pc);
      }
    }
    __syncthreads();
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) qB[pc][kb] = *(const bf16x8*)(Qs + rho * KP + kb * 16 + 8 * hh);
    __syncthreads();
  }
  // the dense key tile starts (and is kept) all-zero between tiles
  for (int x = tid; x < NP * kBC * KP / 8; x += NT) ((uint4*)Kd)[x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();

  float m_run = -INFINITY, l_run = 0.f;
  floatx16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  const int wave_i_max = i0 + (wave * 32 + 31) % p.BR;  // largest position in this wave
  const int blk_last = min(n, i0 + p.BR) - 1;
  const int n_keys = p.causal ? blk_last + 1 : n;
  const int ntiles = (n_keys + kBC - 1) / kBC;
  const int64_t kv_base = ((int64_t)b * p.Hkv + hkv) * n;
  const int nke = kBC * k;

  uint32_t ent[KE];  // (key << 8) | coordinate of this thread's scattered entries
  for (int jt = 0; jt < ntiles; ++jt) {
    const int j0 = jt * kBC;

    // ---- [A] key codes -> dense bf16 pieces; V tile -> LDS ----
#pragma unroll
    for (int r = 0; r < KE; ++r) {
      const int e = tid + r * NT;
      ent[r] = 0xffffffffu;
      if (e < nke) {
        const int c = (int)(((float)e + 0.5f) * p.inv_k);
        const int t = e - c * k;
        const int j = j0 + c;
        if (j < n) {
          const int64_t gi = (kv_base + j) * k + t;
          const int f = load_idx(p.k_idx, gi, p.idx16, dmask);
          const float x = load_val(p.k_val, gi, p.valbf16);
          ent[r] = ((uint32_t)c << 8) | (uint32_t)f;
#pragma unroll
          for (int pc = 0; pc < NP; ++pc) Kd[(pc * kBC + c) * KP + f] = bf16_piece(x, pc);
        }
      }
    }
    if constexpr (VBF16) {
      uint16_t* Vt = (uint16_t*)vt;
      const uint16_t* Vg = (const uint16_t*)p.v;
      constexpr int NDP = D / 2;
      constexpr int ITEMS = NDP * (kBC / 8);
      for (int it = tid; it < ITEMS; it += NT) {
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
        *(uint4*)(Vt + (2 * dp) * VP + kg * 8) = lo;
        *(uint4*)(Vt + (2 * dp + 1) * VP + kg * 8) = hi;
      }
    } else {
      float* Vs = (float*)vt;
      const float* Vg = (const float*)p.v;
      constexpr int N4 = kBC * D / 4;
      for (int it = tid; it < N4; it += NT) {
        const int j = it / (D / 4);
        const int c4 = it % (D / 4);
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (j0 + j < n) val = *(const float4*)(Vg + (kv_base + j0 + j) * D + 4 * c4);
        *(float4*)(Vs + j * D + 4 * c4) = val;
      }
    }
    __syncthreads();

    // ---- [B] scores on MFMA, online softmax, P.V on MFMA ----
    const bool act0 = !p.causal || wave_i_max >= j0;
    const bool act1 = !p.causal || wave_i_max >= j0 + 32;
    if (act0) {
      floatx16 sc[2];
#pragma unroll
      for (int s = 0; s < 2; ++s) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[s][r] = 0.f;
        if (s == 0 || act1) {
#pragma unroll
          for (int kb = 0; kb < NKB; ++kb) {
            bf16x8 ka[NP];
#pragma unroll
            for (int pc = 0; pc < NP; ++pc)
              ka[pc] = *(const bf16x8*)(Kd + (pc * kBC + s * 32 + l32) * KP + kb * 16 + 8 * hh);
            // smaller terms first
            if constexpr (NP == 3) {
              sc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[2], qB[0][kb], sc[s], 0, 0, 0);
              sc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1], qB[1][kb], sc[s], 0, 0, 0);
              sc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[2][kb], sc[s], 0, 0, 0);
            }
            sc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1], qB[0][kb], sc[s], 0, 0, 0);
            sc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[1][kb], sc[s], 0, 0, 0);
            sc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[0][kb], sc[s], 0, 0, 0);
          }
        }
      }
      // lane: query row rho; register r of sub-tile s holds key
      // j0 + 32 s + 8 (r / 4) + 4 hh + (r % 4)
      float mt = -INFINITY;
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = j0 + 32 * s + 8 * (r >> 2) + 4 * hh + (r & 3);
          const bool ok = row_ok && j < n && (!p.causal || j <= my_i);
          sc[s][r] = ok ? sc[s][r] * p.scale_log2 : -INFINITY;
          mt = fmaxf(mt, sc[s][r]);
        }
      mt = fmaxf(mt, swap_halves(mt));
      const float m_new = fmaxf(m_run, mt);
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      const float alpha = exp2f(m_run - m_use);
      float rs = 0.f;
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sc[s][r] = exp2f(sc[s][r] - m_use);
          rs += sc[s][r];
        }
      rs += swap_halves(rs);
      l_run = l_run * alpha + rs;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;

      if constexpr (VBF16) {
        const uint16_t* Vt = (const uint16_t*)vt;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          if (s == 1 && !act1) break;
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            bf16x8 pb;
#pragma unroll
            for (int e = 0; e < 8; ++e) pb[e] = (__bf16)sc[s][8 * kk + e];
            const int kbase = 32 * s + 16 * kk + 4 * hh;  // keys kbase+0..3, kbase+8..11
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
              const uint16_t* row = Vt + (db * 32 + l32) * VP + kbase;
              const uint2 v0 = *(const uint2*)row;
              const uint2 v1 = *(const uint2*)(row + 8);
              const u32x4 vw = {v0.x, v0.y, v1.x, v1.y};
              const bf16x8 va = __builtin_bit_cast(bf16x8, vw);
              acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, acc[db], 0, 0, 0);
            }
          }
        }
      } else {
        const float* Vs = (const float*)vt;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          if (s == 1 && !act1) break;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int jj = 32 * s + 8 * (r >> 2) + 4 * hh + (r & 3);
#pragma unroll
            for (int db = 0; db < NDB; ++db)
              acc[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(Vs[jj * D + db * 32 + l32], sc[s][r],
                                                             acc[db], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();

    // ---- [C] clear the scattered key entries ----
#pragma unroll
    for (int r = 0; r < KE; ++r) {
      if (ent[r] != 0xffffffffu) {
        const int c = (int)(ent[r] >> 8), f = (int)(ent[r] & 0xffu);
#pragma unroll
        for (int pc = 0; pc < NP; ++pc) Kd[(pc * kBC + c) * KP + f] = 0;
      }
    }
    __syncthreads();
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

template <int D, bool VBF16, int NW, int KM>
hipError_t launch_km(const FwdParams& p, int B, hipStream_t stream) {
  constexpr int bytes = lds_bytes<D, VBF16, NW>();
  static bool configured = false;  // per instantiation
  if (bytes > 65536 && !configured) {
    hipError_t e = hipFuncSetAttribute((const void*)sfa_fwd_kernel<D, VBF16, NW, KM>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    configured = true;
  }
  dim3 grid(p.nqb, B * p.Hkv), block(NW * 64);
  hipLaunchKernelGGL((sfa_fwd_kernel<D, VBF16, NW, KM>), grid, block, bytes, stream, p);
  return hipGetLastError();
}

template <int D, bool VBF16, int NW>
hipError_t launch_nw(FwdParams p, int B, hipStream_t stream) {
  p.BR = NW * 32 / p.G;
  p.nqb = (p.n + p.BR - 1) / p.BR;
  return p.k <= 16 ? launch_km<D, VBF16, NW, 16>(p, B, stream)
                   : launch_km<D, VBF16, NW, 128>(p, B, stream);
}

template <int D, bool VBF16>
hipError_t launch_t(const FwdParams& p, int B, hipStream_t stream) {
  // 8 wavefronts (256 rows) per workgroup when that still gives >= 4
  // workgroups per compute unit; else 4 wavefronts.
  const long long wg8 = (long long)((p.n + 256 / p.G - 1) / (256 / p.G)) * B * p.Hkv;
  if (p.G <= 8 && wg8 >= 4LL * 256) return launch_nw<D, VBF16, 8>(p, B, stream);
  return launch_nw<D, VBF16, 4>(p, B, stream);
}

}  // namespace

int fwd_max_group() { return 128; }

hipError_t launch_attn_fwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, int B, int Hq, int Hkv, int n, int d,
                           int k, int causal, float scale, int idx16, int valbf16, int vbf16,
                           int obf16, void* o, float* lse, hipStream_t stream) {
  FwdParams p;
  p.q_idx = q_idx; p.q_val = q_val; p.k_idx = k_idx; p.k_val = k_val; p.v = v;
  p.o = o; p.lse = lse;
  p.Hq = Hq; p.Hkv = Hkv; p.n = n; p.k = k; p.causal = causal;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);
  p.idx16 = idx16; p.valbf16 = valbf16; p.obf16 = obf16;
  p.G = Hq / Hkv;
  p.BR = 0; p.nqb = 0;
  p.inv_k = 1.0f / (float)k;
  if (d == 64) return vbf16 ? launch_t<64, true>(p, B, stream) : launch_t<64, false>(p, B, stream);
  return vbf16 ? launch_t<128, true>(p, B, stream) : launch_t<128, false>(p, B, stream);
}

}  // namespace sfa
