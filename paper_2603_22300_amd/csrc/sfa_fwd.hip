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
// Precision: each code value x (for queries: x = q * scale * log2(e), so the
// scores come out as base-2 exponents) is split into 16-bit pieces whose
// products are exact in float32 and accumulate in float32.
// With bf16 V: two float16 pieces, x0 = f16(x), x1 = f16(x - x0) (round to
// nearest even; the float16 matrix cores keep subnormal operands), and the
// score keeps q0k0 + q0k1 + q1k0: the dropped q1k1 and the rounding of x1
// leave ~3 * 2^-22 of sum|q_u k_u| (plus at most 2^-25 absolute per value
// below the float16 normal range).  A value of magnitude >= 65504 does not
// fit float16: its workgroups are handed to the rerun kernel (below).  With
// float32 V, and in the rerun: three bfloat16 pieces x0 = bf16(x),
// x1 = bf16(x - x0), x2 = bf16(x - x0 - x1), and every term of order <= 2
// (q0k0 + q0k1 + q1k0 + q0k2 + q1k1 + q2k0, ~2^-24).
// 16-bit codes (bf16 or float16 values) with bf16 V: the raw
// values are already MFMA operands, so each 16-coordinate block of the score
// is one exact product on the matrix cores (bf16 or float16 MFMA), and the
// float32 score is multiplied by |scale| * log2(e) before exp2 (the sign of
// scale flips the query values' sign bits).  Per 64-key tile a wavefront then
// issues 16 score MFMAs instead of 48.
// P.V with bf16 V: V is converted to float16 (exact for normal values up to
// 65504) and P enters as float16 (P < 2^15, relative rounding 2^-11), one
// MFMA per block.  A workgroup whose keys hold a V value outside the float16
// range (or a code value too large for the float16 pieces) hands its rows to
// a rerun kernel that reads V as bf16, splits P into Ph + Pl in bf16 and the
// code values into three bf16 pieces (six products, ~2^-24).  With float32
// V, P.V runs on the float32 MFMA.
//
// Workgroup = NW wavefronts = 32*NW query rows: the G query heads of one KV
// head times BR = 32*NW/G positions, so all G heads share each key tile.
// Per tile of 64 keys:
//   [A] the tile's LDS image: the dense key tile Kd[key][piece][coordinate]
//       (bf16 pieces of the codes, zeros elsewhere) and V^T beside it.  With
//       bf16 V the image is prepared once per call by sfa_fwd_prep_kernel and
//       copied global -> LDS by direct-to-LDS loads; otherwise (float32 V,
//       the rerun) each wave zeroes and fills its 64/NW key rows itself;
//   [B] per wavefront, two 32-key sub-tiles: S^T = K~ Q~^T on
//       v_mfma_f32_32x32x16_bf16 (the query pieces live in registers for the
//       whole kernel), leaving each lane with one query row and 16 keys; the
//       causal mask and the online-softmax update (base 2) run on those
//       registers; the probabilities are already in the B-operand layout of
//       O^T += V^T P^T, the second MFMA.
// The next tile's image is in flight during the current one, into the other
// LDS stage, with one barrier per tile.
// Keys whose support does not overlap a query keep score 0 and still enter
// the softmax: the result is exactly softmax(Q~ K~^T * scale) V.
#include <algorithm>

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
  int window, n_global;  // token pattern: |i - j| < window or a global token (window 0: none)
  float scale_log2;  // scale * log2(e)
  // 16-bit codes: |scale| * log2(e), and the sign of scale as a 16-bit sign bit
  float kx_scale;
  uint32_t qsign;
  int kx;  // 0, or the 16-bit code value type taking the one-product path
  // Inverted-index score mode (k <= kIxMaxK, bf16 V): its tile images, and
  // the data-dependent choice between it and the dense product.  The index
  // pre-pass adds every tile's longest bucket into *ix_stat; the index mode
  // runs if the sum is <= ix_thresh, else the dense mode (each launch of the
  // other mode returns at once).  ix == 0: dense mode only.
  int ix;
  const unsigned char* ix_tiles;
  const uint32_t* ix_stat;
  uint32_t ix_thresh;
  int ifmt, vfmt, obf16;
  int G, BR, nqb;
  float inv_k;
  // bf16 V, prepared once per call (sfa_fwd_prep_kernel): every key tile as
  // its LDS stage image (dense bf16 key pieces, float16 V^T) and a V range
  // flag per tile
  const unsigned char* ws_tiles;
  const int* ws_flag;
  // set to nonzero by every workgroup that hands its rows back (zeroed by
  // the pre-pass), so that the rerun launch returns at once when none did
  int* hb_count;
  int vtiles;  // tiles per (batch, KV head): ceil(n / 64)
};

template <int D, int NP>
struct Geo {
  static constexpr int QP = D + 8;           // bf16 pitch of a densified query row (setup)
  static constexpr int KR = NP * D + 8;      // bf16 pitch of a key row: [piece][coordinate] + pad
  static constexpr int VP = kBC + 4;         // bf16 pitch of a transposed V row
  static constexpr int NKB = D / 16;         // 16-coordinate blocks of the score MFMA
  static constexpr int NDB = D / 32;         // 32-wide output blocks
};
// Pitches: a key row of KR bf16 is 4 dwords past a multiple of 32 banks, so
// the 16-byte A-operand reads of consecutive keys hit disjoint banks; a V row
// of 68 bf16 is 2 dwords past, for the 8-byte operand reads.

// The 16-bit V tile in LDS: [dimension][key], pitch VP, padded to whole
// 1 KB blocks so that it is copied by whole-wave 16-byte direct-to-LDS loads.
template <int D>
__host__ __device__ constexpr int vtile_bytes() {
  return (D * (kBC + 4) * 2 + 1023) / 1024 * 1024;
}

// 16-bit pieces per key value: two float16 pieces of a float32 value (bf16
// V), three bfloat16 pieces (float32 V, and the bf16-V rerun); one raw value
// for 16-bit codes (KX = kValBF16 / kValF16).
template <bool VBF16, int KX, bool SAFE = false>
__host__ __device__ constexpr int n_pieces() {
  return KX ? 1 : (VBF16 && !SAFE ? 2 : 3);
}

template <int D, bool VBF16, int KX = 0, bool SAFE = false>
__host__ __device__ constexpr int stage_bytes() {
  constexpr int NP = n_pieces<VBF16, KX, SAFE>();
  return kBC * Geo<D, NP>::KR * 2 + (VBF16 ? vtile_bytes<D>() : kBC * D * 4);
}

// Two LDS stages (next tile written while the current one is read) when they
// fit; the float32-V path (three pieces, float32 V tile) uses one.
template <int D, bool VBF16, int KX = 0, bool SAFE = false>
__host__ __device__ constexpr int n_stages() {
  return 2 * stage_bytes<D, VBF16, KX, SAFE>() <= 160 * 1024 ? 2 : 1;
}

// The densified query rows of the prologue sit past stage 0 with bf16 V, so
// that the first tile's copy into stage 0 overlaps the prologue.
template <int D, bool VBF16, int KX = 0, bool SAFE = false>
__host__ __device__ constexpr int qs_offset() {
  return VBF16 ? stage_bytes<D, VBF16, KX, SAFE>() : 0;
}

template <int D, bool VBF16, int NW, int KX = 0, bool SAFE = false>
__host__ __device__ constexpr int lds_bytes() {
  constexpr int st = n_stages<D, VBF16, KX, SAFE>() * stage_bytes<D, VBF16, KX, SAFE>();
  constexpr int qs = qs_offset<D, VBF16, KX, SAFE>() + NW * 32 * Geo<D, 2>::QP * 2;
  return st > qs ? st : qs;
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

// float16 piece `pc` of x (0: nearest float16; 1: float16 of x - x0, which is
// exact in float32).  Finite only for |x| < 65520; callers hand larger values
// to the bf16-piece rerun.
__device__ __forceinline__ uint16_t f16_piece(float x, int pc) {
  const _Float16 h = (_Float16)x;
  if (pc == 0) return __builtin_bit_cast(uint16_t, h);
  return __builtin_bit_cast(uint16_t, (_Float16)(x - (float)h));
}
// Code values (query values with scale * log2(e) folded in) from this
// magnitude on take the bf16-piece rerun: float16 pieces would overflow.
constexpr float kF16PieceMax = 65504.f;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// two float32 (given as bits) -> packed float16, round to nearest even
__device__ __forceinline__ uint32_t f16_pair(uint32_t a, uint32_t b) {
  const f16x2 h = {(_Float16)__uint_as_float(a), (_Float16)__uint_as_float(b)};
  return __builtin_bit_cast(uint32_t, h);
}

// The running row maximum is raised only when a tile's maximum exceeds it by
// more than this (log2 units), so the accumulators are rescaled rarely; O and
// LSE use the same stale maximum.
constexpr float kLazyMax = 8.f;
// An interior tile whose exponents are bounded (Cauchy-Schwarz on the code
// norms) by m_run + kBoundMax skips the maxima: its probabilities stay below
// 2^15, inside the float16 range of the P.V operand.
constexpr float kBoundMax = 15.f;

// Bits written into the first output element of a workgroup's rows when the
// float16 path meets a V tile outside the float16 range: a NaN payload that
// the arithmetic does not produce (it yields the default NaN).  Should a
// computed NaN carry it anyway, the rerun only recomputes the same result.
constexpr uint16_t kHandBack16 = 0x7fa5u;
constexpr uint32_t kHandBack32 = 0x7fa5a5a5u;

// One workgroup: query block qb of (batch, KV head) bh.
// SAFE (bf16 V only): V is staged as bf16 and P.V uses P = Ph + Pl on the
// bf16 MFMA, every tile on the generic path; the code values are split into
// three bf16 pieces (every product of order <= 2 kept, any finite magnitude);
// it reruns the workgroups that the float16 path handed back.
// KX (bf16 V, 16-bit codes): kValBF16 or kValF16, the code values' type.  The
// raw query and key values are the MFMA operands (bf16 or float16), so each
// score is one exact product sum; the scale is applied to the float32 scores.
template <int D, bool VBF16, int NW, int KM, bool SAFE, int KX = 0>
__device__ __forceinline__ void fwd_block(const FwdParams& p, const int qb, const int bh) {
  static_assert(VBF16 || !SAFE, "the rerun is for bf16 V");
  static_assert(KX == 0 || (VBF16 && !SAFE), "16-bit codes: bf16 V");
  constexpr int NT = NW * 64;
  constexpr int R = NW * 32;
  constexpr int NP = n_pieces<VBF16, KX, SAFE>();
  // two float16 pieces (bf16 V, 32-bit codes, not the rerun): the three
  // score products run on the float16 matrix cores
  constexpr bool F16P = NP == 2 && KX == 0 && !SAFE;
  using Gm = Geo<D, NP>;
  constexpr int QP = Gm::QP, KR = Gm::KR, VP = Gm::VP, NKB = Gm::NKB, NDB = Gm::NDB;
  constexpr int NS = n_stages<D, VBF16, KX, SAFE>();
  constexpr int SB = stage_bytes<D, VBF16, KX, SAFE>();
  constexpr int KW = kBC / NW;                 // key rows owned (zeroed, filled) by a wave
  constexpr int KEL = (KW * KM + 63) / 64;     // key-code entries per lane and tile
  constexpr int NDP = D / 2;
  constexpr int VITEMS = VBF16 ? NDP * (kBC / 8) : kBC * D / 4;
  constexpr int VI = (VITEMS + NT - 1) / NT;   // V items per thread and tile
  constexpr int VW = VBF16 ? 8 : 4;            // registers per V item
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  uint16_t* Qs = (uint16_t*)(smem + qs_offset<D, VBF16, KX, SAFE>());  // setup only: [R][QP]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;
  const int l32 = lane & 31;
  const int k = p.k;
  const int n = p.n;
  const int dmask = D - 1;

  const int b = bh / p.Hkv;
  const int hkv = bh - b * p.Hkv;
  const int i0 = qb * p.BR;

  // row of this lane: query head hkv*G + rho / BR at position i0 + rho % BR
  const int rho = wave * 32 + l32;
  const int my_i = i0 + rho % p.BR;
  const int my_hq = hkv * p.G + rho / p.BR;
  const bool row_ok = my_i < n;

  const int blk_last = min(n, i0 + p.BR) - 1;
  // Key tiles this workgroup visits: all up to the causal limit, or with a
  // token window (and no global row here) the global tiles [0, gt_end) and
  // the window tiles [wt_begin, ntiles_all) -- tiles in the gap are skipped.
  const bool win = p.window > 0;
  int n_keys = p.causal ? blk_last + 1 : n;
  int gt_end = 0, wt_begin = 0;
  if (win && i0 >= p.n_global) {
    if (!p.causal) n_keys = min(n, blk_last + p.window);
    gt_end = (p.n_global + kBC - 1) / kBC;
    wt_begin = max(0, i0 - p.window + 1) / kBC;
    if (wt_begin <= gt_end) gt_end = wt_begin = 0;  // no gap
  }
  const int ntiles_all = (n_keys + kBC - 1) / kBC;
  const int ntiles = gt_end + ntiles_all - wt_begin;
  // key tile of list position t (t == ntiles gives ntiles_all: past the end)
  auto tile_at = [&](int t) { return t < gt_end ? t : wt_begin + (t - gt_end); };

  // bf16 V: key tiles arrive as prepared stage images, copied global -> LDS
  // by the memory unit (16 bytes per lane, 1 KB per wave instruction);
  // completion is awaited with vmcnt before the barrier that publishes them.
  constexpr bool kDMA = VBF16 && !SAFE;
  auto dma_stage = [&](int stage, int jt) {
    static_assert(SB % 1024 == 0, "stage images are whole 1 KB blocks");
    constexpr int NB = SB / 1024, NJ = (NB + NW - 1) / NW;
    // wave-uniform base + 32-bit lane offset: the scalar-base address form
    const unsigned char* src = p.ws_tiles + ((int64_t)bh * p.vtiles + jt) * SB;
    unsigned char* dst = smem + stage * SB;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = wave + j * NW;  // 1 KB block of the image
      if (j + 1 < NJ || i < NB)
        __builtin_amdgcn_global_load_lds(src + (uint32_t)(i * 1024 + lane * 16),
                                         (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                         16, 0, 0);
    }
  };
  auto wait_dma = [&]() {
    if constexpr (kDMA) __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  };

  // V range flags of the workgroup's key tiles (thread tid: list positions
  // tid, tid + NT, ...): the first is loaded now, all are tested once the
  // query operand is built (a flagged workgroup writes nothing before that).
  int vflag = 0;
  if constexpr (kDMA) {
    if (tid < ntiles) vflag = p.ws_flag[(int64_t)bh * p.vtiles + tile_at(tid)];
  }

  // ---------------- query operand: NP bf16 pieces of the densified rows ----
  // The query values carry scale * log2(e): the score tiles come out as the
  // base-2 exponents t = s * scale * log2(e) of the softmax, sign included.
  // With 16-bit codes the operand is the raw value (sign of scale folded in)
  // and the scores are multiplied by cs = |scale| * log2(e) after the MFMA.
  // Code entry e of the block is term e % k of row r = e / k, the query head
  // hkv*G + r / BR at position i0 + r % BR (BR is a power of two).
  const int lbr = __builtin_ctz(p.BR);
  auto q_entry = [&](int e, int& at, float& x) {
    const int r = (int)(((float)e + 0.5f) * p.inv_k);
    const int i = i0 + (r & (p.BR - 1));
    at = -1;
    x = 0.f;
    if (e < R * k && i < n) {
      const int hq = hkv * p.G + (r >> lbr);
      const int64_t gi = (((int64_t)b * p.Hq + hq) * n + i) * k + (e - r * k);
      at = r * QP + load_idx(p.q_idx, gi, p.ifmt, dmask);
      if constexpr (KX != 0)  // the 16-bit pattern, carried in a float register
        x = __uint_as_float((uint32_t)((const uint16_t*)p.q_val)[gi] ^ p.qsign);
      else
        x = p.scale_log2 * load_val(p.q_val, gi, p.vfmt);
    }
  };
  // With k <= 16 every thread's entries fit in registers: they are loaded
  // once, ahead of the first tile's copy, and serve all pieces.
  constexpr int QE = KM <= 16 ? R * KM / NT : 1;
  int q_at[QE];
  float q_x[QE];
  if constexpr (KM <= 16) {
#pragma unroll
    for (int u = 0; u < QE; ++u) q_entry(tid + NT * u, q_at[u], q_x[u]);
  }
  if constexpr (kDMA && NS == 2) {
    if (ntiles > 0) dma_stage(0, tile_at(0));  // stage 0; Qs lies past it
  }

  // Pieces are scattered into the same coordinates, so the rows are zeroed
  // once and each piece overwrites the previous one.
  for (int x = tid; x < R * QP / 8; x += NT) ((uint4*)Qs)[x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  // a query value too large for float16 pieces hands the workgroup back
  bool qbig = false;
  auto q_piece = [&](float x, int pc) -> uint16_t {
    if constexpr (KX != 0) {
      return (uint16_t)__float_as_uint(x);
    } else if constexpr (F16P) {
      qbig |= fabsf(x) >= kF16PieceMax;
      return f16_piece(x, pc);
    } else {
      return bf16_piece(x, pc);
    }
  };
  bf16x8 qB[NP][NKB];  // 16-bit pieces (float16 bits when F16P)
#pragma unroll
  for (int pc = 0; pc < NP; ++pc) {
    if (pc > 0) __syncthreads();  // the previous piece is read
    if constexpr (KM <= 16) {
#pragma unroll
      for (int u = 0; u < QE; ++u)
        if (q_at[u] >= 0) Qs[q_at[u]] = q_piece(q_x[u], pc);
    } else {
      for (int e = tid; e < R * k; e += NT) {
        int at;
        float x;
        q_entry(e, at, x);
        if (at >= 0) Qs[at] = q_piece(x, pc);
      }
    }
    __syncthreads();
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) qB[pc][kb] = *(const bf16x8*)(Qs + rho * QP + kb * 16 + 8 * hh);
  }

  if constexpr (kDMA) {
    // A tile of this workgroup's key range flagged by the pre-pass (a V value
    // outside the float16 range, or a key value too large for the float16
    // pieces), or a query value too large for them: hand the rows back to the
    // bf16 rerun before doing any work.
    for (int t = tid + NT; t < ntiles; t += NT)
      vflag |= p.ws_flag[(int64_t)bh * p.vtiles + tile_at(t)];
    if (__syncthreads_or(vflag != 0 || qbig)) {
      wait_dma();  // the stage copy lands before the workgroup's LDS is released
      if (tid == 0) {
        const int64_t orow0 = ((int64_t)b * p.Hq + hkv * p.G) * n + i0;  // row rho = 0
        if (p.obf16) ((uint16_t*)p.o)[orow0 * D] = kHandBack16;
        else ((uint32_t*)p.o)[orow0 * D] = kHandBack32;
        *p.hb_count = 1;
      }
      return;
    }
  }

  // Cauchy-Schwarz bound on this row's exponents: |t_ij| <= qn * |k_j| (the
  // overlap sum runs over a subset of the coordinates), with a margin for the
  // bf16 pieces and float32 rounding.
  const float cs = KX ? p.kx_scale : 1.f;  // score units -> base-2 exponent units
  float qn = 0.f;
  if constexpr (KX != 0) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint16_t bits = __builtin_bit_cast(uint16_t, qB[0][kb][e]);
        const float x = KX == kValF16 ? f16_bits_to_f32(bits) : bf16_bits_to_f32(bits);
        qn = fmaf(x, x, qn);
      }
    qn = sqrtf(pair_sum(qn)) * cs * (1.f + 1.f / 256.f);
  } else if constexpr (NP == 2) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float x;
        if constexpr (F16P)
          x = (float)__builtin_bit_cast(f16x8, qB[0][kb])[e] +
              (float)__builtin_bit_cast(f16x8, qB[1][kb])[e];
        else
          x = (float)qB[0][kb][e] + (float)qB[1][kb][e];
        qn = fmaf(x, x, qn);
      }
    qn = sqrtf(pair_sum(qn)) * (1.f + 1.f / 256.f);
  }

  float m_run = -INFINITY, l_run = 0.f;
  // Interior tiles start their score accumulators at -m_run (the C operand of
  // the first MFMA), so they come out as t - m_run, the argument of exp2
  // (16-bit codes: at -m_run / cs, giving (t - m_run) / cs).
  constexpr bool kFast = NS == 2 && VBF16 && !SAFE;
  floatx16 negm, zero16;
#pragma unroll
  for (int r = 0; r < 16; ++r) zero16[r] = 0.f;
  auto set_m = [&](float m) {
    m_run = m;
    if constexpr (kFast) {
      const float c0 = KX ? -m / cs : -m;
#pragma unroll
      for (int r = 0; r < 16; ++r) negm[r] = c0;
    }
  };
  floatx16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  const int wave_i_max = i0 + (wave * 32 + 31) % p.BR;  // largest position in this wave
  const int wave_i_min = p.BR >= 32 ? i0 + (wave * 32) % p.BR : i0;
  const int64_t kv_base = ((int64_t)b * p.Hkv + hkv) * n;

  // ---- global -> registers for one tile ----
  // Per-lane offsets are loop-invariant; loads are unconditional (indices
  // clamped into the arrays on the last tile only) and the dtype branches are
  // uniform, so nothing waits on them until write_tile.
  int k_off[KEL], k_row[KEL];
#pragma unroll
  for (int r = 0; r < KEL; ++r) {
    int el = lane + 64 * r;
    const bool ok = el < KW * k;
    el = ok ? el : KW * k - 1;
    const int cl = (int)(((float)el + 0.5f) * p.inv_k);
    k_row[r] = ok ? wave * KW + cl : -1;
    k_off[r] = (wave * KW + cl) * k + (el - cl * k);
  }
  int kf[KEL];
  float kx[KEL];
  uint32_t vr[VI][VW];
  // Uniform per-(batch, KV head) bases; per-lane offsets fit 32 bits (n*d and
  // n*k are at most 2^29, checked on the host), so the loads take the form
  // scalar base + 32-bit vector offset.
  const unsigned isz = idx_bytes(p.ifmt), ksz = val_bytes(p.vfmt);
  const unsigned char* kidx_b = (const unsigned char*)p.k_idx + kv_base * k * isz;
  const unsigned char* kval_b = (const unsigned char*)p.k_val + kv_base * k * ksz;
  const unsigned char* v_b = (const unsigned char*)p.v + kv_base * D * (VBF16 ? 2 : 4);
  auto load_tile = [&](int jt) {
    if constexpr (kDMA) return;
    const int j0 = jt * kBC;
    const bool full = j0 + kBC <= n;
    uint32_t ge[KEL];  // code element within this KV head
#pragma unroll
    for (int r = 0; r < KEL; ++r) {
      if (full) {
        ge[r] = (uint32_t)(j0 * k + k_off[r]);
      } else {
        const int row = k_row[r] < 0 ? 0 : k_row[r];
        const int j = min(j0 + row, n - 1);
        ge[r] = (uint32_t)(j * k + (k_off[r] - row * k));
      }
    }
    if (p.ifmt == kIdxI16) {
#pragma unroll
      for (int r = 0; r < KEL; ++r) kf[r] = *(const int16_t*)(kidx_b + ge[r] * 2u);
    } else if (p.ifmt == kIdxU8) {
#pragma unroll
      for (int r = 0; r < KEL; ++r) kf[r] = *(const uint8_t*)(kidx_b + ge[r]);
    } else {
#pragma unroll
      for (int r = 0; r < KEL; ++r) kf[r] = *(const int32_t*)(kidx_b + ge[r] * 4u);
    }
    if (p.vfmt == kValBF16) {
#pragma unroll
      for (int r = 0; r < KEL; ++r) kx[r] = __uint_as_float((uint32_t)*(const uint16_t*)(kval_b + ge[r] * 2u) << 16);
    } else if (p.vfmt == kValF16) {
#pragma unroll
      for (int r = 0; r < KEL; ++r) kx[r] = f16_bits_to_f32(*(const uint16_t*)(kval_b + ge[r] * 2u));
    } else {
#pragma unroll
      for (int r = 0; r < KEL; ++r) kx[r] = *(const float*)(kval_b + ge[r] * 4u);
    }
#pragma unroll
    for (int r = 0; r < VI; ++r) {
      const int it = min(tid + r * NT, VITEMS - 1);
      if constexpr (VBF16) {
        const int dp = it % NDP, kg = it / NDP;
        if (full) {
          const uint32_t off = (uint32_t)((j0 + kg * 8) * D + 2 * dp) * 2u;
#pragma unroll
          for (int e = 0; e < 8; ++e) vr[r][e] = *(const uint32_t*)(v_b + off + e * D * 2);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int j = min(j0 + kg * 8 + e, n - 1);
            vr[r][e] = *(const uint32_t*)(v_b + (uint32_t)(j * D + 2 * dp) * 2u);
          }
        }
      } else {
        const int j = min(j0 + it / (D / 4), n - 1), c4 = it % (D / 4);
        const uint4 val = *(const uint4*)(v_b + (uint32_t)(j * D + 4 * c4) * 4u);
        vr[r][0] = val.x; vr[r][1] = val.y; vr[r][2] = val.z; vr[r][3] = val.w;
      }
    }
  };
  // ---- registers -> LDS stage: zero own key rows, scatter own codes, V ----
  // Stage layout: Kd[key][piece][coordinate] (pitch KR), then the V tile.
  auto write_tile_keys = [&](int stage, int jt) {
    if constexpr (kDMA) return;
    const int j0 = jt * kBC;
    uint16_t* Kd = (uint16_t*)(smem + stage * SB);
    // zero the coordinate part of this wave's KW key rows (straight-line)
    constexpr int RU4 = NP * D / 8;  // uint4 per row, padding excluded
    static_assert((KW * RU4) % 64 == 0, "row zeroing must be whole wave steps");
#pragma unroll
    for (int i = 0; i < KW * RU4 / 64; ++i) {
      const int x = lane + 64 * i;
      const int row = x / RU4, col = x - row * RU4;
      *(uint4*)(Kd + (wave * KW + row) * KR + col * 8) = make_uint4(0u, 0u, 0u, 0u);
    }
    // scatter this lane's codes; entries outside the sequence write into the
    // row padding (never read), so the code stays branch-free
#pragma unroll
    for (int r = 0; r < KEL; ++r) {
      const bool ok = k_row[r] >= 0 && j0 + k_row[r] < n;
      const int row = k_row[r] < 0 ? 0 : k_row[r];
      const int f = kf[r] & dmask;
#pragma unroll
      for (int pc = 0; pc < NP; ++pc)
        Kd[row * KR + (ok ? pc * D + f : NP * D + pc)] = bf16_piece(kx[r], pc);
    }
  };
  auto write_tile_v = [&](int stage, int jt) {
    const int j0 = jt * kBC;
    unsigned char* vt = smem + stage * SB + kBC * KR * 2;
#pragma unroll
    for (int r = 0; r < VI; ++r) {
      const int it = tid + r * NT;
      if (VITEMS % NT != 0 && it >= VITEMS) break;
      if constexpr (kDMA) {
        break;
      } else if constexpr (VBF16) {
        uint16_t* Vt = (uint16_t*)vt;
        const int dp = it % NDP, kg = it / NDP;
        uint32_t w[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) w[e] = (j0 + kg * 8 + e < n) ? vr[r][e] : 0u;
        uint2 lo0, lo1, hi0, hi1;
        lo0.x = (w[0] & 0xffffu) | (w[1] << 16); hi0.x = (w[0] >> 16) | (w[1] & 0xffff0000u);
        lo0.y = (w[2] & 0xffffu) | (w[3] << 16); hi0.y = (w[2] >> 16) | (w[3] & 0xffff0000u);
        lo1.x = (w[4] & 0xffffu) | (w[5] << 16); hi1.x = (w[4] >> 16) | (w[5] & 0xffff0000u);
        lo1.y = (w[6] & 0xffffu) | (w[7] << 16); hi1.y = (w[6] >> 16) | (w[7] & 0xffff0000u);
        uint16_t* r0 = Vt + (2 * dp) * VP + kg * 8;
        uint16_t* r1 = r0 + VP;
        *(uint2*)r0 = lo0; *(uint2*)(r0 + 4) = lo1;
        *(uint2*)r1 = hi0; *(uint2*)(r1 + 4) = hi1;
      } else {
        float* Vs = (float*)vt;
        const int j = it / (D / 4), c4 = it % (D / 4);
        const bool ok = j0 + j < n;
        *(uint4*)(Vs + j * D + 4 * c4) = ok ? make_uint4(vr[r][0], vr[r][1], vr[r][2], vr[r][3])
                                            : make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };

  auto write_tile = [&](int stage, int jt) {
    write_tile_keys(stage, jt);
    write_tile_v(stage, jt);
  };
  // the first tile in stage 0 (bf16 V: its copy was issued with the query loads)
  if (ntiles > 0 && NS == 2) {
    if constexpr (kDMA) {
      wait_dma();
    } else {
      load_tile(tile_at(0));
      write_tile(0, tile_at(0));
    }
  }
  __syncthreads();

  // ---- building blocks of a key tile -------------------------------------
  // S^T for keys 32 s .. 32 s + 31 of the tile, this wave's 32 rows: lane
  // (row rho) register r holds key 32 s + 8 (r / 4) + 4 hh + (r % 4).
  auto score_sub = [&](floatx16& o, int s, const uint16_t* Kd, const floatx16& init) {
    o = init;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      bf16x8 ka[NP];
#pragma unroll
      for (int pc = 0; pc < NP; ++pc)
        ka[pc] = *(const bf16x8*)(Kd + (s * 32 + l32) * KR + pc * D + kb * 16 + 8 * hh);
      if constexpr (KX == kValF16) {
        o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[0]),
                                                   __builtin_bit_cast(f16x8, qB[0][kb]), o, 0, 0, 0);
        continue;
      } else if constexpr (KX == kValBF16) {
        o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[0][kb], o, 0, 0, 0);
        continue;
      }
      if constexpr (F16P) {  // smaller terms first
        o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[1]),
                                                   __builtin_bit_cast(f16x8, qB[0][kb]), o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[0]),
                                                   __builtin_bit_cast(f16x8, qB[1][kb]), o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[0]),
                                                   __builtin_bit_cast(f16x8, qB[0][kb]), o, 0, 0, 0);
        continue;
      }
      // smaller terms first
      if constexpr (NP == 3) {
        o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[2], qB[0][kb], o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1], qB[1][kb], o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[2][kb], o, 0, 0, 0);
      }
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1], qB[0][kb], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[1][kb], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[0][kb], o, 0, 0, 0);
    }
  };
  // largest value of a sub-tile (no mask), combined over the two lanes of the row
  auto sub_max = [&](const floatx16& o) {
    float hi = o[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) hi = fmaxf(hi, o[r]);
    return pair_max(hi);
  };
  // P in float16 for the fp16 V tile (values < 2^kBoundMax, 11-bit mantissa)
  auto to_f16 = [&](const floatx16& pr, f16x8 (&pf)[2]) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kk][e] = (_Float16)pr[8 * kk + e];
  };
  // V^T operand of the 16-key PV block kk of sub-tile s from the fp16 LDS tile
  // (keys kbase+0..3 and kbase+8..11 of this lane half)
  auto va_load = [&](f16x8 (&va)[NDB], int s, int kk, const uint16_t* Vt) {
    const int kbase = 32 * s + 16 * kk + 4 * hh;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const uint16_t* row = Vt + (db * 32 + l32) * VP + kbase;
      const uint2 v0 = *(const uint2*)row;
      const uint2 v1 = *(const uint2*)(row + 8);
      const u32x4 vw = {v0.x, v0.y, v1.x, v1.y};
      va[db] = __builtin_bit_cast(f16x8, vw);
    }
  };
  auto pv_terms = [&](const f16x8 (&va)[NDB], const f16x8& pf) {
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va[db], pf, acc[db], 0, 0, 0);
  };
  auto pv16_sub = [&](int s, const f16x8 (&pf)[2], const uint16_t* Vt) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      f16x8 va[NDB];
      va_load(va, s, kk, Vt);
      pv_terms(va, pf[kk]);
    }
  };
  // bf16 V tile (rerun): O^T += V^T P^T with P = Ph + Pl in bfloat16,
  // Pl = bf16(P - Ph), relative error ~2^-17 per weight.
  auto pv_sub_bf16 = [&](int s, const floatx16& pr, const uint16_t* Vt) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kbase = 32 * s + 16 * kk + 4 * hh;
      bf16x8 ph, pl;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ph[e] = (__bf16)pr[8 * kk + e];
        pl[e] = (__bf16)(pr[8 * kk + e] - (float)ph[e]);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint16_t* row = Vt + (db * 32 + l32) * VP + kbase;
        const uint2 v0 = *(const uint2*)row;
        const uint2 v1 = *(const uint2*)(row + 8);
        const u32x4 vw = {v0.x, v0.y, v1.x, v1.y};
        const bf16x8 va = __builtin_bit_cast(bf16x8, vw);
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pl, acc[db], 0, 0, 0);
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, ph, acc[db], 0, 0, 0);
      }
    }
  };
  auto rescale = [&](float alpha) {
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;
  };

  // ---- generic sub-tile: any mask, first tile, large jumps of the maximum --
  // One 32-key sub-tile s with its own online-softmax update (keeps a single
  // score tile live).
  auto generic_sub = [&](int j0, int s, const uint16_t* Kd, const unsigned char* vt) {
    floatx16 sc;
    score_sub(sc, s, Kd, zero16);
    // base-2 exponents t; masked keys get t = -inf
    float mt = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (KX != 0) sc[r] *= cs;
      const int j = j0 + 32 * s + 8 * (r >> 2) + 4 * hh + (r & 3);
      const bool ok = row_ok && j < n && (!p.causal || j <= my_i) &&
                      (!win || abs(my_i - j) < p.window || j < p.n_global || my_i < p.n_global);
      sc[r] = ok ? sc[r] : -INFINITY;
      mt = fmaxf(mt, sc[r]);
    }
    mt = pair_max(mt);
    const bool upd = mt > m_run + kLazyMax;
    const float m_new = upd ? mt : m_run;
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    if (__builtin_amdgcn_ballot_w64(upd)) {
      rescale(upd ? fast_exp2(m_run - m_use) : 1.f);
      set_m(m_new);
    }
    float rs = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) { sc[r] = fast_exp2(sc[r] - m_use); rs += sc[r]; }
    l_run += rs;
    if constexpr (VBF16) {
      const uint16_t* Vt = (const uint16_t*)vt;
      if constexpr (!SAFE) {
        f16x8 pf[2];
        to_f16(sc, pf);
        pv16_sub(s, pf, Vt);
      } else {
        pv_sub_bf16(s, sc, Vt);
      }
    } else {
      const float* Vs = (const float*)vt;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jj = 32 * s + 8 * (r >> 2) + 4 * hh + (r & 3);
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          acc[db] = __builtin_amdgcn_mfma_f32_32x32x2f32(Vs[jj * D + db * 32 + l32], sc[r],
                                                         acc[db], 0, 0, 0);
      }
    }
  };

  // ---- interior tile, software-pipelined by 32-key sub-tile ---------------
  // A: scores(0)  B: scores(1) || softmax(0)  C: P.V(0) || softmax(1)
  // D: P.V(1) || next tile's LDS writes.  Within B, C and D the source is
  // sliced by hand (one MFMA group plus its share of independent VALU work,
  // operands read one slice ahead), so that the matrix pipe and the VALU
  // work side by side.  The maximum stays
  // fixed unless a sub-tile exceeds it by 2^kLazyMax: after A that hands the
  // tile to generic_tile (returns false); after B it is fixed up in place.
  auto ka_load = [&](bf16x8 (&ka)[NP], int s, int kb, const uint16_t* Kd) {
#pragma unroll
    for (int pc = 0; pc < NP; ++pc)
      ka[pc] = *(const bf16x8*)(Kd + (s * 32 + l32) * KR + pc * D + kb * 16 + 8 * hh);
  };
  auto score_terms = [&](floatx16& o, const bf16x8 (&ka)[NP], int kb) {
    if constexpr (KX == kValF16) {
      o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[0]),
                                                 __builtin_bit_cast(f16x8, qB[0][kb]), o, 0, 0, 0);
    } else if constexpr (KX == kValBF16) {
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[0][kb], o, 0, 0, 0);
    } else if constexpr (F16P) {
      o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[1]),
                                                 __builtin_bit_cast(f16x8, qB[0][kb]), o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[0]),
                                                 __builtin_bit_cast(f16x8, qB[1][kb]), o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, ka[0]),
                                                 __builtin_bit_cast(f16x8, qB[0][kb]), o, 0, 0, 0);
    } else {
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[1], qB[0][kb], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[1][kb], o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0], qB[0][kb], o, 0, 0, 0);
    }
  };
  // probability of value r (exp of the lane's score), as float16 into pf
  auto exp_h = [&](const floatx16& o, int r, float& rs, f16x8 (&pf)[2]) {
    const float pr = fast_exp2(KX ? o[r] * cs : o[r]);
    rs += pr;
    pf[r >> 3][r & 7] = (_Float16)pr;
  };

  // bounded: no exponent of the tile can exceed m_run + kBoundMax (checked
  // from the norms), so the maxima are not needed
  // (The empty volatile asm keeps the maxima inside their branch: without it
  // the compiler computes them unconditionally.)
  auto fast_tile = [&](const uint16_t* Kd, const uint16_t* Vt, int jt_next, int stage_next,
                       bool bounded) {
    // ---- A ----
    // The phases that are matrix-core work only (A and D) run at raised wave
    // priority, so that the other wavefront of the SIMD, in its softmax,
    // does not hold back their MFMA issue (measured: -3% per tile).
    floatx16 s0, s1;
    __builtin_amdgcn_s_setprio(1);
    score_sub(s0, 0, Kd, negm);
    __builtin_amdgcn_s_setprio(0);
    if (!bounded) {
      asm volatile("");
      if (__builtin_amdgcn_ballot_w64(sub_max(s0) * cs > kLazyMax)) return false;
    }
    // ---- B: scores(1) || softmax(0) ----
    f16x8 p0[2];
    float rs = 0.f;
    {
      s1 = negm;
      bf16x8 ka[2][NP];
      ka_load(ka[0], 1, 0, Kd);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        if (kb + 1 < NKB) ka_load(ka[(kb + 1) & 1], 1, kb + 1, Kd);
        score_terms(s1, ka[kb & 1], kb);
        // 16 probabilities of sub-tile 0 spread over the NKB slices
#pragma unroll
        for (int q = 0; q < 16 / NKB; ++q) exp_h(s0, kb * (16 / NKB) + q, rs, p0);
      }
    }
    l_run += rs;
    if (!bounded) {
      asm volatile("");
      const float mt1 = sub_max(s1) * cs;  // largest t - m_run of sub-tile 1
      const bool up1 = mt1 > kLazyMax;
      if (__builtin_amdgcn_ballot_w64(up1)) {
        const float dm = up1 ? mt1 : 0.f;
        rescale(fast_exp2(-dm));  // also rescales sub-tile 0's share of l
        set_m(m_run + dm);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          p0[r >> 3][r & 7] = (_Float16)fast_exp2((KX ? s0[r] * cs : s0[r]) - dm);
          s1[r] -= KX ? dm / cs : dm;
        }
      }
    }
    // ---- C: P.V(0) || softmax(1) ----
    f16x8 p1[2];
    rs = 0.f;
    f16x8 va[2][NDB];
    va_load(va[0], 0, 0, Vt);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      va_load(va[(kk + 1) & 1], kk == 0 ? 0 : 1, kk == 0 ? 1 : 0, Vt);  // next PV block
      pv_terms(va[kk & 1], p0[kk]);
#pragma unroll
      for (int q = 0; q < 8; ++q) exp_h(s1, 8 * kk + q, rs, p1);
    }
    l_run += rs;
    __builtin_amdgcn_s_setprio(1);
    // ---- D: P.V(1) || next tile's LDS writes ----
    va_load(va[1], 1, 1, Vt);
    pv_terms(va[0], p1[0]);
    write_tile_keys(stage_next, jt_next);
    pv_terms(va[1], p1[1]);
    write_tile_v(stage_next, jt_next);
    __builtin_amdgcn_s_setprio(0);
    return true;
  };

  // a 32-key sub-tile from key a on is seen by some row of this wave: it holds
  // a global key, the wave a global row, or it meets some row's window
  auto in_window = [&](int a) {
    return !win || a < p.n_global || wave_i_min < p.n_global ||
           (a + 31 > wave_i_min - p.window && a < wave_i_max + p.window);
  };
  for (int t = 0; t < ntiles; ++t) {
    const int jt = tile_at(t), jt_next = tile_at(t + 1);
    const int j0 = jt * kBC;
    const int stage = NS == 2 ? (t & 1) : 0;
    if constexpr (NS == 1) {
      load_tile(jt);
      write_tile(0, jt);
      __syncthreads();
    } else {
      load_tile(jt_next);  // past the end it reads clamped, valid addresses; unused
      if constexpr (kDMA) {
        if (t + 1 < ntiles) dma_stage(stage ^ 1, jt_next);
      }
    }
    const uint16_t* Kd = (const uint16_t*)(smem + stage * SB);
    const unsigned char* vt = smem + stage * SB + kBC * KR * 2;
    const bool act0 = (!p.causal || wave_i_max >= j0) && in_window(j0);
    const bool act1 = (!p.causal || wave_i_max >= j0 + 32) && in_window(j0 + 32);
    // the token window cuts into this tile for some row of the wave
    const bool wcut = win && j0 + kBC > p.n_global &&
                      (wave_i_min < p.n_global || wave_i_max - j0 >= p.window ||
                       j0 + kBC - 1 - wave_i_min >= p.window);
    const bool need_mask = j0 + kBC > n || (p.causal && j0 + kBC - 1 > wave_i_min) || wcut ||
                           __builtin_amdgcn_ballot_w64(!row_ok || m_run == -INFINITY) != 0;
    bool done = false;
    if constexpr (NS == 2 && VBF16 && !SAFE) {
      if (act0 && act1 && !need_mask) {
        // largest key norm of the tile, kept by the prepared image in the
        // padding of key row 0
        const float kn = *(const float*)(Kd + NP * D);
        const bool bounded = !__builtin_amdgcn_ballot_w64(!(qn * kn <= m_run + kBoundMax));
        done = fast_tile(Kd, (const uint16_t*)vt, jt_next, stage ^ 1, bounded);
      }
    }
    if (!done) {
      if (act0) generic_sub(j0, 0, Kd, vt);
      if (act1) generic_sub(j0, 1, Kd, vt);
      if constexpr (NS == 2) write_tile(stage ^ 1, jt_next);
    }
    wait_dma();
    __syncthreads();
  }
  l_run = pair_sum(l_run);  // lane-partial row sums -> row sums

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

// d = 64, bf16 V, 4 wavefronts: at most 168 VGPRs, so that three
// workgroups (three waves per SIMD) share a compute unit, as their LDS
// allows; with two, short sequences were latency-bound (measured: the gpt2s
// shape's forward kernel 77 -> 54 us).
template <int D, bool VBF16, int NW, int KM, int KX>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(D == 64 && VBF16 && NW == 4 ? 3 : 1)))
void sfa_fwd_kernel(FwdParams p) {
  // longest causal blocks first
  // Workgroups are dispatched round-robin over the 8 XCDs (each with its own
  // L2): with the (batch, KV head) count a multiple of 8, XCD x runs the KV
  // heads congruent to x, so one L2 serves all query blocks of a head, which
  // sweep its key tiles together.  Longest causal blocks first either way.
  const int nbh = (int)gridDim.y;
  int qb = (int)blockIdx.x, bh = (int)blockIdx.y;
  if (nbh % 8 == 0) {
    const int id = qb + bh * p.nqb;
    const int xcd = id & 7, j = id >> 3;
    qb = j % p.nqb;
    bh = xcd + 8 * (j / p.nqb);
    if constexpr (D == 64 && VBF16 && NW == 4) {
      // Three of these workgroups share a compute unit, all resident at
      // once, so nothing evens out their causal lengths later: successive
      // heads of an XCD take the blocks longest-first, shortest-first and
      // half-rotated, which mixes long and short blocks on a compute unit
      // under in-order dispatch (measured: gpt2s shape 54 -> 50 us).
      const int r = (j / p.nqb) % 3;
      if (r == 1) qb = p.nqb - 1 - qb;
      else if (r == 2) qb = (qb + p.nqb / 2) % p.nqb;
    }
  }
  if (p.ix && *p.ix_stat <= p.ix_thresh) return;  // the index mode takes this call
  fwd_block<D, VBF16, NW, KM, false, KX>(p, p.nqb - 1 - qb, bh);
}

// Whether workgroup t = bh * nqb + qb was handed back (its first output
// element holds the hand-back bits).
__device__ __forceinline__ bool handed_back(const FwdParams& p, int t, int D) {
  const int qb = t % p.nqb, bh = t / p.nqb;
  const int b = bh / p.Hkv, hkv = bh - b * p.Hkv;
  const int64_t orow0 = ((int64_t)b * p.Hq + hkv * p.G) * p.n + (int64_t)qb * p.BR;
  return p.obf16 ? ((const uint16_t*)p.o)[orow0 * D] == kHandBack16
                 : ((const uint32_t*)p.o)[orow0 * D] == kHandBack32;
}

// bf16-V rerun, launched after sfa_fwd_kernel on the same stream: a
// persistent grid checks every workgroup's hand-back mark (one load per
// thread) and recomputes only the marked ones.
template <int D, int NW, int KM>
__global__ __launch_bounds__(NW * 64) void sfa_fwd_rerun_kernel(FwdParams p, int nbh) {
  constexpr int NT = NW * 64;
  if (*p.hb_count == 0) return;  // no workgroup was handed back
  const int total = p.nqb * nbh;
  const int stride = (int)gridDim.x;
  for (int base = (int)blockIdx.x; base < total; base += stride * NT) {
    const int t = base + (int)threadIdx.x * stride;
    if (!__syncthreads_or(t < total && handed_back(p, t, D))) continue;
    for (int c = 0; c < NT; ++c) {
      const int tc = base + c * stride;
      if (tc >= total) break;
      if (!__syncthreads_or(threadIdx.x == 0 && handed_back(p, tc, D))) continue;
      fwd_block<D, true, NW, KM, true>(p, tc % p.nqb, tc / p.nqb);
      __syncthreads();  // LDS is reused by the next workgroup
    }
  }
}

// ---------------------------------------------------------------------------
// Inverted-index score mode (Sec. 3.2: intersect the supports through the
// keys' active features), for small k.
//
// Each key tile's inverted index is built once per call by
// sfa_fwd_ix_prep_kernel into the forward's workspace: bucket b = 2u + p
// lists the tile's keys of parity p that hold coordinate u, as (key, value)
// entries sorted by bucket, with the bucket bounds, the tile's largest key
// norm and the float16 V^T tile of the dense image beside them.  The forward
// copies a tile's index into LDS with direct-to-LDS loads (the next tile in
// flight).  The two lanes of a query row (key parities p = 0, 1) walk the
// buckets of the row's nonzeros (u, q_u): for each entry (key c, k_cu) of
// bucket 2u + p they add q_u * k_cu into S[row][c] of the wave's private
// score block.  Only overlapping coordinates cost work; every score entry
// has one owner lane (the key's parity), so the adds are plain
// read-modify-writes, and each entry sums its overlaps in the row's code
// order (float32 products and sums).  The wave reads its scores back in the
// P.V operand layout, clears the entries it touched by a second walk, and
// runs the online softmax and float16 P.V of the dense mode.
// ---------------------------------------------------------------------------
// Largest k of the index mode, which runs at d = 128 only: beyond k = 2, and
// at d = 64 (half the dense score work), the dense product on the matrix
// cores is faster on every input measured.
constexpr int kIxMaxK = 2;
constexpr int kIxD = 128;

template <int D, int KM>
struct IxGeo {
  static constexpr int NBND = 2 * D + 2;                        // bucket bounds 0..2D (+1 pad)
  static constexpr int ENT = (NBND * 2 + 15) / 16 * 16;          // entries (uint2) start, bytes
  static constexpr int NORM = ENT + kBC * KM * 8;                // largest key norm (float)
  static constexpr int VT = (NORM + 16 + 1023) / 1024 * 1024;    // float16 V^T tile
  static constexpr int SB = VT + vtile_bytes<D>();               // image bytes (whole KB)
  static constexpr int SPK = kBC + 4;                            // score block row pitch (floats)
};

template <int D, int NW, int KM>
__host__ __device__ constexpr int ix_lds_bytes() {
  return 2 * IxGeo<D, KM>::SB + NW * 32 * IxGeo<D, KM>::SPK * 4;
}

// Index images: image t of (batch, KV head) bh holds keys 64t .. 64t+63.
// The bucket order within a bucket follows the counting sort's atomics; it
// does not change any result (a key enters a bucket once, and a score entry
// sums its coordinates in the query row's order).  flag t as for the dense
// images (a V value outside the float16 range).
template <int D, int KM>
__global__ __launch_bounds__(256) void sfa_fwd_ix_prep_kernel(
    const void* __restrict__ k_idx, const void* __restrict__ k_val, const uint16_t* __restrict__ v,
    int n, int k, int ifmt, int vfmt, int vtiles, unsigned char* __restrict__ ws_tiles,
    int* __restrict__ ws_flag, uint32_t* __restrict__ ix_stat) {
  using Gx = IxGeo<D, KM>;
  constexpr int VP = kBC + 4;
  __shared__ __attribute__((aligned(16))) unsigned char T[Gx::SB];
  __shared__ uint32_t cnt[2 * D];
  __shared__ float kn2[kBC];
  uint16_t* off = (uint16_t*)T;
  uint2* ent = (uint2*)(T + Gx::ENT);
  uint16_t* Vt = (uint16_t*)(T + Gx::VT);
  const int t = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int j0 = t * kBC;
  const int nk = min(kBC, n - j0);  // keys of the tile
  for (int i = tid; i < Gx::SB / 16; i += 256) ((uint4*)T)[i] = make_uint4(0u, 0u, 0u, 0u);
  for (int i = tid; i < 2 * D; i += 256) cnt[i] = 0u;
  __syncthreads();
  const int64_t c0 = ((int64_t)bh * n + j0) * k;  // first code element of the tile
  constexpr int EPT = (kBC * KM + 255) / 256;     // code entries per thread
  int eb[EPT], es[EPT], ec[EPT];
  float ev[EPT];
#pragma unroll
  for (int r = 0; r < EPT; ++r) {
    const int e = tid + 256 * r;
    eb[r] = -1;
    if (e < nk * k) {
      const int c = e / k;
      ec[r] = c;
      eb[r] = 2 * load_idx(k_idx, c0 + e, ifmt, D - 1) + (c & 1);
      ev[r] = load_val(k_val, c0 + e, vfmt);
      es[r] = (int)atomicAdd(&cnt[eb[r]], 1u);
    }
  }
  __syncthreads();
  if (tid < 64) {  // exclusive scan of the 2D bucket counts, F consecutive per lane
    constexpr int F = 2 * D / 64;
    uint32_t c[F], local = 0;
#pragma unroll
    for (int f = 0; f < F; ++f) { c[f] = cnt[tid * F + f]; local += c[f]; }
    uint32_t incl = local;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(incl, o, 64);
      if (tid >= o) incl += y;
    }
    uint32_t run = incl - local, big = 0;
#pragma unroll
    for (int f = 0; f < F; ++f) { off[tid * F + f] = (uint16_t)run; run += c[f]; big = max(big, c[f]); }
    if (tid == 63) off[2 * D] = (uint16_t)incl;
    big = wave_umax(big);  // the tile's longest bucket
    if (tid == 0) atomicAdd(ix_stat, big);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < EPT; ++r)
    if (eb[r] >= 0) ent[off[eb[r]] + es[r]] = make_uint2((uint32_t)ec[r], __float_as_uint(ev[r]));
  // largest Euclidean norm of the tile's key codes (times 1 + 2^-8)
  if (tid < kBC) {
    float acc = 0.f;
    if (tid < nk)
      for (int e = 0; e < k; ++e) {
        const float x = load_val(k_val, c0 + (int64_t)tid * k + e, vfmt);
        acc = fmaf(x, x, acc);
      }
    kn2[tid] = acc;
  }
  __syncthreads();
  if (tid == 0) {
    float mx = 0.f;
    for (int j = 0; j < kBC; ++j) mx = fmaxf(mx, kn2[j]);
    *(float*)(T + Gx::NORM) = sqrtf(mx) * (1.f + 1.f / 256.f);
  }
  // V^T as float16, [dimension][key], and the V range flag (as the dense image)
  const uint16_t* src = v + ((int64_t)bh * n + j0) * D;
  bool over = false;
  for (int c = tid; c < kBC * D / 8; c += 256) {
    const int j = c / (D / 8), d0 = (c % (D / 8)) * 8;
    if (j >= nk) break;
    const uint4 w4 = *(const uint4*)(src + (int64_t)j * D + d0);
    const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      over |= (w[e] & 0x7fffu) >= 0x4780u || ((w[e] >> 16) & 0x7fffu) >= 0x4780u;
      Vt[(d0 + 2 * e) * VP + j] = __builtin_bit_cast(uint16_t, (_Float16)bf16_bits_to_f32(w[e] & 0xffffu));
      Vt[(d0 + 2 * e + 1) * VP + j] = __builtin_bit_cast(uint16_t, (_Float16)bf16_bits_to_f32(w[e] >> 16));
    }
  }
  const int any = __syncthreads_or(over);
  uint4* dst = (uint4*)(ws_tiles + ((int64_t)bh * vtiles + t) * Gx::SB);
  for (int i = tid; i < Gx::SB / 16; i += 256) dst[i] = ((const uint4*)T)[i];
  if (tid == 0) ws_flag[(int64_t)bh * vtiles + t] = any ? 1 : 0;
}

// One workgroup of the index mode: query block qb of (batch, KV head) bh.
template <int D, int NW, int KM>
__device__ __forceinline__ void fwd_block_ix(const FwdParams& p, const int qb, const int bh) {
  using Gx = IxGeo<D, KM>;
  constexpr int NT = NW * 64, SB = Gx::SB, SPK = Gx::SPK, NDB = D / 32, VP = kBC + 4;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;  // P.V operand half; in the walks, the key parity
  const int l32 = lane & 31;
  const int k = p.k;
  const int n = p.n;
  const int b = bh / p.Hkv;
  const int hkv = bh - b * p.Hkv;
  const int i0 = qb * p.BR;
  const int rho = wave * 32 + l32;
  const int my_i = i0 + rho % p.BR;
  const int my_hq = hkv * p.G + rho / p.BR;
  const bool row_ok = my_i < n;
  float* Srow = (float*)(smem + 2 * SB) + (wave * 32 + l32) * SPK;  // S[row][key]

  const int blk_last = min(n, i0 + p.BR) - 1;
  const bool win = p.window > 0;
  int n_keys = p.causal ? blk_last + 1 : n;
  int gt_end = 0, wt_begin = 0;
  if (win && i0 >= p.n_global) {
    if (!p.causal) n_keys = min(n, blk_last + p.window);
    gt_end = (p.n_global + kBC - 1) / kBC;
    wt_begin = max(0, i0 - p.window + 1) / kBC;
    if (wt_begin <= gt_end) gt_end = wt_begin = 0;
  }
  const int ntiles_all = (n_keys + kBC - 1) / kBC;
  const int ntiles = gt_end + ntiles_all - wt_begin;
  auto tile_at = [&](int t) { return t < gt_end ? t : wt_begin + (t - gt_end); };
  auto dma_stage = [&](int stage, int jt) {
    constexpr int NB = SB / 1024, NJ = (NB + NW - 1) / NW;
    const unsigned char* src = p.ix_tiles + ((int64_t)bh * p.vtiles + jt) * SB;
    unsigned char* dst = smem + stage * SB;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int i = wave + j * NW;
      if (j + 1 < NJ || i < NB)
        __builtin_amdgcn_global_load_lds(src + (uint32_t)(i * 1024 + lane * 16),
                                         (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                         16, 0, 0);
    }
  };
  auto wait_dma = [&]() { __builtin_amdgcn_s_waitcnt(0x0f70); };  // vmcnt(0)

  int vflag = 0;
  if (tid < ntiles) vflag = p.ws_flag[(int64_t)bh * p.vtiles + tile_at(tid)];
  // the row's nonzeros: bucket 2u + (this lane's key parity) and q_u * scale * log2(e)
  int qbk[KM];
  float qx[KM];
  float qn = 0.f;
#pragma unroll
  for (int t = 0; t < KM; ++t) {
    qbk[t] = -1;
    qx[t] = 0.f;
    if (t < k && row_ok) {
      const int64_t gi = (((int64_t)b * p.Hq + my_hq) * n + my_i) * k + t;
      qbk[t] = 2 * load_idx(p.q_idx, gi, p.ifmt, D - 1) + hh;
      qx[t] = p.scale_log2 * load_val(p.q_val, gi, p.vfmt);
      qn = fmaf(qx[t], qx[t], qn);
    }
  }
  qn = sqrtf(qn) * (1.f + 1.f / 256.f);  // Cauchy-Schwarz bound of the row's exponents per unit key norm
  if (ntiles > 0) dma_stage(0, tile_at(0));
  // the wave's score block starts at zero; the walks leave it at zero
  for (int x = lane; x < 32 * SPK / 4; x += 64)
    ((float4*)((float*)(smem + 2 * SB) + wave * 32 * SPK))[x] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int t = tid + NT; t < ntiles; t += NT) vflag |= p.ws_flag[(int64_t)bh * p.vtiles + tile_at(t)];
  if (__syncthreads_or(vflag != 0)) {
    wait_dma();
    if (tid == 0) {
      const int64_t orow0 = ((int64_t)b * p.Hq + hkv * p.G) * n + i0;
      if (p.obf16) ((uint16_t*)p.o)[orow0 * D] = kHandBack16;
      else ((uint32_t*)p.o)[orow0 * D] = kHandBack32;
      *p.hb_count = 1;
    }
    return;
  }

  float m_run = -INFINITY, l_run = 0.f;
  floatx16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;
  const int wave_i_max = i0 + (wave * 32 + 31) % p.BR;
  const int wave_i_min = p.BR >= 32 ? i0 + (wave * 32) % p.BR : i0;
  auto in_window = [&](int a) {
    return !win || a < p.n_global || wave_i_min < p.n_global ||
           (a + 31 > wave_i_min - p.window && a < wave_i_max + p.window);
  };
  // Walk the row's buckets: add q_u k_cu into S[row][c] (zero: clear the
  // entries instead).  The bucket bounds of all the row's terms are read
  // first; a bucket holds a key at most once, so its entries go four at a
  // time (four reads, then four read-modify-writes); a key met again under a
  // later term is read after the earlier write (a wave's LDS operations run
  // in order).
  auto walk = [&](const uint16_t* off, const uint2* ent, bool zero) {
    int e0[KM], e1[KM];
#pragma unroll
    for (int t = 0; t < KM; ++t) {
      const int bk = qbk[t] < 0 ? 0 : qbk[t];
      e0[t] = off[bk];
      e1[t] = qbk[t] < 0 ? e0[t] : off[bk + 1];
    }
#pragma unroll
    for (int t = 0; t < KM; ++t) {
      for (int e = e0[t]; e < e1[t]; e += 4) {
        uint2 en[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) en[u] = ent[min(e + u, e1[t] - 1)];
        if (zero) {
#pragma unroll
          for (int u = 0; u < 4; ++u) Srow[en[u].x] = 0.f;
        } else {
          float sv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) sv[u] = Srow[en[u].x];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (e + u < e1[t]) Srow[en[u].x] = fmaf(qx[t], __uint_as_float(en[u].y), sv[u]);
        }
      }
    }
  };
  auto pv_sub = [&](int s, const floatx16& pr, const uint16_t* Vt) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      f16x8 pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (_Float16)pr[8 * kk + e];
      const int kbase = 32 * s + 16 * kk + 4 * hh;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint16_t* row = Vt + (db * 32 + l32) * VP + kbase;
        const uint2 v0 = *(const uint2*)row;
        const uint2 v1 = *(const uint2*)(row + 8);
        const u32x4 vw = {v0.x, v0.y, v1.x, v1.y};
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, vw), pf,
                                                         acc[db], 0, 0, 0);
      }
    }
  };

  wait_dma();
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int jt = tile_at(t), jt_next = tile_at(t + 1);
    const int j0 = jt * kBC;
    const int stage = t & 1;
    if (t + 1 < ntiles) dma_stage(stage ^ 1, jt_next);
    const unsigned char* img = smem + stage * SB;
    const uint16_t* off = (const uint16_t*)img;
    const uint2* ent = (const uint2*)(img + Gx::ENT);
    const uint16_t* Vt = (const uint16_t*)(img + Gx::VT);
    const bool act0 = (!p.causal || wave_i_max >= j0) && in_window(j0);
    const bool act1 = (!p.causal || wave_i_max >= j0 + 32) && in_window(j0 + 32);
    if (act0 || act1) {
      walk(off, ent, false);
      floatx16 sc[2];
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 x = *(const float4*)(Srow + 32 * s + 8 * g + 4 * hh);
          sc[s][4 * g + 0] = x.x; sc[s][4 * g + 1] = x.y; sc[s][4 * g + 2] = x.z; sc[s][4 * g + 3] = x.w;
        }
      walk(off, ent, true);
      const bool wcut = win && j0 + kBC > p.n_global &&
                        (wave_i_min < p.n_global || wave_i_max - j0 >= p.window ||
                         j0 + kBC - 1 - wave_i_min >= p.window);
      const bool need_mask = j0 + kBC > n || (p.causal && j0 + kBC - 1 > wave_i_min) || wcut ||
                             __builtin_amdgcn_ballot_w64(!row_ok || m_run == -INFINITY) != 0;
      const float kn = *(const float*)(img + Gx::NORM);
      // every exponent of the tile is below m_run + kBoundMax: no maxima needed
      const bool bounded =
          !need_mask && !__builtin_amdgcn_ballot_w64(!(qn * kn <= m_run + kBoundMax));
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        if (!(s == 0 ? act0 : act1)) continue;
        floatx16 x = sc[s];
        float m_use = m_run;
        if (!bounded) {
          float mt = -INFINITY;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int j = j0 + 32 * s + 8 * (r >> 2) + 4 * hh + (r & 3);
            const bool ok = !need_mask ||
                            (row_ok && j < n && (!p.causal || j <= my_i) &&
                             (!win || abs(my_i - j) < p.window || j < p.n_global ||
                              my_i < p.n_global));
            x[r] = ok ? x[r] : -INFINITY;
            mt = fmaxf(mt, x[r]);
          }
          mt = pair_max(mt);
          const bool upd = mt > m_run + kLazyMax;
          const float m_new = upd ? mt : m_run;
          m_use = (m_new == -INFINITY) ? 0.f : m_new;
          if (__builtin_amdgcn_ballot_w64(upd)) {
            const float alpha = upd ? fast_exp2(m_run - m_use) : 1.f;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < NDB; ++db)
#pragma unroll
              for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;
            m_run = m_new;
          }
        }
        float rs = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) { x[r] = fast_exp2(x[r] - m_use); rs += x[r]; }
        l_run += rs;
        pv_sub(s, x, Vt);
      }
    }
    wait_dma();
    __syncthreads();
  }
  l_run = pair_sum(l_run);

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

template <int D, int NW, int KM>
__global__ __launch_bounds__(NW * 64) void sfa_fwd_ix_kernel(FwdParams p) {
  // workgroup placement as sfa_fwd_kernel (XCD-aware, longest causal blocks first)
  const int nbh = (int)gridDim.y;
  int qb = (int)blockIdx.x, bh = (int)blockIdx.y;
  if (nbh % 8 == 0) {
    const int id = qb + bh * p.nqb;
    const int xcd = id & 7, j = id >> 3;
    qb = j % p.nqb;
    bh = xcd + 8 * (j / p.nqb);
  }
  if (*p.ix_stat > p.ix_thresh) return;  // skewed buckets: the dense mode takes this call
  fwd_block_ix<D, NW, KM>(p, p.nqb - 1 - qb, bh);
}

// Stage images for bf16 V, built once per call: image t of (batch, KV head) bh
// is exactly what the forward kernel holds in LDS for keys 64t .. 64t+63:
//   - the dense key tile [key][piece][coordinate] (pitch KR) with the codes'
//     values as float16 pieces x0 = f16(x), x1 = f16(x - x0) at their
//     coordinates and zeros elsewhere (KX: 16-bit codes, the raw values,
//     one piece);
//   - V^T as float16, [dimension][key] (pitch kBC + 4);
//   - in the padding of key row 0, the largest Euclidean norm of the tile's
//     key codes (times 1 + 2^-8), which bounds the tile's scores.
// Keys past n and the rest of the padding are zero.  flag t is set when a V value of the
// tile lies outside the float16 range (|v| >= 65536, inf, NaN), or (32-bit
// codes) a key value is too large for float16 pieces (|x| >= 65504).  bf16 ->
// float16 is exact for 2^-14 <= |v| <= 65504; below that it rounds to the
// float16 subnormal grid (absolute error <= 2^-25).
// Every global load of the tile is issued before the first use (one memory
// round trip, then the LDS work, then the stores): with k <= 16 the code
// entries and the V chunks sit in registers, and the norms of the tile's 64
// keys are taken by lanes 0-63 from loads of their own.
template <int D, int KX>
__global__ __launch_bounds__(256) void sfa_fwd_prep_kernel(
    const void* __restrict__ k_idx, const void* __restrict__ k_val, const uint16_t* __restrict__ v,
    int n, int k, int ifmt, int vfmt, int vtiles, unsigned char* __restrict__ ws_tiles,
    int* __restrict__ ws_flag, const uint32_t* __restrict__ ix_stat, uint32_t ix_thresh,
    int* __restrict__ hb_count) {
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *hb_count = 0;
  constexpr int NP = n_pieces<true, KX>();
  constexpr int KR = Geo<D, NP>::KR, VP = kBC + 4, SB = stage_bytes<D, true, KX>();
  constexpr int KE = kBC * 16 / 256;   // code entries per thread for k <= 16
  constexpr int VC = kBC * D / 8 / 256;  // 16-byte V chunks per thread
  static_assert(KE * 256 == kBC * 16 && VC * 256 * 8 == kBC * D, "whole tiles per thread");
  __shared__ __attribute__((aligned(16))) uint16_t T[SB / 2];
  uint16_t* Vt = T + kBC * KR;
  const int t = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int j0 = t * kBC;
  const int nk = min(kBC, n - j0);                // keys of this tile
  const int64_t c0 = ((int64_t)bh * n + j0) * k;  // first code element of the tile
  const bool small_k = k <= 16;

  // ---- global loads ----
  int ci[KE];
  float cx[KE];
#pragma unroll
  for (int i = 0; i < KE; ++i) {
    const int e = tid + 256 * i;
    ci[i] = -1;
    cx[i] = 0.f;
    if (small_k && e < nk * k) {
      ci[i] = load_idx(k_idx, c0 + e, ifmt, D - 1);
      cx[i] = KX != 0 ? __uint_as_float((uint32_t)((const uint16_t*)k_val)[c0 + e])
                      : load_val(k_val, c0 + e, vfmt);
    }
  }
  const uint16_t* src = v + ((int64_t)bh * n + j0) * D;
  uint4 vw[VC];
#pragma unroll
  for (int i = 0; i < VC; ++i) {  // chunk c: key c / (D / 8), dimensions 8 (c % (D / 8)) + 0..7
    const int c = tid + 256 * i, j = c / (D / 8), d0 = (c % (D / 8)) * 8;
    vw[i] = j < nk ? *(const uint4*)(src + (int64_t)j * D + d0) : make_uint4(0u, 0u, 0u, 0u);
  }
  float kx[16];  // lanes 0-63: the code values of key tid (k <= 16)
#pragma unroll
  for (int e = 0; e < 16; ++e)
    kx[e] = (small_k && tid < nk && e < k) ? load_val(k_val, c0 + (int64_t)tid * k + e, vfmt) : 0.f;
  if (ix_stat && *ix_stat <= ix_thresh) return;  // the index mode takes this call

  for (int i = tid; i < SB / 16; i += 256) ((uint4*)T)[i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  bool over = false;
  auto put = [&](int j, int f, float x) {  // x: the value (KX: its 16-bit pattern)
    if constexpr (KX != 0) {
      T[j * KR + f] = (uint16_t)__float_as_uint(x);
    } else {
      over |= fabsf(x) >= kF16PieceMax;
      T[j * KR + f] = f16_piece(x, 0);
      T[j * KR + D + f] = f16_piece(x, 1);
    }
  };
  if (small_k) {
#pragma unroll
    for (int i = 0; i < KE; ++i)
      if (ci[i] >= 0) put((tid + 256 * i) / k, ci[i], cx[i]);
  } else {
    for (int e = tid; e < nk * k; e += 256)
      put(e / k, load_idx(k_idx, c0 + e, ifmt, D - 1),
          KX != 0 ? __uint_as_float((uint32_t)((const uint16_t*)k_val)[c0 + e])
                  : load_val(k_val, c0 + e, vfmt));
  }
  // largest Euclidean norm of the tile's key codes (padding of key row 0),
  // each key's squares summed in code order
  if (tid < kBC) {
    float acc = 0.f;
    if (small_k) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc = fmaf(kx[e], kx[e], acc);
    } else if (tid < nk) {
      for (int e = 0; e < k; ++e) {
        const float x = load_val(k_val, c0 + (int64_t)tid * k + e, vfmt);
        acc = fmaf(x, x, acc);
      }
    }
    const float mx = wave_max_dpp(acc);  // wave 0, all 64 lanes
    if (tid == 0) *(float*)(T + NP * D) = sqrtf(mx) * (1.f + 1.f / 256.f);
  }
#pragma unroll
  for (int i = 0; i < VC; ++i) {
    const int c = tid + 256 * i, j = c / (D / 8), d0 = (c % (D / 8)) * 8;
    if (j >= nk) continue;  // keys past n stay zero
    const uint32_t w[4] = {vw[i].x, vw[i].y, vw[i].z, vw[i].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      over |= (w[e] & 0x7fffu) >= 0x4780u || ((w[e] >> 16) & 0x7fffu) >= 0x4780u;
      Vt[(d0 + 2 * e) * VP + j] = __builtin_bit_cast(uint16_t, (_Float16)bf16_bits_to_f32(w[e] & 0xffffu));
      Vt[(d0 + 2 * e + 1) * VP + j] = __builtin_bit_cast(uint16_t, (_Float16)bf16_bits_to_f32(w[e] >> 16));
    }
  }
  const int any = __syncthreads_or(over);
  uint4* dst = (uint4*)(ws_tiles + ((int64_t)bh * vtiles + t) * SB);
  for (int i = tid; i < SB / 16; i += 256) dst[i] = ((const uint4*)T)[i];
  if (tid == 0) ws_flag[(int64_t)bh * vtiles + t] = any ? 1 : 0;
}

template <int D, bool VBF16, int NW, int KM, int KX>
hipError_t launch_km(const FwdParams& p, int B, hipStream_t stream) {
  constexpr int bytes = lds_bytes<D, VBF16, NW, KX>();
  constexpr int rbytes = lds_bytes<D, true, NW, 0, true>();  // the rerun: three bf16 pieces
  // once per instantiation (a function-local static: initialised once, also
  // under concurrent first calls)
  static const hipError_t configured = [] {
    hipError_t e = hipSuccess;
    if (bytes > 65536)
      e = hipFuncSetAttribute((const void*)sfa_fwd_kernel<D, VBF16, NW, KM, KX>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess && VBF16 && rbytes > 65536)
      e = hipFuncSetAttribute((const void*)sfa_fwd_rerun_kernel<D, NW, KM>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, rbytes);
    return e;
  }();
  if (configured != hipSuccess) return configured;
  dim3 grid(p.nqb, B * p.Hkv), block(NW * 64);
  hipLaunchKernelGGL((sfa_fwd_kernel<D, VBF16, NW, KM, KX>), grid, block, bytes, stream, p);
  if constexpr (VBF16) {
    // one resident workgroup per compute unit (LDS-bound)
    const int total = p.nqb * B * p.Hkv;
    dim3 rgrid(total < 256 ? total : 256);
    hipLaunchKernelGGL((sfa_fwd_rerun_kernel<D, NW, KM>), rgrid, block, rbytes, stream, p, B * p.Hkv);
  }
  return hipGetLastError();
}

// Index score mode: its forward (returning at once when the dense mode was
// chosen); the dense forward and the rerun follow on the stream.
template <int D, int NW, int KM>
hipError_t launch_ix(const FwdParams& p, int B, hipStream_t stream) {
  constexpr int bytes = ix_lds_bytes<D, NW, KM>();
  static const hipError_t configured = [] {  // once per instantiation
    return hipFuncSetAttribute((const void*)sfa_fwd_ix_kernel<D, NW, KM>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  }();
  if (configured != hipSuccess) return configured;
  dim3 grid(p.nqb, B * p.Hkv), block(NW * 64);
  hipLaunchKernelGGL((sfa_fwd_ix_kernel<D, NW, KM>), grid, block, bytes, stream, p);
  return hipGetLastError();
}

template <int D, bool VBF16, int NW>
hipError_t launch_nw(FwdParams p, int B, hipStream_t stream) {
  p.BR = NW * 32 / p.G;
  p.nqb = (p.n + p.BR - 1) / p.BR;
  if constexpr (VBF16 && D == kIxD) {
    if (p.ix) {
      const hipError_t e = launch_ix<D, NW, kIxMaxK>(p, B, stream);
      if (e != hipSuccess) return e;
    }
  }
  if constexpr (VBF16) {
    if (p.kx == kValBF16)
      return p.k <= 16 ? launch_km<D, true, NW, 16, kValBF16>(p, B, stream)
                       : launch_km<D, true, NW, 128, kValBF16>(p, B, stream);
    if (p.kx == kValF16)
      return p.k <= 16 ? launch_km<D, true, NW, 16, kValF16>(p, B, stream)
                       : launch_km<D, true, NW, 128, kValF16>(p, B, stream);
  }
  return p.k <= 16 ? launch_km<D, VBF16, NW, 16, 0>(p, B, stream)
                   : launch_km<D, VBF16, NW, 128, 0>(p, B, stream);
}

template <int D, bool VBF16>
hipError_t launch_t(const FwdParams& p, int B, hipStream_t stream) {
  // 8 wavefronts (256 rows) per workgroup when that still gives >= 4
  // workgroups per compute unit; else 4 wavefronts.  d = 64 with bf16 V
  // always takes 4: three such workgroups fit a compute unit (12 waves,
  // against 8 for one 8-wave workgroup), faster at every length measured
  // (n = 1024, 4096, 16384).
  const long long wg8 = (long long)((p.n + 256 / p.G - 1) / (256 / p.G)) * B * p.Hkv;
  if (!(D == 64 && VBF16) && p.G <= 8 && wg8 >= 4LL * 256) return launch_nw<D, VBF16, 8>(p, B, stream);
  return launch_nw<D, VBF16, 4>(p, B, stream);
}

}  // namespace

// The index mode's choice: mean longest bucket per tile at most this (the
// walks of a wave last as long as its longest bucket).
constexpr uint32_t kIxMeanLongest = 6;

__global__ void sfa_fwd_ix_stat_zero_kernel(uint32_t* stat) { stat[threadIdx.x] = 0u; }

int fwd_max_group() { return 128; }

// Workspace (bf16 V): the dense tile images, one V range flag per tile, the
// hand-back count (own 256-byte block), the index-mode tile images and the
// index mode's statistic.
size_t fwd_workspace_bytes(int B, int Hkv, int n, int d, int vbf16) {
  if (!vbf16) return 0;
  const size_t tiles = (size_t)B * Hkv * (size_t)((n + kBC - 1) / kBC);
  const size_t sb = d == 64 ? stage_bytes<64, true>() : stage_bytes<128, true>();
  const size_t ix = d == kIxD ? tiles * IxGeo<kIxD, kIxMaxK>::SB + 256 : 0;
  return tiles * sb + (tiles * 4 + 255) / 256 * 256 + 256 + ix;
}

hipError_t launch_attn_fwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, int B, int Hq, int Hkv, int n, int d,
                           int k, int causal, int window, int n_global, float scale, int ifmt,
                           int vfmt, int vbf16, int obf16, void* o, float* lse, void* ws,
                           hipStream_t stream) {
  FwdParams p;
  p.q_idx = q_idx; p.q_val = q_val; p.k_idx = k_idx; p.k_val = k_val; p.v = v;
  p.o = o; p.lse = lse;
  p.Hq = Hq; p.Hkv = Hkv; p.n = n; p.k = k; p.causal = causal;
  p.window = window; p.n_global = n_global;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);
  p.ifmt = ifmt; p.vfmt = vfmt; p.obf16 = obf16;
  // 16-bit code values with bf16 V take the one-product score path (a zero
  // scale keeps the piece path: its scores are all zero)
  p.kx = vbf16 && vfmt != kValF32 && scale != 0.f ? vfmt : 0;
  p.kx_scale = (float)(fabs((double)scale) * 1.4426950408889634);
  p.ix = vbf16 && k <= kIxMaxK && d == kIxD;
  p.ix_tiles = nullptr;
  p.ix_stat = nullptr;
  p.ix_thresh = 0;
  p.qsign = scale < 0.f ? 0x8000u : 0u;
  p.G = Hq / Hkv;
  p.BR = 0; p.nqb = 0;
  p.inv_k = 1.0f / (float)k;
  p.vtiles = (n + kBC - 1) / kBC;
  p.ws_tiles = (const unsigned char*)ws;
  p.ws_flag = nullptr;
  p.hb_count = nullptr;
  if (vbf16) {
    const size_t tiles = (size_t)B * Hkv * p.vtiles;
    const size_t sb = d == 64 ? stage_bytes<64, true>() : stage_bytes<128, true>();
    const size_t sbx = IxGeo<kIxD, kIxMaxK>::SB;
    p.ws_flag = (const int*)((unsigned char*)ws + tiles * sb);
    p.hb_count = (int*)((unsigned char*)ws + tiles * sb + (tiles * 4 + 255) / 256 * 256);
    unsigned char* wx = (unsigned char*)p.hb_count + 256;
    uint32_t* stat = (uint32_t*)(wx + tiles * sbx);
    dim3 grid(p.vtiles, B * Hkv), block(256);
    unsigned char* wt = (unsigned char*)ws;
    int* wf = (int*)p.ws_flag;
    const uint16_t* vb = (const uint16_t*)v;
    const uint32_t* gstat = nullptr;  // the dense pre-pass skips itself if the index mode runs
    if (p.ix) {
      p.ix_tiles = wx;
      p.ix_stat = stat;
      p.ix_thresh = (uint32_t)std::min<size_t>(tiles * kIxMeanLongest, 0xffffffffu);
      gstat = stat;
      hipLaunchKernelGGL(sfa_fwd_ix_stat_zero_kernel, dim3(1), dim3(1), 0, stream, stat);
      hipLaunchKernelGGL((sfa_fwd_ix_prep_kernel<kIxD, kIxMaxK>), grid, block, 0, stream, k_idx,
                         k_val, vb, n, k, ifmt, vfmt, p.vtiles, wx, wf, stat);
    }
#define SFA_PREP(DD, KK)                                                                        \
  hipLaunchKernelGGL((sfa_fwd_prep_kernel<DD, KK>), grid, block, 0, stream, k_idx, k_val, vb, n, \
                     k, ifmt, vfmt, p.vtiles, wt, wf, gstat, p.ix_thresh, p.hb_count)
    if (d == 64) {
      if (p.kx == kValBF16) SFA_PREP(64, kValBF16);
      else if (p.kx == kValF16) SFA_PREP(64, kValF16);
      else SFA_PREP(64, 0);
    } else {
      if (p.kx == kValBF16) SFA_PREP(128, kValBF16);
      else if (p.kx == kValF16) SFA_PREP(128, kValF16);
      else SFA_PREP(128, 0);
    }
#undef SFA_PREP
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (d == 64) return vbf16 ? launch_t<64, true>(p, B, stream) : launch_t<64, false>(p, B, stream);
  return vbf16 ? launch_t<128, true>(p, B, stream) : launch_t<128, false>(p, B, stream);
}

}  // namespace sfa
