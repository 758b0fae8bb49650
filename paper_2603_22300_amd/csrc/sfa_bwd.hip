// SFA backward with the straight-through estimator (Sec. 3.1, Eq. (6)) on
// gfx950.
//
// With P the attention weights of the forward (recomputed from its LSE),
//   dV = P^T dO,  dP = dO V^T,  dS = P o (dP - D),  D_i = dO_i . O_i,
//   dQ~ = scale dS K~,  dK~ = scale dS^T Q~,
// and Eq. (6) makes the gradient of a query (key) coordinate that of its code
// value on the support and zero elsewhere: the outputs are dQ~ and dK~ read
// at the codes' coordinates (dq_val, dk_val), plus dV.  As in the forward,
// the products run on the matrix cores on densified codes; every operand is
// split into two bf16 pieces x = x0 + x1 and each product keeps the three
// terms a0 b0 + a0 b1 + a1 b0 (relative error ~2^-16 of sum |a b|), with
// float32 accumulation.  An operand stored in bf16 (V, dO, and the code
// values when they are bf16: CEX) has a zero low piece, so the products with
// that piece are left out; the sums are unchanged (they only added zeros).
//
// Kernels (all on the caller's stream):
//   sfa_bwd_qprep_kernel  per (batch, query head, 32-row tile): an image of
//       Q~ and dO as bf16 pieces, plus log2(e) * LSE and D for the 32 rows;
//   sfa_bwd_kprep_kernel  per (batch, KV head, 32-key tile): an image of K~
//       and V;
//   sfa_bwd_dq_kernel     query-parallel (like the forward): S^T = K~ Q~^T,
//       dP^T = V dO^T, dS^T, dQ~^T += K~^T dS^T over the allowed key tiles;
//   sfa_bwd_dkv_kernel    key-parallel: S = Q~ K~^T, dP = dO V^T, dS,
//       dV^T += dO^T P and dK~^T += Q~^T dS over the query tiles of every
//       query head of the KV head;
//   sfa_bwd_dkvf_kernel   both products from one S, P, dP, dS per tile pair
//       (d = 64, bf16 V and O, in place of the two above);
//   sfa_bwd_split_sum_kernel  under a token window with global tokens, the
//       sum of the partial dv, dk_val of key block 0, whose sweep over every
//       query tile is split over several work items.
// Every output element is owned by one wavefront (or, for a split block, by
// the sum kernel, which adds the parts in a fixed order): no atomics.  The tile
// images are copied global -> LDS with direct-to-LDS loads.  When the
// (batch, KV head) pairs split evenly over the 8 XCDs and there is no token
// window, the dq, dk and dv kernels run persistent grids whose workgroups on
// one XCD sweep the same tiles in step, so that each image comes from HBM
// about once per row of blocks.
#include <algorithm>
#include <type_traits>

#include "sfa_device.h"
#include "sfa_launch.h"

namespace sfa {
namespace {

constexpr int kT = 32;         // rows (queries or keys) per tile image
constexpr int kNW = 8;         // dk, dv: wavefronts per workgroup (two per SIMD)
constexpr int kNWQ = 8;        // dq: wavefronts per workgroup (two per SIMD)
constexpr float kLog2e = 1.44269504088896340736f;

// Tile images: 32 rows, each row the bf16 pieces of two arrays side by side,
// [Q~ piece 0 | Q~ piece 1 | dO pieces] in the query image and
// [K~ piece 0 | K~ piece 1 | V pieces] in the key image.  OEX / VEX: dO / V
// are stored in bf16, so their low pieces are zero and only the high piece
// is kept.  A row is a run of 16-byte chunks, padded by 64 bytes (a pitch of
// 16 or 48 banks modulo the 64 LDS banks), and chunk c of row r is stored at
// chunk c ^ ((r / 4) % 4).  The one layout then serves, free of LDS bank
// conflicts, both the row operands (16-byte reads, a row per lane) and the
// transposed operands (ds_read_b64_tr_b16: 8 bytes of a row per lane, four
// consecutive rows per 16 lanes): no transposed copy is stored.  The query
// image ends with log2(e) * LSE and D of its 32 rows.
template <int D, bool OEX = false, bool VEX = false>
struct Img {
  static constexpr int PO = OEX ? 1 : 2, PV = VEX ? 1 : 2;  // pieces kept of dO and V
  static constexpr int C2 = 2 * D / 8;                       // first chunk of dO / V in a row
  static constexpr int QRB = (2 + PO) * D * 2 + 64, KRB = (2 + PV) * D * 2 + 64;  // row pitches, bytes
  static_assert((QRB / 4) % 64 == 16 || (QRB / 4) % 64 == 48, "query rows: conflict-free pitch");
  static_assert((KRB / 4) % 64 == 16 || (KRB / 4) % 64 == 48, "key rows: conflict-free pitch");
  static constexpr int Q_L2 = kT * QRB, Q_D = Q_L2 + kT * 4;
  static constexpr int QB = (Q_D + kT * 4 + 1023) / 1024 * 1024;
  static constexpr int KB = (kT * KRB + 1023) / 1024 * 1024;
  static constexpr int NKB = D / 16, NDB = D / 32;
};

// Byte offset of bf16 column `col` of row r in an image of row pitch RB.
template <int RB>
__device__ __forceinline__ int img_pos(int r, int col) {
  return r * RB + 16 * ((col >> 3) ^ ((r >> 2) & 3)) + 2 * (col & 7);
}

struct BwdParams {
  const void* q_idx;
  const void* q_val;
  const void* k_idx;
  const void* k_val;
  const void* v;
  const void* o;
  const float* lse;
  const void* dout;
  float* dq;
  float* dk;
  float* dv;
  unsigned char* qimg;
  unsigned char* kimg;
  int Hq, Hkv, G, n, k, causal;
  int window, n_global;  // token pattern: |i - j| < window or a global token (window 0: none)
  int ifmt, vfmt, vbf16, obf16;
  int nt;    // tiles per head: ceil(n / 32)
  int BR;    // query positions per dq workgroup: 256 / G
  int nqb;   // dq workgroups per (batch, KV head)
  int lg;    // log2(G): the matrix-core kernels run power-of-two groups
  int nkb;   // dk / dv key blocks (256 keys) per (batch, KV head)
  int pr;    // persistent grid of the launch: workgroups per XCD (0: one workgroup per block)
  int pm;    // persistent grid of the launch: blocks per XCD
  // Token window with global tokens: key block 0 holds the global keys, which
  // every query sees, so its sweep is far longer than any other block's; it
  // is split over nsplit work items (1: no split), which write partial dv and
  // dk_val for the block's keys ([nsplit][B * Hkv][kSplitKeys][d] floats
  // each, dk_val rows k long) for sfa_bwd_split_sum_kernel to add up.
  int nsplit;
  int bhkv;  // B * Hkv
  float* part_dv;
  float* part_dk;
  float scale, c;  // c = scale * log2(e)
};

__device__ __forceinline__ void split2(float x, uint16_t& h, uint16_t& l) {
  const uint32_t hb = f32_to_bf16_rne(x);
  h = (uint16_t)hb;
  l = (uint16_t)f32_to_bf16_rne(x - bf16_bits_to_f32(hb));
}

// The same split for two values at once, packed: word 0 holds the high
// pieces of (x0, x1), word 1 the low pieces; the rounding to nearest-even is
// the hardware conversion (v_cvt_pk_bf16_f32), identical to split2 for
// finite values.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void split2_pair(float x0, float x1, uint32_t& hw, uint32_t& lw) {
  const f32x2 v = {x0, x1};
  hw = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
  const f32x2 r = {x0 - __uint_as_float(hw << 16), x1 - __uint_as_float(hw & 0xffff0000u)};
  lw = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, bf16x2));
}

__device__ __forceinline__ float load_f(const void* p, int64_t i, int bf16) {
  return bf16 ? bf16_bits_to_f32(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}

// c += a1 b0 + a0 b1 + a0 b0 (smaller terms first).  A1 / B1 false: that
// operand is exact in bf16 (its low piece is zero), so its term is skipped.
template <bool A1 = true, bool B1 = true>
__device__ __forceinline__ void mfma3(floatx16& c, const bf16x8 (&a)[2], const bf16x8 (&b)[2]) {
  if constexpr (A1) c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[0], c, 0, 0, 0);
  if constexpr (B1) c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], c, 0, 0, 0);
}

// Copy `bytes` (a multiple of 1 KB) global -> LDS, whole-wave 16-byte
// direct-to-LDS loads spread over the workgroup's waves.
template <int NW>
__device__ __forceinline__ void dma(const unsigned char* src, unsigned char* dst, int bytes, int wave,
                                    int lane) {
  for (int i = wave; i < bytes / 1024; i += NW)
    __builtin_amdgcn_global_load_lds(src + i * 1024 + lane * 16,
                                     (__attribute__((address_space(3))) void*)(dst + i * 1024), 16,
                                     0, 0);
}

__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0f70); }  // vmcnt(0)

constexpr int kQS = 3;  // query-image stages of the key-parallel kernels

// Split of key block 0's sweep under a token window with global tokens.
constexpr int kMaxSplit = 16;         // most work items sharing the sweep
constexpr int kSplitKeys = kNW * kT;  // keys of a split block (the fused kernel's 128 fit)

// Bytes of one part's partial dv and dk_val (dk_val rows are k <= d long).
inline size_t split_part_bytes(int bhkv, int d) {
  return (size_t)2 * bhkv * kSplitKeys * d * sizeof(float);
}

// vmcnt(N): at most N of this wave's loads outstanding.  Loads retire in issue
// order, so with N no larger than the number of copies this wave issued for
// the most recent image, every earlier image is complete.
template <int N>
__device__ __forceinline__ void wait_vm_n() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0f70 | N);
}

// Workgroup (x, y) of a grid (nx, nbh) -> (block, bh): workgroups go
// round-robin over the 8 XCDs, each with its own L2; with nbh a multiple of 8,
// XCD c runs the (batch, KV head) pairs congruent to c, so one L2 serves every
// workgroup of a head.
__device__ __forceinline__ void xcd_map(int nx, int& x, int& bh) {
  x = (int)blockIdx.x;
  bh = (int)blockIdx.y;
  if (gridDim.y % 8 == 0) {
    const int id = x + bh * nx;
    const int j = id >> 3;
    x = j % nx;
    bh = (id & 7) + 8 * (j / nx);
  }
}

// Per-lane byte offsets into a tile image of row pitch RB (see Img).
//   Row operand (B of 32x32x16): lane (l32, hh) reads row l32, columns
//   8 (c0 + 2 kb + hh) .. + 7 for a chunk c0 that is a multiple of 4:
//   row[kb & 1] + 16 (c0 + 4 (kb / 2)).
//   Transposed operand (A of 32x32x16, the image's rows as its k index in
//   the order of the MFMA output layout): lane (l32, hh) needs columns
//   8 c0 + l32 of rows 16 kk + 4 hh + (0..3) and 16 kk + 4 hh + 8 + (0..3).
//   A transposing read hands lane i of a 16-lane group element i % 4 of
//   the 8 bytes addressed by lane 4 e + i / 4 of the group, as its element
//   e; so lane j of group g addresses row 4 hh + j / 4 (+ 8), columns
//   8 c0 + 16 (g % 2) + 4 (j % 4) + (0..3): tr[0] / tr[1] + (16 kk) RB + 16 c0.
template <int RB>
struct LaneOff {
  int row[2], tr[2];
  __device__ __forceinline__ explicit LaneOff(int lane) {
    const int l32 = lane & 31, hh = lane >> 5, g = lane >> 4, j = lane & 15;
    row[0] = l32 * RB + 16 * (hh ^ ((l32 >> 2) & 3));
    row[1] = row[0] ^ 32;
    tr[0] = (4 * hh + (j >> 2)) * RB + 8 * (j & 1) + 16 * ((2 * (g & 1) + ((j >> 1) & 1)) ^ hh);
    tr[1] = (tr[0] ^ 32) + 8 * RB;
  }
};

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ i16x4 lds_read_tr(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}

// Transposed operand of 32 columns from chunk c0 on, rows from 16 kk on.
template <int RB>
__device__ __forceinline__ bf16x8 tr_operand(const unsigned char* img, const LaneOff<RB>& o, int kk,
                                             int c0) {
  const int off = 16 * kk * RB + 16 * c0;
  const i16x4 a = lds_read_tr(img + o.tr[0] + off);
  const i16x4 b = lds_read_tr(img + o.tr[1] + off);
  const u32x2 x = __builtin_bit_cast(u32x2, a), y = __builtin_bit_cast(u32x2, b);
  const u32x4 w = {x.x, x.y, y.x, y.y};
  return __builtin_bit_cast(bf16x8, w);
}

// Row operand: chunk c0 + 2 kb + hh of the lane's row.
template <int RB>
__device__ __forceinline__ bf16x8 row_operand(const unsigned char* img, const LaneOff<RB>& o, int kb,
                                              int c0) {
  return *(const bf16x8*)(img + o.row[kb & 1] + 16 * (c0 + 4 * (kb >> 1)));
}

// ---------------------------------------------------------------------------
// images
// ---------------------------------------------------------------------------

template <int D, bool OEX>
__global__ __launch_bounds__(256) void sfa_bwd_qprep_kernel(BwdParams p) {
  using I = Img<D, OEX>;
  constexpr int RB = I::QRB;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* img = smem;
  float* l2 = (float*)(smem + I::Q_L2);
  float* dd = (float*)(smem + I::Q_D);
  const int t = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;  // bh = b * Hq + hq
  const int n = p.n, k = p.k;
  const int64_t r0 = (int64_t)bh * n + (int64_t)t * kT;  // first row of the tile
  for (int i = tid; i < I::QB / 16; i += 256) ((uint4*)smem)[i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  for (int e = tid; e < kT * k; e += 256) {
    const int r = e / k;
    if (t * kT + r >= n) break;
    const int f = load_idx(p.q_idx, r0 * k + e, p.ifmt, D - 1);
    uint16_t h, l;
    split2(load_val(p.q_val, r0 * k + e, p.vfmt), h, l);
    *(uint16_t*)(img + img_pos<RB>(r, f)) = h;
    *(uint16_t*)(img + img_pos<RB>(r, D + f)) = l;
  }
  // dO pieces, and D = dO . O with 8 threads per row (fixed reduction order)
  {
    const int r = tid >> 3, part = tid & 7;
    const bool ok = t * kT + r < n;
    float acc = 0.f;
    for (int x = 0; x < D / 8; ++x) {
      const int dim = part * (D / 8) + x;
      float g = 0.f, o = 0.f;
      if (ok) {
        g = load_f(p.dout, (r0 + r) * D + dim, p.obf16);
        o = load_f(p.o, (r0 + r) * D + dim, p.obf16);
      }
      acc = fmaf(g, o, acc);
      uint16_t h, l;
      split2(g, h, l);
      *(uint16_t*)(img + img_pos<RB>(r, 2 * D + dim)) = h;
      if constexpr (!OEX) *(uint16_t*)(img + img_pos<RB>(r, 3 * D + dim)) = l;  // (bf16 dO: l = 0)
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    acc += __shfl_xor(acc, 4, 64);
    if (part == 0) {
      // rows past n: P = exp2(s c - inf) = 0 and D = 0, so they add nothing
      l2[r] = ok ? p.lse[r0 + r] * kLog2e : INFINITY;
      dd[r] = ok ? acc : 0.f;
    }
  }
  __syncthreads();
  uint4* dst = (uint4*)(p.qimg + ((int64_t)bh * p.nt + t) * I::QB);
  for (int i = tid; i < I::QB / 16; i += 256) dst[i] = ((const uint4*)smem)[i];
}

template <int D, bool VEX>
__global__ __launch_bounds__(256) void sfa_bwd_kprep_kernel(BwdParams p) {
  using I = Img<D, false, VEX>;
  constexpr int RB = I::KRB;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* img = smem;
  const int t = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;  // bh = b * Hkv + hkv
  const int n = p.n, k = p.k;
  const int64_t r0 = (int64_t)bh * n + (int64_t)t * kT;
  for (int i = tid; i < I::KB / 16; i += 256) ((uint4*)smem)[i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  for (int e = tid; e < kT * k; e += 256) {
    const int r = e / k;
    if (t * kT + r >= n) break;
    const int f = load_idx(p.k_idx, r0 * k + e, p.ifmt, D - 1);
    uint16_t h, l;
    split2(load_val(p.k_val, r0 * k + e, p.vfmt), h, l);
    *(uint16_t*)(img + img_pos<RB>(r, f)) = h;
    *(uint16_t*)(img + img_pos<RB>(r, D + f)) = l;
  }
  for (int e = tid; e < kT * D; e += 256) {
    const int r = e / D, dim = e - r * D;
    if (t * kT + r >= n) break;
    uint16_t h, l;
    split2(load_f(p.v, (r0 + r) * D + dim, p.vbf16), h, l);
    *(uint16_t*)(img + img_pos<RB>(r, 2 * D + dim)) = h;
    if constexpr (!VEX) *(uint16_t*)(img + img_pos<RB>(r, 3 * D + dim)) = l;  // (bf16 V: l = 0)
  }
  __syncthreads();
  uint4* dst = (uint4*)(p.kimg + ((int64_t)bh * p.nt + t) * I::KB);
  for (int i = tid; i < I::KB / 16; i += 256) dst[i] = ((const uint4*)smem)[i];
}

// Row operands (lane = row l32, columns 8 c0 + 16 kb + 8 hh ..) of the NP
// pieces from chunk c0 on, straight from an image in global memory (a piece
// not stored is zero); two per-lane offsets and immediate ones, as in LDS.
template <int D, int RB, int NP>
__device__ __forceinline__ void load_rows_b(const unsigned char* img, int c0, int lane,
                                            bf16x8 (&b)[2][D / 16]) {
  const LaneOff<RB> o(lane);
#pragma unroll
  for (int pc = 0; pc < 2; ++pc)
#pragma unroll
    for (int kb = 0; kb < D / 16; ++kb) b[pc][kb] = pc < NP ? row_operand(img, o, kb, c0 + pc * D / 8) : bf16x8{};
}

// ---------------------------------------------------------------------------
// dq: query-parallel
// ---------------------------------------------------------------------------

// VEX / OEX / CEX: V / dO / the code values are stored in bf16, so their
// low pieces are zero.
template <int D, bool VEX, bool OEX, bool CEX>
__global__ __launch_bounds__(kNWQ * 64) void sfa_bwd_dq_kernel(BwdParams p) {
  using I = Img<D, OEX, VEX>;
  constexpr int NKB = I::NKB, NDB = I::NDB, QRB = I::QRB, KRB = I::KRB, C2 = I::C2;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = p.n;
  const LaneOff<KRB> ko(lane);
  // Work items: (batch x KV head, block of BR positions), the longest causal
  // blocks first.  Persistent grid (p.pr > 0) as in the key-parallel kernels
  // below, with the key tiles swept upward on even rows and downward on odd
  // ones.
  for (int prow = 0;; ++prow) {
    int xb, bh;
    bool down = false;
    if (p.pr > 0) {
      const int w = (int)blockIdx.x >> 3;
      if (prow * p.pr >= p.pm) break;
      const int idx = prow * p.pr + ((prow & 1) ? p.pr - 1 - w : w);
      if (idx >= p.pm) continue;  // last row: the next one breaks
      xb = idx % p.nqb;
      bh = ((int)blockIdx.x & 7) + 8 * (idx / p.nqb);
      down = prow & 1;
    } else {
      if (prow > 0) break;
      xcd_map(p.nqb, xb, bh);
    }
    const int qb = p.nqb - 1 - xb;  // longest causal blocks first
    const int b = bh / p.Hkv, hkv = bh - b * p.Hkv;
    const int i0 = qb * p.BR;
    // wave: 32 consecutive positions of one query head (BR is a multiple of 32)
    const int hq = hkv * p.G + (wave * kT) / p.BR;
    const int pos0 = i0 + (wave * kT) % p.BR;
    const int my_i = pos0 + l32;
    const bool wave_ok = pos0 < n;
    const bool row_ok = my_i < n;
    const int wave_i_max = min(pos0 + kT - 1, n - 1);

    bf16x8 qB[2][NKB], dB[2][NKB];
    float L2 = INFINITY, Dq = 0.f;
    if (wave_ok) {
      const unsigned char* qimg = p.qimg + ((int64_t)(b * p.Hq + hq) * p.nt + pos0 / kT) * I::QB;
      load_rows_b<D, QRB, 2>(qimg, 0, lane, qB);
      load_rows_b<D, QRB, I::PO>(qimg, C2, lane, dB);
      L2 = ((const float*)(qimg + I::Q_L2))[l32];
      Dq = ((const float*)(qimg + I::Q_D))[l32];
    } else {
#pragma unroll
      for (int pc = 0; pc < 2; ++pc)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          qB[pc][kb] = bf16x8{};
          dB[pc][kb] = bf16x8{};
        }
    }
    floatx16 acc[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

    const int blk_last = min(n, i0 + p.BR) - 1;
    // Key tiles of the block: all up to the causal limit, or with a token
    // window (and no global row here) the global tiles [0, gt_end) and the
    // window tiles [wt_begin, nkt_all); the gap between them is skipped.
    const bool win = p.window > 0;
    int kend = p.causal ? blk_last + 1 : n;
    int gt_end = 0, wt_begin = 0;
    if (win && i0 >= p.n_global) {
      if (!p.causal) kend = min(n, blk_last + p.window);
      gt_end = (p.n_global + kT - 1) / kT;
      wt_begin = max(0, i0 - p.window + 1) / kT;
      if (wt_begin <= gt_end) gt_end = wt_begin = 0;  // no gap
    }
    const int nkt = gt_end + (kend + kT - 1) / kT - wt_begin;
    auto tile_at = [&](int t) {
      if (down) t = nkt - 1 - t;
      return t < gt_end ? t : wt_begin + (t - gt_end);
    };
    // a key tile from j0 on meets the window of some row of this wave
    auto in_window = [&](int j0) {
      return !win || j0 < p.n_global || pos0 < p.n_global ||
             (j0 + kT - 1 > pos0 - p.window && j0 < wave_i_max + p.window);
    };
    const unsigned char* kimg0 = p.kimg + (int64_t)bh * p.nt * I::KB;
    if (nkt > 0) dma<kNWQ>(kimg0 + (int64_t)tile_at(0) * I::KB, smem, I::KB, wave, lane);
    wait_vm();
    __syncthreads();
    for (int t = 0; t < nkt; ++t) {
      const int stage = t & 1;
      const int jt = tile_at(t);
      // reads through `cur`, the copy of the next tile through `nxt` (restrict:
      // no compiler wait on the copy before the reads)
      auto tile = [&](const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt) {
      if (t + 1 < nkt) dma<kNWQ>(kimg0 + (int64_t)tile_at(t + 1) * I::KB, nxt, I::KB, wave, lane);
      const int j0 = jt * kT;
      if (wave_ok && (!p.causal || wave_i_max >= j0) && in_window(j0)) {
        const unsigned char* K = cur;
        floatx16 s, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          bf16x8 a[2], v[2];
#pragma unroll
          for (int pc = 0; pc < 2; ++pc) {
            a[pc] = row_operand(K, ko, kb, pc * D / 8);
            v[pc] = pc < I::PV ? row_operand(K, ko, kb, C2 + pc * D / 8) : bf16x8{};
          }
          const bf16x8 qq[2] = {qB[0][kb], qB[1][kb]};
          const bf16x8 gg[2] = {dB[0][kb], dB[1][kb]};
          mfma3<!CEX, !CEX>(s, a, qq);   // S^T = K~ Q~^T   (keys x queries)
          mfma3<!VEX, !OEX>(dp, v, gg);  // dP^T = V dO^T
        }
        // dS^T = P^T o (dP^T - D); lane = query my_i, register r = key j0 + 8(r/4) + 4hh + r%4
        // every (row, key) pair of the tile allowed: no element mask (rows past
        // n have L2 = +inf, hence P = 0, either way)
        const bool wcut = win && j0 + kT > p.n_global && wave_i_max >= p.n_global &&
                          (pos0 < p.n_global || wave_i_max - j0 >= p.window ||
                           j0 + kT - 1 - pos0 >= p.window);
        const bool full = j0 + kT <= n && (!p.causal || j0 + kT - 1 <= pos0) && !wcut;
        u32x4 dsw[2][2];  // [kk][piece], as bf16 pairs
        // one straight-line body per case (FULL: no element mask), chosen once
        // per tile: a mask test per element would become a branch per element
        auto ds_tile = [&](auto full_c) {
          constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
          for (int r = 0; r < 16; r += 2) {
            float ds[2];
#pragma unroll
            for (int x = 0; x < 2; ++x) {
              float pr = __builtin_amdgcn_exp2f(fmaf(s[r + x], p.c, -L2));
              if constexpr (!FULL) {
                const int j = j0 + 8 * ((r + x) >> 2) + 4 * hh + ((r + x) & 3);
                const bool ok = row_ok && j < n && (!p.causal || j <= my_i) &&
                                (!win || abs(my_i - j) < p.window || j < p.n_global || my_i < p.n_global);
                pr = ok ? pr : 0.f;
              }
              ds[x] = pr * (dp[r + x] - Dq);
            }
            uint32_t hw, lw;
            split2_pair(ds[0], ds[1], hw, lw);
            dsw[r >> 3][0][(r & 7) >> 1] = hw;
            dsw[r >> 3][1][(r & 7) >> 1] = lw;
          }
        };
        if (full) ds_tile(std::true_type{});
        else ds_tile(std::false_type{});
        bf16x8 dsb[2][2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int pc = 0; pc < 2; ++pc) dsb[kk][pc] = __builtin_bit_cast(bf16x8, dsw[kk][pc]);
        // dQ~^T += K~^T dS^T   (coordinates x queries)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const bf16x8 a[2] = {tr_operand(K, ko, kk, 4 * db), tr_operand(K, ko, kk, D / 8 + 4 * db)};
            mfma3<!CEX, true>(acc[db], a, dsb[kk]);
          }
        }
      }
      };
      tile(smem + stage * I::KB, smem + (stage ^ 1) * I::KB);
      wait_vm();
      __syncthreads();
    }

    // dq_val = scale * dQ~ at the row's support: stage dQ~ through LDS
    // (the key stages are free now), four waves at a time:
    // [wave % 4][query][coordinate], pitch D + 4.
    float* L = (float*)smem + (wave & 3) * kT * (D + 4);
#pragma unroll
    for (int round = 0; round < kNWQ / 4; ++round) {
      if (wave / 4 == round) {
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            L[l32 * (D + 4) + db * 32 + 8 * (r >> 2) + 4 * hh + (r & 3)] = acc[db][r];
      }
      __syncthreads();
      if (wave / 4 == round && row_ok) {
        const int64_t row = ((int64_t)b * p.Hq + hq) * n + my_i;
        for (int t = hh; t < p.k; t += 2) {
          const int u = load_idx(p.q_idx, row * p.k + t, p.ifmt, D - 1);
          p.dq[row * p.k + t] = p.scale * L[l32 * (D + 4) + u];
        }
      }
      __syncthreads();
    }
  }  // work items
}

// ---------------------------------------------------------------------------
// dk, dv: key-parallel, one kernel each
// ---------------------------------------------------------------------------
// PART kDV: S, P, dV^T += dO^T P.   PART kDK: S, dP, dS, dK~^T += Q~^T dS.
// Split in two so that each fits two wavefronts per SIMD (256 VGPRs); both
// recompute S.
constexpr int kDV = 0, kDK = 1;

template <int D, bool VEX, bool OEX, bool CEX, int PART>
__global__ __launch_bounds__(kNW * 64) void sfa_bwd_dkv_kernel(BwdParams p) {
  using I = Img<D, OEX, VEX>;
  constexpr int NKB = I::NKB, NDB = I::NDB, QRB = I::QRB, KRB = I::KRB, C2 = I::C2, QB = I::QB;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = p.n;
  const LaneOff<QRB> qo(lane);
  // Work items: (batch x KV head, block of 256 keys).  Without the persistent
  // grid a workgroup runs one item, placed by xcd_map.  With it (p.pr > 0,
  // B * Hkv a multiple of 8) the grid is 8 x pr workgroups, all resident:
  // workgroup id runs on XCD id & 7 (round-robin dispatch) in slot id >> 3,
  // and XCD c takes the KV heads congruent to c, their blocks in rows of pr,
  // slots reversed on every other row, query tiles swept downward on even
  // rows and upward on odd ones.  Under causal masking a block's sweep
  // shortens as its first key grows; with this order the workgroups of an
  // XCD start each row together or end it together, and in between stay on
  // the same query tile, so one L2 fetch of an image serves all of them.
  // With p.nsplit > 1 (one workgroup per block only) the first p.nsplit
  // items of a head are the parts of key block 0's sweep.
  for (int prow = 0;; ++prow) {
    int xb, bh, seg = 0;
    bool up = false;
    if (p.pr > 0) {
      const int w = (int)blockIdx.x >> 3;
      if (prow * p.pr >= p.pm) break;
      const int idx = prow * p.pr + ((prow & 1) ? p.pr - 1 - w : w);
      if (idx >= p.pm) continue;  // last row: the next one breaks
      xb = idx % p.nkb;
      bh = ((int)blockIdx.x & 7) + 8 * (idx / p.nkb);
      up = prow & 1;
    } else {
      if (prow > 0) break;
      xcd_map((int)gridDim.x, xb, bh);
      seg = xb < p.nsplit ? xb : 0;
      xb = xb < p.nsplit ? 0 : xb - p.nsplit + 1;
    }
    const bool part = p.nsplit > 1 && xb == 0;  // a part of block 0's sweep: partial results
    const int b = bh / p.Hkv, hkv = bh - b * p.Hkv;
    const int j0b = xb * (kNW * kT);  // most key tiles first: smallest j0 first
    const int jw0 = j0b + wave * kT;
    const int my_j = jw0 + l32;
    const bool wave_ok = jw0 < n;
    const bool key_ok = my_j < n;

    bf16x8 kB[2][NKB], vB[2][NKB];
    if (wave_ok) {
      const unsigned char* kimg = p.kimg + ((int64_t)bh * p.nt + jw0 / kT) * I::KB;
      load_rows_b<D, KRB, 2>(kimg, 0, lane, kB);
      if constexpr (PART == kDK) load_rows_b<D, KRB, I::PV>(kimg, C2, lane, vB);
    } else {
#pragma unroll
      for (int pc = 0; pc < 2; ++pc)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          kB[pc][kb] = bf16x8{};
          vB[pc][kb] = bf16x8{};
        }
    }
    floatx16 acc[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

    // Query tiles of all G heads that see some key of the block, the G heads
    // of a tile together, in the downward order: the range [t_lo, t_hi] from
    // the highest tile, then (non-causal window) the global query tiles below
    // it, [0, gq_end).  Without a window t_hi is the last tile.  `up` runs
    // the same order backwards.
    const bool win = p.window > 0;
    int t_lo = p.causal ? j0b / kT : 0, t_hi = p.nt - 1, gq_end = 0;
    if (win && j0b >= p.n_global) {
      const int jlast = min(n, j0b + kNW * kT) - 1;
      t_hi = min(p.nt - 1, (jlast + p.window - 1) / kT);
      if (!p.causal) {
        t_lo = max(0, j0b - p.window + 1) / kT;
        gq_end = min(t_lo, (p.n_global + kT - 1) / kT);
      }
    }
    const int nrange = t_hi - t_lo + 1;
    const int total = p.G * (nrange + gq_end);
    // this item's steps of the sweep: [it_lo, it_lo + cnt)
    const int it_lo = part ? (int)((int64_t)total * seg / p.nsplit) : 0;
    const int cnt = part ? (int)((int64_t)total * (seg + 1) / p.nsplit) - it_lo : total;
    // step it of the item -> position in the downward order
    auto ord = [&](int it) { return up ? total - 1 - (it_lo + it) : it_lo + it; };
    auto tile_of = [&](int it) {
      const int x = ord(it) >> p.lg;
      return x < nrange ? t_hi - x : gq_end - 1 - (x - nrange);
    };
    // a query tile from q0 on meets the window of some key of this wave
    auto in_window = [&](int q0) {
      return !win || q0 < p.n_global || jw0 < p.n_global ||
             (q0 < jw0 + kT - 1 + p.window && q0 + kT - 1 > jw0 - p.window);
    };
    auto qimg_of = [&](int it) {
      return p.qimg + ((int64_t)(b * p.Hq + hkv * p.G + (ord(it) & (p.G - 1))) * p.nt + tile_of(it)) * QB;
    };
    // three stages: the image two tiles ahead is in flight while a tile is
    // consumed (vmcnt waits only for the one needed next)
    // every wave copies at least QB / 1024 / kNW blocks of an image
    constexpr int kMinCopies = QB / 1024 / kNW;
    if (cnt > 0) dma<kNW>(qimg_of(0), smem, QB, wave, lane);
    if (cnt > 1) dma<kNW>(qimg_of(1), smem + QB, QB, wave, lane);
    if (cnt > 1) wait_vm_n<kMinCopies>(); else wait_vm();
    __syncthreads();
    for (int it = 0; it < cnt; ++it) {
      // The tile's LDS reads go through `cur` and the copy two tiles ahead
      // through `nxt`, both restrict: the compiler then knows the copy cannot
      // alias those reads and does not wait for it before them.
      auto tile = [&](const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt) {
      if (it + 2 < cnt) dma<kNW>(qimg_of(it + 2), nxt, QB, wave, lane);
      const int q0 = tile_of(it) * kT;
      if (wave_ok && (!p.causal || q0 + kT - 1 >= jw0) && in_window(q0)) {
        const unsigned char* Q = cur;
        const float* l2 = (const float*)(Q + I::Q_L2);
        const float* dd = (const float*)(Q + I::Q_D);
        floatx16 s, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          bf16x8 a[2];
#pragma unroll
          for (int pc = 0; pc < 2; ++pc) a[pc] = row_operand(Q, qo, kb, pc * D / 8);
          const bf16x8 kk2[2] = {kB[0][kb], kB[1][kb]};
          mfma3<!CEX, !CEX>(s, a, kk2);  // S = Q~ K~^T   (queries x keys)
          if constexpr (PART == kDK) {
            bf16x8 g[2];
#pragma unroll
            for (int pc = 0; pc < 2; ++pc)
              g[pc] = pc < I::PO ? row_operand(Q, qo, kb, C2 + pc * D / 8) : bf16x8{};
            const bf16x8 vv2[2] = {vB[0][kb], vB[1][kb]};
            mfma3<!OEX, !VEX>(dp, g, vv2);  // dP = dO V^T
          }
        }
        // lane = key my_j; register r = query row q0 + 8(r/4) + 4hh + r%4
        // every (query, key) pair of the tile allowed: no element mask (queries
        // past n have L2 = +inf, hence P = 0, either way)
        const bool wcut = win && q0 + kT > p.n_global && jw0 + kT > p.n_global &&
                          (q0 < p.n_global || jw0 < p.n_global || q0 + kT - 1 - jw0 >= p.window ||
                           jw0 + kT - 1 - q0 >= p.window);
        const bool full = jw0 + kT <= n && (!p.causal || q0 >= jw0 + kT - 1) && !wcut;
        u32x4 xw[2][2];  // [kk][piece]: P (dV) or dS (dK), as bf16 pairs
        // one straight-line body per case (FULL: no element mask), chosen once
        // per tile
        auto px_tile = [&](auto full_c) {
        constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const float4 l4 = *(const float4*)(l2 + 8 * g4 + 4 * hh);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
          float dv4[4] = {0.f, 0.f, 0.f, 0.f};
          if constexpr (PART == kDK) {
            const float4 d4 = *(const float4*)(dd + 8 * g4 + 4 * hh);
            dv4[0] = d4.x; dv4[1] = d4.y; dv4[2] = d4.z; dv4[3] = d4.w;
          }
          float val[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            const int r = 4 * g4 + x;
            float pr = __builtin_amdgcn_exp2f(fmaf(s[r], p.c, -lv[x]));
            if constexpr (!FULL) {
              const int i = q0 + 8 * g4 + 4 * hh + x;
              const bool ok = key_ok && (!p.causal || i >= my_j) &&
                              (!win || abs(i - my_j) < p.window || i < p.n_global || my_j < p.n_global);
              pr = ok ? pr : 0.f;
            }
            val[x] = PART == kDV ? pr : pr * (dp[r] - dv4[x]);
          }
#pragma unroll
          for (int x = 0; x < 4; x += 2) {
            const int r = 4 * g4 + x;
            uint32_t hw, lw;
            split2_pair(val[x], val[x + 1], hw, lw);
            xw[r >> 3][0][(r & 7) >> 1] = hw;
            xw[r >> 3][1][(r & 7) >> 1] = lw;
          }
        }
        };
        if (full) px_tile(std::true_type{});
        else px_tile(std::false_type{});
        bf16x8 xb[2][2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int pc = 0; pc < 2; ++pc) xb[kk][pc] = __builtin_bit_cast(bf16x8, xw[kk][pc]);
        // dV^T += dO^T P  or  dK~^T += Q~^T dS   (dimensions / coordinates x keys)
        constexpr int ca = PART == kDV ? C2 : 0;  // dO or Q~
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            // (dO^T with bf16 dO: the high piece only)
            const bool lo = PART == kDK || I::PO == 2;
            const bf16x8 at[2] = {tr_operand(Q, qo, kk, ca + 4 * db),
                                  lo ? tr_operand(Q, qo, kk, ca + D / 8 + 4 * db) : bf16x8{}};
            if constexpr (PART == kDV) mfma3<!OEX, true>(acc[db], at, xb[kk]);
            else mfma3<!CEX, true>(acc[db], at, xb[kk]);
          }
        }
      }
      };
      tile(smem + (it % kQS) * QB, smem + ((it + 2) % kQS) * QB);
      // the next tile's copies must be complete; the one after may still run
      if (it + 2 < cnt) wait_vm_n<kMinCopies>(); else wait_vm();
      __syncthreads();
    }

    if constexpr (PART == kDV) {
      // dv: lane = key my_j, register r of block db = dimension db*32 + 8(r/4) + 4hh + r%4
      if (key_ok) {
        float* dvr = part ? p.part_dv + (((int64_t)seg * p.bhkv + bh) * kSplitKeys + my_j) * D
                          : p.dv + ((int64_t)bh * n + my_j) * D;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4)
            *(float4*)(dvr + db * 32 + 8 * g4 + 4 * hh) =
                make_float4(acc[db][4 * g4], acc[db][4 * g4 + 1], acc[db][4 * g4 + 2], acc[db][4 * g4 + 3]);
      }
    } else {
      // dk_val = scale * dK~ at the key's support, through LDS, four waves at
      // a time: [wave % 4][key][coordinate], pitch D + 4
      float* L = (float*)smem + (wave & 3) * kT * (D + 4);
#pragma unroll
      for (int round = 0; round < kNW / 4; ++round) {
        if (wave / 4 == round) {
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              L[l32 * (D + 4) + db * 32 + 8 * (r >> 2) + 4 * hh + (r & 3)] = acc[db][r];
        }
        __syncthreads();
        if (wave / 4 == round && key_ok) {
          const int64_t row = (int64_t)bh * n + my_j;
          float* dkr = part ? p.part_dk + (((int64_t)seg * p.bhkv + bh) * kSplitKeys + my_j) * p.k
                            : p.dk + row * p.k;
          for (int t = hh; t < p.k; t += 2) {
            const int u = load_idx(p.k_idx, row * p.k + t, p.ifmt, D - 1);
            dkr[t] = p.scale * L[l32 * (D + 4) + u];
          }
        }
        __syncthreads();
      }
    }
  }  // work items
}

// ---------------------------------------------------------------------------
// dk and dv fused: key-parallel, with S, P, dP and dS computed once per
// (query tile, key tile) for both products (72 MFMAs per 32 x 32 tile pair
// with 32-bit codes and bf16 V / dO at d = 128, against 96 in the two
// kernels above).  A wave's state (K~ and V operands of its 32 keys, the dV
// and dK~ accumulators) takes more registers than two waves per SIMD allow,
// so a workgroup is four waves over 128 keys, at one or two waves per SIMD.
// LDS holds two stages of the whole query image.  Used at d = 64 with bf16 V
// and O (gpt2s shape: 0.46 -> 0.38 ms per backward); at d = 128 the single
// wave per SIMD leaves the dependency chain of a tile (S -> P -> dV, dK)
// exposed and the two kernels above are faster (66.8 against 82.5 ms on
// qwen3_32k).
// ---------------------------------------------------------------------------
constexpr int kNWF = 4;
static_assert(kNWF * kT <= kSplitKeys, "a split fused block fits the partial results");

template <int D, bool VEX, bool OEX>
constexpr bool fused_dkv() { return D == 64 && VEX && OEX; }

template <int D, bool VEX, bool OEX, bool CEX>
__global__ __launch_bounds__(kNWF * 64) void sfa_bwd_dkvf_kernel(BwdParams p) {
  using I = Img<D, OEX, VEX>;
  constexpr int NKB = I::NKB, NDB = I::NDB, QRB = I::QRB, KRB = I::KRB, C2 = I::C2, QB = I::QB;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = p.n;
  const LaneOff<QRB> qo(lane);
  int xb, bh;
  xcd_map((int)gridDim.x, xb, bh);
  // the first p.nsplit items of a head are the parts of key block 0's sweep
  const int seg = xb < p.nsplit ? xb : 0;
  xb = xb < p.nsplit ? 0 : xb - p.nsplit + 1;
  const bool part = p.nsplit > 1 && xb == 0;  // partial results
  const int b = bh / p.Hkv, hkv = bh - b * p.Hkv;
  const int j0b = xb * (kNWF * kT);  // most query tiles first: smallest j0 first
  const int jw0 = j0b + wave * kT;
  const int my_j = jw0 + l32;
  const bool wave_ok = jw0 < n;
  const bool key_ok = my_j < n;

  bf16x8 kB[2][NKB], vB[2][NKB];
  if (wave_ok) {
    const unsigned char* kimg = p.kimg + ((int64_t)bh * p.nt + jw0 / kT) * I::KB;
    load_rows_b<D, KRB, 2>(kimg, 0, lane, kB);
    load_rows_b<D, KRB, I::PV>(kimg, C2, lane, vB);
  } else {
#pragma unroll
    for (int pc = 0; pc < 2; ++pc)
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        kB[pc][kb] = bf16x8{};
        vB[pc][kb] = bf16x8{};
      }
  }
  floatx16 accV[NDB], accK[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      accV[db][r] = 0.f;
      accK[db][r] = 0.f;
    }

  // query tiles that see a key of the block, swept from the highest down,
  // the G heads of a tile together (as in sfa_bwd_dkv_kernel)
  const bool win = p.window > 0;
  int t_lo = p.causal ? j0b / kT : 0, t_hi = p.nt - 1, gq_end = 0;
  if (win && j0b >= p.n_global) {
    const int jlast = min(n, j0b + kNWF * kT) - 1;
    t_hi = min(p.nt - 1, (jlast + p.window - 1) / kT);
    if (!p.causal) {
      t_lo = max(0, j0b - p.window + 1) / kT;
      gq_end = min(t_lo, (p.n_global + kT - 1) / kT);
    }
  }
  const int nrange = t_hi - t_lo + 1;
  const int total = p.G * (nrange + gq_end);
  // this item's steps of the sweep: [it_lo, it_lo + cnt)
  const int it_lo = part ? (int)((int64_t)total * seg / p.nsplit) : 0;
  const int cnt = part ? (int)((int64_t)total * (seg + 1) / p.nsplit) - it_lo : total;
  auto tile_of = [&](int it) {
    const int x = (it_lo + it) >> p.lg;
    return x < nrange ? t_hi - x : gq_end - 1 - (x - nrange);
  };
  auto in_window = [&](int q0) {
    return !win || q0 < p.n_global || jw0 < p.n_global ||
           (q0 < jw0 + kT - 1 + p.window && q0 + kT - 1 > jw0 - p.window);
  };
  auto qimg_of = [&](int it) {
    return p.qimg + ((int64_t)(b * p.Hq + hkv * p.G + ((it_lo + it) & (p.G - 1))) * p.nt + tile_of(it)) * QB;
  };
  if (cnt > 0) dma<kNWF>(qimg_of(0), smem, QB, wave, lane);
  wait_vm();
  __syncthreads();
  for (int it = 0; it < cnt; ++it) {
    // reads through `cur`, the copy of the next image through `nxt`
    auto tile = [&](const unsigned char* __restrict__ cur, unsigned char* __restrict__ nxt) {
    if (it + 1 < cnt) dma<kNWF>(qimg_of(it + 1), nxt, QB, wave, lane);
    const int q0 = tile_of(it) * kT;
    if (wave_ok && (!p.causal || q0 + kT - 1 >= jw0) && in_window(q0)) {
      const float* l2 = (const float*)(cur + I::Q_L2);
      const float* dd = (const float*)(cur + I::Q_D);
      floatx16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        bf16x8 a[2], g[2];
#pragma unroll
        for (int pc = 0; pc < 2; ++pc) {
          a[pc] = row_operand(cur, qo, kb, pc * D / 8);
          g[pc] = pc < I::PO ? row_operand(cur, qo, kb, C2 + pc * D / 8) : bf16x8{};
        }
        const bf16x8 kk2[2] = {kB[0][kb], kB[1][kb]};
        const bf16x8 vv2[2] = {vB[0][kb], vB[1][kb]};
        mfma3<!CEX, !CEX>(s, a, kk2);   // S = Q~ K~^T   (queries x keys)
        mfma3<!OEX, !VEX>(dp, g, vv2);  // dP = dO V^T
      }
      // lane = key my_j; register r = query row q0 + 8(r/4) + 4hh + r%4.
      // Every (query, key) pair of a full tile is allowed: no element mask
      // (queries past n have L2 = +inf, hence P = 0, either way).
      const bool wcut = win && q0 + kT > p.n_global && jw0 + kT > p.n_global &&
                        (q0 < p.n_global || jw0 < p.n_global || q0 + kT - 1 - jw0 >= p.window ||
                         jw0 + kT - 1 - q0 >= p.window);
      const bool full = jw0 + kT <= n && (!p.causal || q0 >= jw0 + kT - 1) && !wcut;
      u32x4 pw[2][2], sw[2][2];  // [kk][piece]: P and dS as bf16 pairs
      // (one body with the mask test per element: the two-body form of the
      // kernels above costs this kernel its second wave per SIMD)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const float4 l4 = *(const float4*)(l2 + 8 * g4 + 4 * hh);
        const float4 d4 = *(const float4*)(dd + 8 * g4 + 4 * hh);
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
        const float dv4[4] = {d4.x, d4.y, d4.z, d4.w};
        float pv[4], sv[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const int r = 4 * g4 + x;
          const int i = q0 + 8 * g4 + 4 * hh + x;
          float pr;
          if (full) {
            pr = __builtin_amdgcn_exp2f(fmaf(s[r], p.c, -lv[x]));
          } else {
            const bool ok = key_ok && (!p.causal || i >= my_j) &&
                            (!win || abs(i - my_j) < p.window || i < p.n_global || my_j < p.n_global);
            pr = ok ? __builtin_amdgcn_exp2f(fmaf(s[r], p.c, -lv[x])) : 0.f;
          }
          pv[x] = pr;
          sv[x] = pr * (dp[r] - dv4[x]);
        }
#pragma unroll
        for (int x = 0; x < 4; x += 2) {
          const int r = 4 * g4 + x;
          uint32_t hw, lw;
          split2_pair(pv[x], pv[x + 1], hw, lw);
          pw[r >> 3][0][(r & 7) >> 1] = hw;
          pw[r >> 3][1][(r & 7) >> 1] = lw;
          split2_pair(sv[x], sv[x + 1], hw, lw);
          sw[r >> 3][0][(r & 7) >> 1] = hw;
          sw[r >> 3][1][(r & 7) >> 1] = lw;
        }
      }
      // dV^T += dO^T P  and  dK~^T += Q~^T dS   (dimensions / coordinates x keys)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 pb[2] = {__builtin_bit_cast(bf16x8, pw[kk][0]), __builtin_bit_cast(bf16x8, pw[kk][1])};
        const bf16x8 sb[2] = {__builtin_bit_cast(bf16x8, sw[kk][0]), __builtin_bit_cast(bf16x8, sw[kk][1])};
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8 ao[2] = {tr_operand(cur, qo, kk, C2 + 4 * db),
                                I::PO == 2 ? tr_operand(cur, qo, kk, C2 + D / 8 + 4 * db) : bf16x8{}};
          mfma3<!OEX, true>(accV[db], ao, pb);
          const bf16x8 aq[2] = {tr_operand(cur, qo, kk, 4 * db), tr_operand(cur, qo, kk, D / 8 + 4 * db)};
          mfma3<!CEX, true>(accK[db], aq, sb);
        }
      }
    }
    };
    tile(smem + (it & 1) * QB, smem + ((it + 1) & 1) * QB);
    wait_vm();  // the next image has landed
    __syncthreads();
  }

  // dv: lane = key my_j, register r of block db = dimension db*32 + 8(r/4) + 4hh + r%4
  if (key_ok) {
    float* dvr = part ? p.part_dv + (((int64_t)seg * p.bhkv + bh) * kSplitKeys + my_j) * D
                      : p.dv + ((int64_t)bh * n + my_j) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *(float4*)(dvr + db * 32 + 8 * g4 + 4 * hh) =
            make_float4(accV[db][4 * g4], accV[db][4 * g4 + 1], accV[db][4 * g4 + 2], accV[db][4 * g4 + 3]);
  }
  // dk_val = scale * dK~ at the key's support, through LDS (the stages are
  // free): [wave][key][coordinate], pitch D + 4
  float* L = (float*)smem + wave * kT * (D + 4);
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      L[l32 * (D + 4) + db * 32 + 8 * (r >> 2) + 4 * hh + (r & 3)] = accK[db][r];
  __syncthreads();
  if (key_ok) {
    const int64_t row = (int64_t)bh * n + my_j;
    float* dkr = part ? p.part_dk + (((int64_t)seg * p.bhkv + bh) * kSplitKeys + my_j) * p.k
                      : p.dk + row * p.k;
    for (int t = hh; t < p.k; t += 2) {
      const int u = load_idx(p.k_idx, row * p.k + t, p.ifmt, D - 1);
      dkr[t] = p.scale * L[l32 * (D + 4) + u];
    }
  }
}

// Workspace bytes of the tile images in the largest layout (float32 dO and V).
inline size_t bwd_image_bytes(int B, int Hq, int Hkv, int n, int d) {
  const size_t nt = (size_t)((n + kT - 1) / kT);
  const size_t qb = d == 64 ? Img<64>::QB : Img<128>::QB;
  const size_t kb = d == 64 ? Img<64>::KB : Img<128>::KB;
  return (size_t)B * Hq * nt * qb + (size_t)B * Hkv * nt * kb;
}

// Parts a split sweep may use for these sizes: at most kMaxSplit, with their
// partial results at most 1/8 of the tile images' bytes (short sequences
// would otherwise pay more for them than for the images); 0 (no split) when
// fewer than two fit.  The workspace holds this many parts' results.
inline int split_parts_max(int B, int Hq, int Hkv, int n, int d) {
  const size_t m = bwd_image_bytes(B, Hq, Hkv, n, d) / 8 / split_part_bytes(B * Hkv, d);
  return m >= 2 ? (int)std::min<size_t>(m, kMaxSplit) : 0;
}

// dv and dk_val of key block 0's keys after a split sweep: the sum of the
// parts' partial results, in part order (the same on every run).  Workgroup
// (x, bh) takes keys 16 x .. 16 x + 15 of head bh.
__global__ __launch_bounds__(256) void sfa_bwd_split_sum_kernel(BwdParams p, int D) {
  const int bh = blockIdx.y, j0 = blockIdx.x * 16;
  const int nk = min(16, p.n - j0);
  if (nk <= 0) return;
  const size_t ps = (size_t)p.bhkv * kSplitKeys;  // keys between two parts
  for (int e = threadIdx.x; e < nk * D; e += 256) {
    const int j = j0 + e / D, c = e % D;
    const float* src = p.part_dv + ((size_t)bh * kSplitKeys + j) * D + c;
    float acc = 0.f;
    for (int sg = 0; sg < p.nsplit; ++sg) acc += src[sg * ps * D];
    p.dv[((int64_t)bh * p.n + j) * D + c] = acc;
  }
  for (int e = threadIdx.x; e < nk * p.k; e += 256) {
    const int j = j0 + e / p.k, t = e % p.k;
    const float* src = p.part_dk + ((size_t)bh * kSplitKeys + j) * p.k + t;
    float acc = 0.f;
    for (int sg = 0; sg < p.nsplit; ++sg) acc += src[sg * ps * p.k];
    p.dk[((int64_t)bh * p.n + j) * p.k + t] = acc;
  }
}

template <int D, bool VEX, bool OEX, bool CEX>
hipError_t launch_d(BwdParams p, int B, hipStream_t stream) {
  using I = Img<D, OEX, VEX>;
  // LDS of the dq kernel (two key-image stages, or the gather of dQ~ that
  // follows, four waves at a time) and of the fused dk / dv kernel (two
  // query-image stages, or its gather)
  constexpr int kDqLds = std::max(2 * I::KB, 4 * kT * (D + 4) * 4);
  constexpr int kFLds = std::max(2 * I::QB, kNWF * kT * (D + 4) * 4);
  // once per instantiation (a function-local static: initialised once, also
  // under concurrent first calls): kernel attributes, and the resident
  // workgroups per XCD of the persistent grids (per CU x CUs / 8)
  struct Cfg {
    hipError_t e;
    int res_dq, res_dv, res_dk;
  };
  static const Cfg cfg = [] {
    Cfg c{hipSuccess, 0, 0, 0};
    hipError_t& e = c.e;
    const void* fns[5] = {(const void*)sfa_bwd_qprep_kernel<D, OEX>, (const void*)sfa_bwd_kprep_kernel<D, VEX>,
                          (const void*)sfa_bwd_dq_kernel<D, VEX, OEX, CEX>,
                          (const void*)sfa_bwd_dkv_kernel<D, VEX, OEX, CEX, kDV>,
                          (const void*)sfa_bwd_dkv_kernel<D, VEX, OEX, CEX, kDK>};
    const int bytes[5] = {I::QB, I::KB, kDqLds, kQS * I::QB, kQS * I::QB};
    for (int f = 0; f < 5 && e == hipSuccess; ++f)
      if (bytes[f] > 65536) e = hipFuncSetAttribute(fns[f], hipFuncAttributeMaxDynamicSharedMemorySize, bytes[f]);
    if constexpr (fused_dkv<D, VEX, OEX>()) {
      if (e == hipSuccess && kFLds > 65536)
        e = hipFuncSetAttribute((const void*)sfa_bwd_dkvf_kernel<D, VEX, OEX, CEX>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, kFLds);
    }
    int dev = 0, cus = 0, nb_dq = 0, nb_dv = 0, nb_dk = 0;
    if (e == hipSuccess) e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &nb_dq, (const void*)sfa_bwd_dq_kernel<D, VEX, OEX, CEX>, kNWQ * 64, kDqLds);
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &nb_dv, (const void*)sfa_bwd_dkv_kernel<D, VEX, OEX, CEX, kDV>, kNW * 64, kQS * I::QB);
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &nb_dk, (const void*)sfa_bwd_dkv_kernel<D, VEX, OEX, CEX, kDK>, kNW * 64, kQS * I::QB);
    c.res_dq = nb_dq * cus / 8;
    c.res_dv = nb_dv * cus / 8;
    c.res_dk = nb_dk * cus / 8;
    return c;
  }();
  if (cfg.e != hipSuccess) return cfg.e;
  const int res_dq = cfg.res_dq, res_dv = cfg.res_dv, res_dk = cfg.res_dk;
  static_assert(kQS * I::QB >= 4 * kT * (D + 4) * 4, "dk gather (four waves at a time) fits the stages");
  static_assert(kQS * I::QB <= 160 * 1024 - 512, "the query-image stages fit LDS");
  static_assert(I::QB / 1024 / kNW >= 1, "each wave copies part of each image");
  // the key images follow the query images in the workspace, then the
  // partial results of a split block
  p.kimg = p.qimg + (size_t)B * p.Hq * p.nt * I::QB;
  const int parts = split_parts_max(B, p.Hq, p.Hkv, p.n, D);
  p.part_dv = (float*)(p.kimg + (size_t)B * p.Hkv * p.nt * I::KB);
  p.part_dk = p.part_dv + (size_t)parts * p.bhkv * kSplitKeys * D;
  // Under a token window with global tokens, key block 0 (which holds them)
  // sweeps every query tile, a windowed block about (its keys + the window)
  // / 32 of them (twice the window without causal masking): block 0's sweep
  // is split so that no part is much longer than a windowed block's.
  // (Blocks past the first that hold global keys, n_global > their first
  // key, keep their whole sweep.)
  p.nsplit = 1;
  if (p.window > 0 && p.n_global > 0 && parts >= 2) {
    const int keys = fused_dkv<D, VEX, OEX>() ? kNWF * kT : kNW * kT;
    const int typ = (keys + (p.causal ? 1 : 2) * p.window) / kT + 1;
    p.nsplit = std::min(parts, std::max(1, (p.nt + typ - 1) / typ));
  }
  const dim3 blk(256);
  hipLaunchKernelGGL((sfa_bwd_qprep_kernel<D, OEX>), dim3(p.nt, B * p.Hq), blk, I::QB, stream, p);
  hipLaunchKernelGGL((sfa_bwd_kprep_kernel<D, VEX>), dim3(p.nt, B * p.Hkv), blk, I::KB, stream, p);
  // persistent grids when the KV heads split evenly over the 8 XCDs
  // (not under a token window: there every block sweeps the same number of
  // tiles, and the one-workgroup-per-block grid measured faster)
  const bool pers = (B * p.Hkv) % 8 == 0 && p.window == 0;
  {
    BwdParams pq = p;
    pq.pm = B * p.Hkv / 8 * p.nqb;
    pq.pr = pers ? max(1, min(res_dq, pq.pm)) : 0;
    const dim3 gq = pers ? dim3(8 * pq.pr) : dim3(p.nqb, B * p.Hkv);
    hipLaunchKernelGGL((sfa_bwd_dq_kernel<D, VEX, OEX, CEX>), gq, dim3(kNWQ * 64), kDqLds, stream, pq);
  }
  static_assert(kFLds <= 160 * 1024, "fused dk/dv stages");
  if constexpr (fused_dkv<D, VEX, OEX>()) {
    const int nkf = (p.n + kNWF * kT - 1) / (kNWF * kT);
    hipLaunchKernelGGL((sfa_bwd_dkvf_kernel<D, VEX, OEX, CEX>), dim3(nkf + p.nsplit - 1, B * p.Hkv),
                       dim3(kNWF * 64), kFLds, stream, p);
    if (p.nsplit > 1)
      hipLaunchKernelGGL(sfa_bwd_split_sum_kernel, dim3(kNWF * kT / 16, B * p.Hkv), dim3(256), 0, stream, p, D);
    return hipGetLastError();
  }
  p.nkb = (p.n + kNW * kT - 1) / (kNW * kT);
  p.pm = B * p.Hkv / 8 * p.nkb;
  BwdParams pv = p, pk = p;
  pv.pr = pers ? max(1, min(res_dv, p.pm)) : 0;
  pk.pr = pers ? max(1, min(res_dk, p.pm)) : 0;
  // (a split sweep only with a token window, which has no persistent grid)
  const dim3 gv = pers ? dim3(8 * pv.pr) : dim3(p.nkb + p.nsplit - 1, B * p.Hkv);
  const dim3 gk = pers ? dim3(8 * pk.pr) : dim3(p.nkb + p.nsplit - 1, B * p.Hkv);
  hipLaunchKernelGGL((sfa_bwd_dkv_kernel<D, VEX, OEX, CEX, kDV>), gv, dim3(kNW * 64), kQS * I::QB,
                     stream, pv);
  hipLaunchKernelGGL((sfa_bwd_dkv_kernel<D, VEX, OEX, CEX, kDK>), gk, dim3(kNW * 64), kQS * I::QB,
                     stream, pk);
  if (p.nsplit > 1)
    hipLaunchKernelGGL(sfa_bwd_split_sum_kernel, dim3(kNW * kT / 16, B * p.Hkv), dim3(256), 0, stream, p, D);
  return hipGetLastError();
}

}  // namespace

// a dq wave's 32 rows must be one query head: G <= 8 (and <= 4 would do for dk/dv)
int bwd_max_group() { return kNWQ; }

size_t bwd_workspace_bytes(int B, int Hq, int Hkv, int n, int d) {
  return bwd_image_bytes(B, Hq, Hkv, n, d) +
         (size_t)split_parts_max(B, Hq, Hkv, n, d) * split_part_bytes(B * Hkv, d);
}

hipError_t launch_attn_bwd(const void* q_idx, const void* q_val, const void* k_idx,
                           const void* k_val, const void* v, const void* o, const float* lse,
                           const void* dout, int B, int Hq, int Hkv, int n, int d, int k,
                           int causal, int window, int n_global, float scale, int ifmt,
                           int vfmt, int vbf16, int obf16, float* dq, float* dk, float* dv,
                           void* ws, hipStream_t stream) {
  BwdParams p;
  p.q_idx = q_idx; p.q_val = q_val; p.k_idx = k_idx; p.k_val = k_val; p.v = v; p.o = o;
  p.lse = lse; p.dout = dout; p.dq = dq; p.dk = dk; p.dv = dv;
  p.Hq = Hq; p.Hkv = Hkv; p.G = Hq / Hkv; p.n = n; p.k = k; p.causal = causal;
  p.window = window; p.n_global = n_global;
  p.ifmt = ifmt; p.vfmt = vfmt; p.vbf16 = vbf16; p.obf16 = obf16;
  p.nt = (n + kT - 1) / kT;
  p.BR = kNWQ * kT / p.G;
  p.nqb = (n + p.BR - 1) / p.BR;
  p.lg = __builtin_ctz((unsigned)p.G);  // G is a power of two here (checked by the caller)
  p.nkb = p.pr = p.pm = 0;  // set by launch_d for the dk / dv kernels
  p.nsplit = 1;
  p.bhkv = B * Hkv;
  p.part_dv = p.part_dk = nullptr;  // set by launch_d
  p.scale = scale;
  p.c = (float)((double)scale * 1.4426950408889634);
  // (images of the bf16 dO / V layouts are smaller than the workspace's)
  p.qimg = (unsigned char*)ws;
  p.kimg = nullptr;  // set by launch_d
  // bf16 code values (exact in one bf16 piece) with bf16 V, O and dO
  const bool cex = vfmt == kValBF16 && vbf16 && obf16;
  if (d == 64) {
    if (cex) return launch_d<64, true, true, true>(p, B, stream);
    if (vbf16) return obf16 ? launch_d<64, true, true, false>(p, B, stream) : launch_d<64, true, false, false>(p, B, stream);
    return obf16 ? launch_d<64, false, true, false>(p, B, stream) : launch_d<64, false, false, false>(p, B, stream);
  }
  if (cex) return launch_d<128, true, true, true>(p, B, stream);
  if (vbf16) return obf16 ? launch_d<128, true, true, false>(p, B, stream) : launch_d<128, true, false, false>(p, B, stream);
  return obf16 ? launch_d<128, false, true, false>(p, B, stream) : launch_d<128, false, false, false>(p, B, stream);
}

}  // namespace sfa
