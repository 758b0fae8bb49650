// Device-side helpers shared by the SFA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sfa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLn2 = 0.69314718055994530942f;

// Number of set bits of `mask` held by lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t wave_ballot(bool p) {
  return __builtin_amdgcn_ballot_w64(p);
}

// float32 -> bfloat16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
  return __uint_as_float(b16 << 16);
}

// Exchange with the lane 32 positions away (the other half of the wave).
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, 64);
}

// Max / sum of x over lanes l and l ^ 32.  One v_permlane32_swap of x with
// itself leaves each lane holding x of both lanes (in an order that differs
// between the halves); max and + are symmetric, so both lanes get the same
// bits.  A VALU instruction, where swap_halves is an LDS permute.
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Unsigned maximum over the wavefront (all 64 lanes active), wave-uniform
// result.  DPP steps make
// every lane of a 16-lane row hold the row's maximum (quad swaps 1 and 2,
// then the half-row and row mirrors); the four row maxima are read by
// readlane and combined on the scalar unit.
__device__ __forceinline__ uint32_t wave_umax(uint32_t x) {
  x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xb1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
  x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4e, 0xf, 0xf, false));   // quad_perm 2,3,0,1
  x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x141, 0xf, 0xf, false));  // row_half_mirror
  x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xf, 0xf, false));  // row_mirror
  const uint32_t r0 = __builtin_amdgcn_readlane(x, 0), r1 = __builtin_amdgcn_readlane(x, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(x, 32), r3 = __builtin_amdgcn_readlane(x, 48);
  return max(max(r0, r1), max(r2, r3));
}

// Float maximum over the wavefront (all 64 lanes active), wave-uniform
// result, without LDS: the DPP steps of wave_umax make each 16-lane row hold
// its maximum, and the four row maxima are read by readlane.
template <int CTRL>
__device__ __forceinline__ float dpp_max_step(float v) {
  return fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v),
                                                             CTRL, 0xf, 0xf, false)));
}

__device__ __forceinline__ float wave_max_dpp(float x) {
  x = dpp_max_step<0xb1>(x);   // quad_perm 1,0,3,2
  x = dpp_max_step<0x4e>(x);   // quad_perm 2,3,0,1
  x = dpp_max_step<0x141>(x);  // row_half_mirror
  x = dpp_max_step<0x140>(x);  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Storage formats of code arrays: indices int32 / int16 / uint8, values
// float32 / bfloat16 / float16 (IEEE binary16).
enum : int { kIdxI32 = 0, kIdxI16 = 1, kIdxU8 = 2 };
enum : int { kValF32 = 0, kValBF16 = 1, kValF16 = 2 };

__host__ __device__ constexpr int idx_bytes(int f) { return f == kIdxI32 ? 4 : (f == kIdxI16 ? 2 : 1); }
__host__ __device__ constexpr int val_bytes(int f) { return f == kValF32 ? 4 : 2; }

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h16);
}

// Loads of one code element by format.  Indices are masked into [0, dmask]
// so a violated precondition cannot address outside the kernel's tables.
__device__ __forceinline__ int load_idx(const void* p, int64_t i, int ifmt, int dmask) {
  const int v = ifmt == kIdxI16 ? (int)((const int16_t*)p)[i]
              : ifmt == kIdxU8 ? (int)((const uint8_t*)p)[i]
                               : ((const int32_t*)p)[i];
  return v & dmask;
}

__device__ __forceinline__ float load_val(const void* p, int64_t i, int vfmt) {
  if (vfmt == kValBF16) return bf16_bits_to_f32(((const uint16_t*)p)[i]);
  if (vfmt == kValF16) return f16_bits_to_f32(((const uint16_t*)p)[i]);
  return ((const float*)p)[i];
}

}  // namespace sfa
