// Wavefront Top-k selection of one row (Sec. 3.1, Eqs. (3)-(4)), shared by
// the coding kernel, the cache append and the decode kernel's in-kernel
// query coding.
//
// The row is held by one wavefront, lane l holding coordinates l + 64 e.
// Selection is an exact radix select on integer magnitude keys:
// key = (bits & 0x7fffffff) + 1, so that the unsigned order of keys is the
// order of |x| on finite floats, subnormals included, and key 0 marks the
// padding lanes beyond d.  The k-th largest key is found one bit at a time
// from the top with ballot + popcount (wave-uniform scalar work); if at some
// bit exactly k keys are at or above the candidate, the kept set is known and
// the search stops early.  Otherwise the ties at the threshold are broken by
// lower index with a ballot prefix count.
#pragma once

#include "sfa_device.h"

namespace sfa {

__device__ __forceinline__ uint32_t topk_key(uint32_t bits, bool valid) {
  return valid ? (bits & 0x7fffffffu) + 1u : 0u;
}

// sel[e]: coordinate lane + 64 e is among the k kept.  Every lane of the
// wavefront must call this with the same k (it is wave-uniform work).
template <int E>
__device__ __forceinline__ void topk_select(const uint32_t (&key)[E], int k, bool (&sel)[E]) {
  // Largest T with #{key >= T} >= k, built from the most significant bit.
  // Finite keys are below 2^31 (bit 31 is never set), so the search starts
  // at bit 30; a NaN's key can reach 2^31 and then simply ranks above every
  // candidate, i.e. above all finite values.
  uint32_t prefix = 0u;
  bool exact = false;
#pragma unroll
  for (int b = 30; b >= 0; --b) {
    const uint32_t cand = prefix | (1u << b);
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) cnt += __popcll(wave_ballot(key[e] >= cand));
    cnt = __builtin_amdgcn_readfirstlane(cnt);
    if (cnt >= k) prefix = cand;
    prefix = __builtin_amdgcn_readfirstlane(prefix);
    if (cnt == k) { exact = true; break; }
  }
  if (exact) {
#pragma unroll
    for (int e = 0; e < E; ++e) sel[e] = key[e] >= prefix;
  } else {
    const uint32_t T = prefix;
    int gt = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) gt += __popcll(wave_ballot(key[e] > T));
    const int need = k - gt;  // ties at T to keep, lowest indices first
    int before = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const uint64_t eq = wave_ballot(key[e] == T);
      const int r = before + lanes_below(eq);
      sel[e] = key[e] > T || (key[e] == T && r < need);
      before += __popcll(eq);
    }
  }
}

// slot[e]: output position of a kept coordinate among the kept ones in
// ascending coordinate order (the number of kept coordinates below it).
template <int E>
__device__ __forceinline__ void topk_slots(const bool (&sel)[E], int (&slot)[E]) {
  int base = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint64_t m = wave_ballot(sel[e]);
    slot[e] = base + lanes_below(m);
    base += __popcll(m);
  }
}

// Stores of one code entry in the requested formats (bf16 and float16
// values round to nearest even).
__device__ __forceinline__ void store_code(void* idx_out, void* val_out, int64_t pos, int u,
                                           uint32_t bits, int ifmt, int vfmt) {
  if (ifmt == kIdxI16) ((int16_t*)idx_out)[pos] = (int16_t)u;
  else if (ifmt == kIdxU8) ((uint8_t*)idx_out)[pos] = (uint8_t)u;
  else ((int32_t*)idx_out)[pos] = u;
  if (vfmt == kValBF16) ((uint16_t*)val_out)[pos] = (uint16_t)f32_to_bf16_rne(__uint_as_float(bits));
  else if (vfmt == kValF16) ((_Float16*)val_out)[pos] = (_Float16)__uint_as_float(bits);
  else ((uint32_t*)val_out)[pos] = bits;
}

}  // namespace sfa
