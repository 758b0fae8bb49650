// Wavefront Top-k selection of one row (Sec. 3.1, Eqs. (3)-(4)), shared by
// the coding kernel, the cache append and the decode kernel's in-kernel
// query coding.
//
// The row is held by one wavefront, lane l holding coordinates l + 64 e.
// Selection is an exact radix select on integer magnitude keys:
// key = (bits & 0x7fffffff) + 1, so that the unsigned order of keys is the
// order of |x| on finite floats, subnormals included, and key 0 marks the
// padding lanes beyond d.  The k-th largest key is found one bit at a time
// from the top with ballot + popcount (wave-uniform scalar work), the
// exponent bits mostly by two probes next to the largest key's exponent; if
// at some step exactly k keys are at or above the candidate, the kept set is
// known and the search stops early.  Otherwise the ties at the threshold are broken by
// lower index with a ballot prefix count.
#pragma once

#include "sfa_device.h"

namespace sfa {

__device__ __forceinline__ uint32_t topk_key(uint32_t bits, bool valid) {
  return valid ? (bits & 0x7fffffffu) + 1u : 0u;
}

// Number of keys at or above cand (wave-uniform).
template <int E>
__device__ __forceinline__ int topk_count_ge(const uint32_t (&key)[E], uint32_t cand) {
  int cnt = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) cnt += __popcll(wave_ballot(key[e] >= cand));
  return __builtin_amdgcn_readfirstlane(cnt);
}

// The search from bit B down, given #{key >= prefix} >= k and fewer than k
// keys at or above prefix + 2^(B+1); then the selection.  If at some bit
// exactly k keys are at or above the candidate, the kept set is known and
// the search stops early; otherwise more than k keys share the threshold T
// and the ties at T are kept lowest index first.
template <int E, int B>
__device__ __forceinline__ void topk_search(const uint32_t (&key)[E], int k, uint32_t prefix,
                                            bool (&sel)[E]) {
  bool exact = false;
#pragma unroll
  for (int b = B; b >= 0; --b) {
    const uint32_t cand = prefix | (1u << b);
    const int cnt = topk_count_ge<E>(key, cand);
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

// sel[e]: coordinate lane + 64 e is among the k kept.  All 64 lanes of the
// wavefront must be active and call this with the same k (it is wave-uniform
// work, and the maximum below reads every lane).
template <int E>
__device__ __forceinline__ void topk_select(const uint32_t (&key)[E], int k, bool (&sel)[E]) {
  // T = the largest value with #{key >= T} >= k.  Finite keys are below 2^31
  // (bit 31 is never set), so its bits are searched from bit 30; a NaN's key
  // can reach 2^31 and then simply ranks above every candidate, i.e. above
  // all finite values.
  //
  // Bits 30..23 of a key are the exponent field of |x| (up to the +1, which
  // keeps the order).  They are found first by probing h << 23 for h = the
  // largest key's field, then one below: if #{key >= h << 23} >= k while
  // #{key >= (h + 1) << 23} < k, T lies in [h << 23, (h + 1) << 23).  For
  // rows of comparable magnitudes (the k-th largest within a factor 4 of the
  // largest) this replaces eight search steps by two probes; otherwise the
  // search runs over those bits as well.
  uint32_t mx = key[0];
#pragma unroll
  for (int e = 1; e < E; ++e) mx = max(mx, key[e]);
  uint32_t h = wave_umax(mx) >> 23;  // (h + 1) << 23 is above every key
  int cnt = topk_count_ge<E>(key, h << 23);
  if (cnt < k) {
    h = h - 1u;  // h >= 1 here: every key is >= 0 and there are at least k
    cnt = topk_count_ge<E>(key, h << 23);
  }
  if (cnt == k) {
#pragma unroll
    for (int e = 0; e < E; ++e) sel[e] = key[e] >= (h << 23);
  } else if (cnt > k) {
    topk_search<E, 22>(key, k, h << 23, sel);
  } else {
    topk_search<E, 30>(key, k, 0u, sel);
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
