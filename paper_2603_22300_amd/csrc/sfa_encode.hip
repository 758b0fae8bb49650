// Row-wise Top-k coding (Sec. 3.1, Eqs. (3)-(4)) on gfx950.
//
// A wavefront codes one row at a time, held in registers (lane l holds
// coordinates l, l+64, ...), walking rows with the next one prefetched.  Selection is an exact radix select on integer magnitude
// keys: key = (bits & 0x7fffffff) + 1, so that the unsigned order of keys is
// the order of |x| on finite floats, subnormals included, and key 0 marks the
// padding lanes beyond d.  The k-th largest key is found one bit at a time
// from the top with ballot + popcount (wave-uniform scalar work); if at some
// bit exactly k keys are at or above the candidate, the kept set is known
// and the search stops early.  Otherwise the ties at the threshold are
// broken by lower index with a ballot prefix count, and each kept entry finds
// its output slot (ascending index) by a second ballot prefix count.
#include "sfa_device.h"
#include "sfa_launch.h"

namespace sfa {

template <int E>  // coordinates per lane: d <= 64 * E
__global__ __launch_bounds__(256) void topk_encode_kernel(
    const float* __restrict__ x, int64_t rows, int d, int k,
    void* __restrict__ idx_out, int idx16, void* __restrict__ val_out, int valbf16) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  // the wave index is made visibly uniform so that the row walk and the
  // whole search below stay in scalar registers
  int64_t row = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (row >= rows) return;  // uniform per wave

  // Persistent wavefronts: the next row's load is in flight while this row
  // is selected.  Loads are unconditional (lanes past d re-read the row's
  // last coordinate and are masked by key 0).
  uint32_t nxt[E];
  auto load_row = [&](int64_t r) {
    const float* xr = x + r * (int64_t)d;
#pragma unroll
    for (int e = 0; e < E; ++e) nxt[e] = __float_as_uint(xr[min(lane + 64 * e, d - 1)]);
  };
  load_row(row);
  for (; row < rows; row += nwaves) {
    uint32_t bits[E], key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      bits[e] = nxt[e];
      key[e] = (lane + 64 * e < d) ? (bits[e] & 0x7fffffffu) + 1u : 0u;
    }
    if (row + nwaves < rows) load_row(row + nwaves);

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

    bool sel[E];
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

    // Output slot = number of kept coordinates with a smaller index.
    int base = 0;
    const int64_t o0 = row * (int64_t)k;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const uint64_t m = wave_ballot(sel[e]);
      const int slot = base + lanes_below(m);
      if (sel[e] && slot < k) {  // exactly k are kept; the bound only hardens the store
        const int64_t pos = o0 + slot;
        const int u = lane + 64 * e;
        if (idx16) ((int16_t*)idx_out)[pos] = (int16_t)u;
        else ((int32_t*)idx_out)[pos] = u;
        if (valbf16) ((uint16_t*)val_out)[pos] = (uint16_t)f32_to_bf16_rne(__uint_as_float(bits[e]));
        else ((uint32_t*)val_out)[pos] = bits[e];
      }
      base += __popcll(m);
    }
  }
}

hipError_t launch_topk_encode(const float* x, int64_t rows, int d, int k, void* idx,
                              int idx16, void* val, int valbf16, hipStream_t stream) {
  // persistent waves: up to 32 per compute unit, 4 per workgroup
  const int64_t need = (rows + 3) / 4;
  const int64_t cap = 256 * 8;
  dim3 grid((unsigned)(need < cap ? need : cap)), block(256);
  if (d <= 64)
    hipLaunchKernelGGL(topk_encode_kernel<1>, grid, block, 0, stream, x, rows, d, k, idx, idx16, val, valbf16);
  else if (d <= 128)
    hipLaunchKernelGGL(topk_encode_kernel<2>, grid, block, 0, stream, x, rows, d, k, idx, idx16, val, valbf16);
  else
    hipLaunchKernelGGL(topk_encode_kernel<4>, grid, block, 0, stream, x, rows, d, k, idx, idx16, val, valbf16);
  return hipGetLastError();
}

}  // namespace sfa
