// Row-wise Top-k coding (Sec. 3.1, Eqs. (3)-(4)) on gfx950.
//
// A wavefront codes one row at a time, held in registers (lane l holds
// coordinates l, l+64, ...), walking rows with the next one prefetched.  The
// selection itself (exact radix select on integer magnitude keys, ties to the
// lower index) is topk_select; each kept entry finds its output slot
// (ascending index) by a ballot prefix count.
#include "sfa_device.h"
#include "sfa_launch.h"
#include "sfa_topk.h"

namespace sfa {

// E: coordinates per lane (d <= 64 * E); IF, VF: output formats (compile-time,
// so the stores carry no format dispatch)
template <int E, int IF, int VF>
__global__ __launch_bounds__(256) void topk_encode_kernel(
    const float* __restrict__ x, int64_t rows, int d, int k,
    void* __restrict__ idx_out, void* __restrict__ val_out) {
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
      key[e] = topk_key(bits[e], lane + 64 * e < d);
    }
    if (row + nwaves < rows) load_row(row + nwaves);

    bool sel[E];
    topk_select<E>(key, k, sel);
    int slot[E];
    topk_slots<E>(sel, slot);
    const int64_t o0 = row * (int64_t)k;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (sel[e] && slot[e] < k)  // exactly k are kept; the bound only hardens the store
        store_code(idx_out, val_out, o0 + slot[e], lane + 64 * e, bits[e], IF, VF);
  }
}

template <int E, int IF>
static void launch_vf(dim3 grid, const float* x, int64_t rows, int d, int k, void* idx, void* val,
                      int vfmt, hipStream_t stream) {
  if (vfmt == kValBF16)
    hipLaunchKernelGGL((topk_encode_kernel<E, IF, kValBF16>), grid, dim3(256), 0, stream, x, rows, d, k, idx, val);
  else if (vfmt == kValF16)
    hipLaunchKernelGGL((topk_encode_kernel<E, IF, kValF16>), grid, dim3(256), 0, stream, x, rows, d, k, idx, val);
  else
    hipLaunchKernelGGL((topk_encode_kernel<E, IF, kValF32>), grid, dim3(256), 0, stream, x, rows, d, k, idx, val);
}

template <int E>
static void launch_if(dim3 grid, const float* x, int64_t rows, int d, int k, void* idx, int ifmt,
                      void* val, int vfmt, hipStream_t stream) {
  if (ifmt == kIdxI16) launch_vf<E, kIdxI16>(grid, x, rows, d, k, idx, val, vfmt, stream);
  else if (ifmt == kIdxU8) launch_vf<E, kIdxU8>(grid, x, rows, d, k, idx, val, vfmt, stream);
  else launch_vf<E, kIdxI32>(grid, x, rows, d, k, idx, val, vfmt, stream);
}

hipError_t launch_topk_encode(const float* x, int64_t rows, int d, int k, void* idx,
                              int ifmt, void* val, int vfmt, hipStream_t stream) {
  // persistent waves: up to 32 per compute unit, 4 per workgroup
  const int64_t need = (rows + 3) / 4;
  const int64_t cap = 256 * 8;
  const dim3 grid((unsigned)(need < cap ? need : cap));
  if (d <= 64) launch_if<1>(grid, x, rows, d, k, idx, ifmt, val, vfmt, stream);
  else if (d <= 128) launch_if<2>(grid, x, rows, d, k, idx, ifmt, val, vfmt, stream);
  else launch_if<4>(grid, x, rows, d, k, idx, ifmt, val, vfmt, stream);
  return hipGetLastError();
}

}  // namespace sfa
