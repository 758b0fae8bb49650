// CSR code storage (Sec. 2's sparse formats; App. J stores codes as CSR with
// int32 indptr, 8-bit indices and fp16 values) brought to the fixed-width
// code rows the attention kernels read.
//
// Row r of the CSR matrix holds entries indptr[r] .. indptr[r+1]-1, at most
// kmax of them.  The fixed row keeps those entries and adds zero-valued
// entries at the lowest coordinates the row does not hold until it has kmax,
// all in ascending index order -- the same matrix, and the same rule the
// Top-k coding uses for rows with fewer than k nonzeros.
//
// One wavefront per row: lane l stands for coordinates l + 64 e.  The row's
// entries are loaded in parallel (one per lane), broadcast one by one with
// readlane and marked on the coordinate they hold; the padding is the first
// free coordinates by a ballot prefix count, and each kept coordinate finds
// its output slot by a second one.
#include "sfa_device.h"
#include "sfa_launch.h"
#include "sfa_topk.h"

namespace sfa {

template <int E>  // coordinates per lane: d <= 64 * E
__global__ __launch_bounds__(256) void sfa_csr_to_codes_kernel(CsrArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * 4;
  int64_t row = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (; row < a.rows; row += stride) {
    const int64_t p0 = a.indptr[row];
    int64_t m = (int64_t)a.indptr[row + 1] - p0;
    m = m < 0 ? 0 : (m > a.kmax ? a.kmax : m);  // longer rows: the first kmax entries
    bool held[E];
    uint32_t vbits[E];
#pragma unroll
    for (int e = 0; e < E; ++e) { held[e] = false; vbits[e] = 0u; }
    for (int c0 = 0; c0 < m; c0 += 64) {
      int u_l = -1;
      uint32_t v_l = 0u;
      if (c0 + lane < m) {
        const int64_t t = p0 + c0 + lane;
        u_l = load_idx(a.indices, t, a.ifmt_in, -1);
        v_l = a.vbytes == 4 ? ((const uint32_t*)a.values)[t] : ((const uint16_t*)a.values)[t];
      }
      const int cn = (int)min((int64_t)64, m - c0);
      for (int j = 0; j < cn; ++j) {
        int u = __builtin_amdgcn_readlane(u_l, j);
        if (u >= a.d) u = -1;  // out-of-range index (violated precondition): ignored
        const uint32_t vb = (uint32_t)__builtin_amdgcn_readlane((int)v_l, j);
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (lane + 64 * e == u) { held[e] = true; vbits[e] = vb; }
      }
    }
    int nheld = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) nheld += __popcll(wave_ballot(held[e]));
    const int need = a.kmax - nheld;  // zero entries to add
    bool sel[E];
    int before = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const bool fr = !held[e] && lane + 64 * e < a.d;
      const uint64_t fm = wave_ballot(fr);
      sel[e] = held[e] || (fr && before + lanes_below(fm) < need);
      before += __popcll(fm);
    }
    int slot[E];
    topk_slots<E>(sel, slot);
    const int64_t o0 = row * a.kmax;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (sel[e] && slot[e] < a.kmax) {
        const int64_t pos = o0 + slot[e];
        const int u = lane + 64 * e;
        if (a.ifmt_out == kIdxI16) ((int16_t*)a.idx_out)[pos] = (int16_t)u;
        else if (a.ifmt_out == kIdxU8) ((uint8_t*)a.idx_out)[pos] = (uint8_t)u;
        else ((int32_t*)a.idx_out)[pos] = u;
        if (a.vbytes == 4) ((uint32_t*)a.val_out)[pos] = vbits[e];
        else ((uint16_t*)a.val_out)[pos] = (uint16_t)vbits[e];
      }
    }
  }
}

hipError_t launch_csr_to_codes(const CsrArgs& a, hipStream_t stream) {
  if (a.rows == 0) return hipSuccess;
  const int64_t need = (a.rows + 3) / 4, cap = 256 * 8;
  dim3 grid((unsigned)(need < cap ? need : cap)), block(256);
  if (a.d <= 64)
    hipLaunchKernelGGL(sfa_csr_to_codes_kernel<1>, grid, block, 0, stream, a);
  else if (a.d <= 128)
    hipLaunchKernelGGL(sfa_csr_to_codes_kernel<2>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(sfa_csr_to_codes_kernel<4>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace sfa
