// SFA decode over the 8-bit cache ("SFA (quant)", App. E: SFA with 8-bit
// activations, whose cached keys and values are int8 rows with a float32
// scale each): launchers of the decode kernel's 8-bit variant
// (sfa_decode_kernel.h); the chunk partials are merged by the same kernel as
// the bf16 decode.  Per cached key and KV head the step reads k int16
// indices, k int8 values, d int8 values and two scales: 184 bytes at
// d = 128, k = 16, against 320 for int16 / bf16 codes and bf16 V.
#include "sfa_decode_kernel.h"

namespace sfa {
namespace {

template <int D, int G, int KC8>
void launch_q8_t(const DecParams& p, int B, hipStream_t stream) {
  dim3 grid(p.nvc > 0 ? p.nvc : p.nch, B * p.Hkv), block(kDecThreads);
  if (p.table)
    hipLaunchKernelGGL((sfa_decode_kernel<D, G, false, KC8, false, true, true>), grid, block, 0,
                       stream, p);
  else
    hipLaunchKernelGGL((sfa_decode_kernel<D, G, false, KC8, false, false, true>), grid, block, 0,
                       stream, p);
}

template <int D, int G>
void launch_q8_k(const DecParams& p, int B, hipStream_t stream) {
  if (p.k == 8) launch_q8_t<D, G, 1>(p, B, stream);
  else if (p.k == 16) launch_q8_t<D, G, 2>(p, B, stream);
  else launch_q8_t<D, G, 4>(p, B, stream);
}

template <int D>
void launch_q8_g(const DecParams& p, int G, int B, hipStream_t stream) {
  switch (G) {
    case 1: launch_q8_k<D, 1>(p, B, stream); break;
    case 2: launch_q8_k<D, 2>(p, B, stream); break;
    case 4: launch_q8_k<D, 4>(p, B, stream); break;
    default: launch_q8_k<D, 8>(p, B, stream); break;
  }
}

}  // namespace

bool decode_q8_supported(int d, int k, int G) {
  return (d == 64 || d == 128) && (k == 8 || k == 16 || k == 32) && G >= 1 && G <= kDecMaxG &&
         (G & (G - 1)) == 0;
}

hipError_t launch_attn_decode_q8(const DecodeArgs& a, hipStream_t stream) {
  const DecParams p = make_dec_params(a);
  const int G = a.Hq / a.Hkv;
  if (a.d == 64) launch_q8_g<64>(p, G, a.B, stream);
  else launch_q8_g<128>(p, G, a.B, stream);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_decode_combine(p, a, stream);
}

}  // namespace sfa
