// SFA decode step (App. B, KV-cache attention) on gfx950: launchers of the
// decode kernel (sfa_decode_kernel.h) for bf16 / float32 V caches, and the
// merge of the context chunks' partials by their LSE.
#include "sfa_decode_kernel.h"

namespace sfa {

// Merge the chunk partials of each (b, h): O = sum_c w_c o_c / sum_c w_c l_c,
// w_c = 2^(m_c - M), LSE = (M + log2 sum_c w_c l_c) ln 2.
template <int D>
__global__ __launch_bounds__(D) void sfa_decode_combine_kernel(
    const float* __restrict__ ws_m, const float* __restrict__ ws_l, const float* __restrict__ ws_o,
    const int32_t* seq_len, int Hq, int Lmax, int nch, int nvc, void* o, int obf16, float* lse) {
  const int bh = blockIdx.x;
  const int b = bh / Hq;
  const int dd = threadIdx.x;
  const int L = seq_len_of(seq_len, b, Lmax);
  // slots written this call: the chunks up to L, or the nvc of a window grid
  const int nc = nvc > 0 ? nvc : (L + kDecChunk - 1) / kDecChunk;
  const int64_t s0 = (int64_t)bh * nch;
  float M = -INFINITY;
  for (int c = 0; c < nc; ++c) M = fmaxf(M, ws_m[s0 + c]);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float lsum = 0.f, osum = 0.f;
  for (int c = 0; c < nc; ++c) {
    const float w = exp2f(ws_m[s0 + c] - Mu);
    lsum += w * ws_l[s0 + c];
    osum += w * ws_o[(s0 + c) * D + dd];
  }
  const float out = lsum > 0.f ? osum / lsum : 0.f;
  if (obf16) ((uint16_t*)o)[(int64_t)bh * D + dd] = (uint16_t)f32_to_bf16_rne(out);
  else ((float*)o)[(int64_t)bh * D + dd] = out;
  if (lse && dd == 0) lse[bh] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
}

size_t decode_workspace_bytes(int B, int Hq, int Lmax, int d) {
  const size_t nch = (size_t)((Lmax + kDecChunk - 1) / kDecChunk);
  return (size_t)B * Hq * nch * (size_t)(d + 2) * sizeof(float);
}

template <int D, int G, bool VBF16, int KC8, bool C8>
static void launch_dec_t(const DecParams& p, int B, hipStream_t stream) {
  dim3 grid(p.nvc > 0 ? p.nvc : p.nch, B * p.Hkv), block(kDecThreads);
  if (p.table)
    hipLaunchKernelGGL((sfa_decode_kernel<D, G, VBF16, KC8, C8, true>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((sfa_decode_kernel<D, G, VBF16, KC8, C8, false>), grid, block, 0, stream, p);
}

template <int D, int G, bool VBF16>
static void launch_dec_kc(const DecParams& p, int B, hipStream_t stream) {
  if constexpr (VBF16) {
    if (p.kifmt == kIdxI16 && p.kvfmt == kValBF16) {
      if (p.k == 8) return launch_dec_t<D, G, VBF16, 1, false>(p, B, stream);
      if (p.k == 16) return launch_dec_t<D, G, VBF16, 2, false>(p, B, stream);
      if (p.k == 32) return launch_dec_t<D, G, VBF16, 4, false>(p, B, stream);
    }
    if (p.kifmt == kIdxU8 && p.kvfmt == kValF16) {
      if (p.k == 8) return launch_dec_t<D, G, VBF16, 1, true>(p, B, stream);
      if (p.k == 16) return launch_dec_t<D, G, VBF16, 2, true>(p, B, stream);
      if (p.k == 32) return launch_dec_t<D, G, VBF16, 4, true>(p, B, stream);
    }
  }
  launch_dec_t<D, G, VBF16, 0, false>(p, B, stream);
}

template <int D, bool VBF16>
static void launch_dec_g(const DecParams& p, int G, int B, hipStream_t stream) {
  switch (G) {
    case 1: launch_dec_kc<D, 1, VBF16>(p, B, stream); break;
    case 2: launch_dec_kc<D, 2, VBF16>(p, B, stream); break;
    case 4: launch_dec_kc<D, 4, VBF16>(p, B, stream); break;
    default: launch_dec_kc<D, 8, VBF16>(p, B, stream); break;
  }
}

int decode_max_group() { return kDecMaxG; }

DecParams make_dec_params(const DecodeArgs& a) {
  DecParams p;
  p.q_idx = a.q_idx; p.q_val = a.q_val; p.kc_idx = a.kc_idx; p.kc_val = a.kc_val; p.v = a.v;
  p.seq_len = a.seq_len;
  p.Hq = a.Hq; p.Hkv = a.Hkv; p.Lmax = a.Lmax; p.k = a.k;
  p.nch = (a.Lmax + kDecChunk - 1) / kDecChunk;
  const size_t nslot = (size_t)a.B * a.Hq * p.nch;
  p.ws_m = (float*)a.ws;
  p.ws_l = p.ws_m + nslot;
  p.ws_o = p.ws_l + nslot;
  p.scale_log2 = (float)((double)a.scale * 1.4426950408889634);
  p.qifmt = a.qifmt; p.qvfmt = a.qvfmt; p.kifmt = a.kifmt; p.kvfmt = a.kvfmt;
  p.q_dense = a.q_dense;
  p.table = a.table;
  p.max_pages = a.max_pages; p.log2P = a.log2P; p.num_pages = a.num_pages;
  p.window = a.window; p.n_global = a.n_global;
  p.nvc = 0;
  if (a.window > 0) {
    // the global chunks, the window's chunks (one more when it straddles a
    // chunk boundary), never more than the whole context
    const int g = min(a.n_global, a.Lmax);
    const int v = (g + kDecChunk - 1) / kDecChunk + (a.window + kDecChunk - 1) / kDecChunk + 1;
    p.nvc = min(v, p.nch);
  }
  p.kc_scale = a.kc_scale;
  p.v_scale = a.v_scale;
  return p;
}

hipError_t launch_decode_combine(const DecParams& p, const DecodeArgs& a, hipStream_t stream) {
  if (a.d == 64)
    hipLaunchKernelGGL(sfa_decode_combine_kernel<64>, dim3(a.B * a.Hq), dim3(64), 0, stream,
                       p.ws_m, p.ws_l, p.ws_o, a.seq_len, a.Hq, a.Lmax, p.nch, p.nvc, a.o,
                       a.obf16, a.lse);
  else
    hipLaunchKernelGGL(sfa_decode_combine_kernel<128>, dim3(a.B * a.Hq), dim3(128), 0, stream,
                       p.ws_m, p.ws_l, p.ws_o, a.seq_len, a.Hq, a.Lmax, p.nch, p.nvc, a.o,
                       a.obf16, a.lse);
  return hipGetLastError();
}

hipError_t launch_attn_decode(const DecodeArgs& a, hipStream_t stream) {
  const DecParams p = make_dec_params(a);
  const int G = a.Hq / a.Hkv, B = a.B;
  if (a.d == 64) {
    if (a.vbf16) launch_dec_g<64, true>(p, G, B, stream); else launch_dec_g<64, false>(p, G, B, stream);
  } else {
    if (a.vbf16) launch_dec_g<128, true>(p, G, B, stream); else launch_dec_g<128, false>(p, G, B, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_decode_combine(p, a, stream);
}

}  // namespace sfa
