// Decode over a sparse-code KV cache (App. B) for head dimensions without
// the tuned kernel: any d <= 256 other than 64 and 128, float32 arithmetic.
//
// Same split of the context as the tuned decode: a workgroup takes one chunk
// of cached keys of one (sequence, KV head) for all G query heads and
// writes a partial (m, l, o) per head; a combine kernel merges the chunks by
// their log-sum-exp.  Inside a chunk, sub-blocks of 256 keys: thread = key
// for the scores (s_h = sum_t kval_t * qd[kidx_t][h], the query codes
// densified in LDS with scale * log2(e) folded in), block-wide maximum and
// sum per head, then thread = output dimension for P.V.  Contiguous or paged
// cache, query codes or a dense query coded here (the shared exact Top-k),
// and the token window of the tuned decode.
#include "sfa_device.h"
#include "sfa_launch.h"
#include "sfa_topk.h"

namespace sfa {
namespace {

constexpr int kGdChunk = kDecodeChunk;  // keys per workgroup: the workspace's partial slots
constexpr int kGdT = 256;       // threads; keys per sub-block
constexpr int kGdW = kGdT / 64;
constexpr int kGdMaxG = 8;

struct GDecParams {
  const float* q_dense;
  const void *q_idx, *q_val, *kc_idx, *kc_val, *v;
  const int32_t* seq_len;
  const int32_t* table;
  int Hq, Hkv, Lmax, d, k, G;
  int page_size, log2P, max_pages, num_pages;
  int window, n_global;
  float scale_log2;
  int qifmt, qvfmt, kifmt, kvfmt, vbf16;
  int nch;
  float *ws_m, *ws_l, *ws_o;  // [B*Hq, nch], [B*Hq, nch], [B*Hq, nch, d]
};

__device__ __forceinline__ int gd_seq_len(const int32_t* seq_len, int b, int Lmax) {
  if (!seq_len) return Lmax;
  const int L = seq_len[b];
  return L < 0 ? 0 : (L > Lmax ? Lmax : L);
}

__device__ __forceinline__ int gd_idx(const void* p, int64_t i, int ifmt, int d) {
  const int u = load_idx(p, i, ifmt, -1);
  return u < 0 ? 0 : (u >= d ? d - 1 : u);
}

// E: coordinates per lane of the in-kernel query coding (d <= 64 * E)
template <int E>
__global__ __launch_bounds__(kGdT) void sfa_decode_generic_kernel(GDecParams p) {
  __shared__ float qd[256 * kGdMaxG];  // [d][G]
  __shared__ float ps[kGdMaxG * kGdT];  // [G][key of the sub-block]
  __shared__ int64_t rows[kGdT];       // cache row of each key of the sub-block
  __shared__ float red[kGdW * kGdMaxG];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int d = p.d, k = p.k, G = p.G;
  const int bh = blockIdx.y, b = bh / p.Hkv, hkv = bh - b * p.Hkv;
  const int chunk = blockIdx.x;
  const int L = gd_seq_len(p.seq_len, b, p.Lmax);
  const int c0 = chunk * kGdChunk;
  if (c0 >= L) return;  // past the sequence: the combine reads only chunks below L
  const int c1 = min(L, c0 + kGdChunk);
  const int64_t slot0 = ((int64_t)b * p.Hq + hkv * G) * p.nch + chunk;  // head h: + h * nch

  // the query densified per head, scaled to base-2 exponents
  for (int x = tid; x < d * G; x += kGdT) qd[x] = 0.f;
  __syncthreads();
  if (p.q_dense) {
    // one wavefront per head codes the dense row (exact Top-k, as the coding
    // kernel); kept coordinates keep their float32 value
    for (int h = wave; h < G; h += kGdW) {
      const float* qr = p.q_dense + ((int64_t)b * p.Hq + hkv * G + h) * d;
      uint32_t bits[E], key[E];
      bool sel[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int c = lane + 64 * e;
        bits[e] = __float_as_uint(qr[min(c, d - 1)]);
        key[e] = topk_key(bits[e], c < d);
      }
      topk_select<E>(key, k, sel);
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (sel[e]) qd[(lane + 64 * e) * G + h] = p.scale_log2 * __uint_as_float(bits[e]);
    }
  } else {
    for (int x = tid; x < G * k; x += kGdT) {
      const int h = x / k, t = x - h * k;
      const int64_t qi = ((int64_t)b * p.Hq + hkv * G + h) * k + t;
      qd[gd_idx(p.q_idx, qi, p.qifmt, d) * G + h] = p.scale_log2 * load_val(p.q_val, qi, p.qvfmt);
    }
  }
  __syncthreads();

  // the query sits at position L - 1; with a window it sees keys j with
  // (L - 1) - j < window, the first n_global keys, and every key if it is a
  // global token itself
  const bool win = p.window > 0;
  const int qpos = L - 1;
  auto allowed = [&](int j) {
    return !win || qpos - j < p.window || j < p.n_global || qpos < p.n_global;
  };
  auto row_of = [&](int j) -> int64_t {
    if (!p.table) return ((int64_t)b * p.Hkv + hkv) * p.Lmax + j;
    int pg = p.table[(int64_t)b * p.max_pages + (j >> p.log2P)];
    pg = min(max(pg, 0), p.num_pages - 1);
    return ((int64_t)pg * p.Hkv + hkv) * p.page_size + (j & (p.page_size - 1));
  };

  float m_run[kGdMaxG], l_run[kGdMaxG], acc[kGdMaxG];
#pragma unroll
  for (int h = 0; h < kGdMaxG; ++h) { m_run[h] = -INFINITY; l_run[h] = 0.f; acc[h] = 0.f; }

  for (int jb = c0; jb < c1; jb += kGdT) {
    const int j = jb + tid;
    const bool ok = j < c1 && allowed(j);
    float s[kGdMaxG];
#pragma unroll
    for (int h = 0; h < kGdMaxG; ++h) s[h] = -INFINITY;
    if (ok) {
      const int64_t row = row_of(j);
      rows[tid] = row;
#pragma unroll
      for (int h = 0; h < kGdMaxG; ++h) s[h] = 0.f;
      for (int t = 0; t < k; ++t) {
        const int64_t ci = row * k + t;
        const int u = gd_idx(p.kc_idx, ci, p.kifmt, d);
        const float x = load_val(p.kc_val, ci, p.kvfmt);
#pragma unroll
        for (int h = 0; h < kGdMaxG; ++h)
          if (h < G) s[h] = fmaf(x, qd[u * G + h], s[h]);
      }
    } else {
      rows[tid] = -1;
    }
    // block maximum per head
#pragma unroll
    for (int h = 0; h < kGdMaxG; ++h) {
      if (h < G) {
        const float mw = wave_max(s[h]);
        if (lane == 0) red[wave * kGdMaxG + h] = mw;
      }
    }
    __syncthreads();
    float alpha[kGdMaxG], m_use[kGdMaxG];
#pragma unroll
    for (int h = 0; h < kGdMaxG; ++h) {
      float mt = -INFINITY;
      if (h < G)
        for (int w = 0; w < kGdW; ++w) mt = fmaxf(mt, red[w * kGdMaxG + h]);
      const float m_new = fmaxf(m_run[h], mt);
      m_use[h] = m_new == -INFINITY ? 0.f : m_new;
      alpha[h] = __builtin_amdgcn_exp2f(m_run[h] - m_use[h]);
      m_run[h] = m_new;
    }
    __syncthreads();  // the maxima are read before red is reused
    // probabilities and their block sums per head
#pragma unroll
    for (int h = 0; h < kGdMaxG; ++h) {
      if (h < G) {
        const float pr = __builtin_amdgcn_exp2f(s[h] - m_use[h]);
        ps[h * kGdT + tid] = pr;
        const float sw = wave_sum(pr);
        if (lane == 0) red[wave * kGdMaxG + h] = sw;
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < kGdMaxG; ++h) {
      if (h < G) {
        float sum = 0.f;
        for (int w = 0; w < kGdW; ++w) sum += red[w * kGdMaxG + h];
        l_run[h] = l_run[h] * alpha[h] + sum;
        acc[h] *= alpha[h];
      }
    }
    // P.V: thread = output dimension
    if (tid < d) {
      const int nk = min(kGdT, c1 - jb);
      for (int jj = 0; jj < nk; ++jj) {
        const int64_t row = rows[jj];
        if (row < 0) continue;  // masked key (uniform)
        const int64_t vi = row * d + tid;
        const float vv = p.vbf16 ? bf16_bits_to_f32(((const uint16_t*)p.v)[vi]) : ((const float*)p.v)[vi];
#pragma unroll
        for (int h = 0; h < kGdMaxG; ++h)
          if (h < G) acc[h] = fmaf(ps[h * kGdT + jj], vv, acc[h]);
      }
    }
    __syncthreads();  // ps, rows and red are rewritten by the next sub-block
  }

#pragma unroll
  for (int h = 0; h < kGdMaxG; ++h) {
    if (h < G) {
      const int64_t slot = slot0 + (int64_t)h * p.nch;
      if (tid < d) p.ws_o[slot * d + tid] = acc[h];
      if (tid == 0) { p.ws_m[slot] = m_run[h]; p.ws_l[slot] = l_run[h]; }
    }
  }
}

// Partials of the chunks below L merged per (b, head): w_c = 2^(m_c - M),
// O = sum_c w_c o_c / sum_c w_c l_c, LSE = (M + log2 sum_c w_c l_c) ln 2.
__global__ __launch_bounds__(kGdT) void sfa_decode_generic_combine_kernel(
    const float* __restrict__ ws_m, const float* __restrict__ ws_l, const float* __restrict__ ws_o,
    const int32_t* seq_len, int Hq, int Lmax, int nch, int d, void* o, int obf16, float* lse) {
  const int bh = blockIdx.x, b = bh / Hq, dd = threadIdx.x;
  const int L = gd_seq_len(seq_len, b, Lmax);
  const int nc = (L + kGdChunk - 1) / kGdChunk;
  const int64_t s0 = (int64_t)bh * nch;
  float M = -INFINITY;
  for (int c = 0; c < nc; ++c) M = fmaxf(M, ws_m[s0 + c]);
  const float Mu = (M == -INFINITY) ? 0.f : M;
  float lsum = 0.f, osum = 0.f;
  for (int c = 0; c < nc; ++c) {
    const float w = exp2f(ws_m[s0 + c] - Mu);
    lsum += w * ws_l[s0 + c];
    if (dd < d) osum += w * ws_o[(s0 + c) * d + dd];
  }
  if (dd < d) {
    const float out = lsum > 0.f ? osum / lsum : 0.f;
    if (obf16) ((uint16_t*)o)[(int64_t)bh * d + dd] = (uint16_t)f32_to_bf16_rne(out);
    else ((float*)o)[(int64_t)bh * d + dd] = out;
  }
  if (lse && dd == 0) lse[bh] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : -INFINITY;
}

}  // namespace

int decode_generic_max_group() { return kGdMaxG; }

hipError_t launch_attn_decode_generic(const DecodeArgs& a, hipStream_t stream) {
  GDecParams p;
  p.q_dense = a.q_dense; p.q_idx = a.q_idx; p.q_val = a.q_val;
  p.kc_idx = a.kc_idx; p.kc_val = a.kc_val; p.v = a.v;
  p.seq_len = a.seq_len; p.table = a.table;
  p.Hq = a.Hq; p.Hkv = a.Hkv; p.Lmax = a.Lmax; p.d = a.d; p.k = a.k; p.G = a.Hq / a.Hkv;
  p.log2P = a.log2P; p.page_size = 1 << a.log2P; p.max_pages = a.max_pages;
  p.num_pages = a.num_pages;
  p.window = a.window; p.n_global = a.n_global;
  p.scale_log2 = (float)((double)a.scale * 1.4426950408889634);
  p.qifmt = a.qifmt; p.qvfmt = a.qvfmt; p.kifmt = a.kifmt; p.kvfmt = a.kvfmt;
  p.vbf16 = a.vbf16;
  p.nch = (a.Lmax + kGdChunk - 1) / kGdChunk;
  const size_t nslot = (size_t)a.B * a.Hq * p.nch;
  p.ws_m = (float*)a.ws;
  p.ws_l = p.ws_m + nslot;
  p.ws_o = p.ws_l + nslot;
  const dim3 grid(p.nch, a.B * a.Hkv), block(kGdT);
  if (a.d <= 64) hipLaunchKernelGGL(sfa_decode_generic_kernel<1>, grid, block, 0, stream, p);
  else if (a.d <= 128) hipLaunchKernelGGL(sfa_decode_generic_kernel<2>, grid, block, 0, stream, p);
  else hipLaunchKernelGGL(sfa_decode_generic_kernel<4>, grid, block, 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sfa_decode_generic_combine_kernel, dim3(a.B * a.Hq), dim3(kGdT), 0, stream,
                     p.ws_m, p.ws_l, p.ws_o, a.seq_len, a.Hq, a.Lmax, p.nch, a.d, a.o, a.obf16,
                     a.lse);
  return hipGetLastError();
}

}  // namespace sfa
