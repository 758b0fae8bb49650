// SFA forward (Sec. 3.1-3.2) for head dimensions without a matrix-core
// kernel: any d <= 256 other than 64 and 128, in plain float32 arithmetic.
//
// A workgroup takes 32 query rows of one query head.  Their codes are
// densified into LDS, scaled by scale * log2(e), so that a score is a base-2
// exponent.  Key tiles of 32 keys are staged as codes (index, value) plus the
// value rows; each key's score against a row is the overlap sum
// s_ij = sum_t kval_jt * qd_i[kidx_jt], k LDS lookups (the keys' supports
// pick the query coordinates; coordinates outside the query's support read
// zeros).  Online softmax per row (exact running maximum), then P.V on the
// vector unit.  Eight threads share a row: keys c8, c8 + 8, ... for the
// scores and dimensions c8, c8 + 8, ... for the output.
#include "sfa_device.h"
#include "sfa_launch.h"

namespace sfa {
namespace {

constexpr int kGR = 32;    // query rows per workgroup
constexpr int kGC = 32;    // keys per tile
constexpr int kGT = 256;   // threads: 8 per row
constexpr int kGDmax = 256;
constexpr int kGNA = kGDmax / 8;  // output dimensions per thread, at most

struct GenParams {
  const void* q_idx;
  const void* q_val;
  const void* k_idx;
  const void* k_val;
  const void* v;
  void* o;
  float* lse;
  int Hq, Hkv, n, d, k, causal, window, n_global;
  float scale_log2;  // scale * log2(e)
  int ifmt, vfmt, vbf16, obf16;
  int nqb;
};

__host__ __device__ constexpr size_t generic_lds_bytes(int d, int k) {
  return sizeof(float) * ((size_t)kGR * d + (size_t)kGC * d + 2 * (size_t)kGC * k +
                          (size_t)kGR * (kGC + 1));
}

// index of a code entry clamped into [0, d): a violated precondition
// (0 <= idx < d) cannot address outside the tables
__device__ __forceinline__ int code_idx(const void* p, int64_t i, int ifmt, int d) {
  const int u = load_idx(p, i, ifmt, -1);
  return u < 0 ? 0 : (u >= d ? d - 1 : u);
}

__device__ __forceinline__ float row_max8(float x) {
  x = fmaxf(x, __shfl_xor(x, 1, 64));
  x = fmaxf(x, __shfl_xor(x, 2, 64));
  return fmaxf(x, __shfl_xor(x, 4, 64));
}

__device__ __forceinline__ float row_sum8(float x) {
  x += __shfl_xor(x, 1, 64);
  x += __shfl_xor(x, 2, 64);
  return x + __shfl_xor(x, 4, 64);
}

__global__ __launch_bounds__(kGT) void sfa_fwd_generic_kernel(GenParams p) {
  extern __shared__ __attribute__((aligned(16))) float gsm[];
  const int d = p.d, k = p.k, n = p.n;
  float* Qd = gsm;                       // [kGR][d] scaled dense query rows
  float* Vs = Qd + kGR * d;              // [kGC][d] value rows of the tile
  float* Kv = Vs + kGC * d;              // [kGC][k] code values of the tile
  int* Ki = (int*)(Kv + kGC * k);        // [kGC][k] code indices of the tile
  float* Ps = (float*)(Ki + kGC * k);    // [kGR][kGC + 1] probabilities

  const int tid = threadIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / p.Hq, hq = bh - b * p.Hq;
  const int hkv = hq / (p.Hq / p.Hkv);
  const int i0 = (p.nqb - 1 - (int)blockIdx.x) * kGR;  // longest causal blocks first
  const int64_t qrow0 = ((int64_t)b * p.Hq + hq) * n;
  const int64_t krow0 = ((int64_t)b * p.Hkv + hkv) * n;

  for (int x = tid; x < kGR * d; x += kGT) Qd[x] = 0.f;
  __syncthreads();
  for (int e = tid; e < kGR * k; e += kGT) {
    const int r = e / k, t = e - r * k, i = i0 + r;
    if (i < n) {
      const int64_t gi = (qrow0 + i) * k + t;
      Qd[r * d + code_idx(p.q_idx, gi, p.ifmt, d)] = p.scale_log2 * load_val(p.q_val, gi, p.vfmt);
    }
  }

  const int r = tid >> 3, c8 = tid & 7;
  const int my_i = i0 + r;
  const bool row_ok = my_i < n;
  const bool win = p.window > 0;
  const int last_i = min(n, i0 + kGR) - 1;
  const int kend = p.causal ? last_i + 1 : n;
  auto allowed = [&](int j) {
    return row_ok && j < n && (!p.causal || j <= my_i) &&
           (!win || abs(my_i - j) < p.window || j < p.n_global || my_i < p.n_global);
  };

  float acc[kGNA];
#pragma unroll
  for (int a = 0; a < kGNA; ++a) acc[a] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  for (int j0 = 0; j0 < kend; j0 += kGC) {
    // a tile in the gap of the token window meets no row of the block
    if (win && i0 >= p.n_global && j0 >= p.n_global &&
        (j0 + kGC - 1 <= i0 - p.window || j0 >= last_i + p.window))
      continue;  // uniform per workgroup
    __syncthreads();  // the previous tile's readers are done
    for (int e = tid; e < kGC * k; e += kGT) {
      const int j = j0 + e / k;
      if (j < n) {
        const int64_t gi = (krow0 + j0) * k + e;
        Ki[e] = code_idx(p.k_idx, gi, p.ifmt, d);
        Kv[e] = load_val(p.k_val, gi, p.vfmt);
      } else {
        Ki[e] = 0;
        Kv[e] = 0.f;
      }
    }
    for (int x = tid; x < kGC * d; x += kGT) {
      const int j = j0 + x / d;
      const int64_t gv = (krow0 + j0) * d + x;
      Vs[x] = j >= n ? 0.f
                     : (p.vbf16 ? bf16_bits_to_f32(((const uint16_t*)p.v)[gv]) : ((const float*)p.v)[gv]);
    }
    __syncthreads();

    // scores of keys c8 + 8 m, as base-2 exponents; masked keys -inf
    float s[kGC / 8];
    float mt = -INFINITY;
#pragma unroll
    for (int m = 0; m < kGC / 8; ++m) {
      const int jj = c8 + 8 * m;
      float sc = 0.f;
      for (int t = 0; t < k; ++t) sc = fmaf(Kv[jj * k + t], Qd[r * d + Ki[jj * k + t]], sc);
      s[m] = allowed(j0 + jj) ? sc : -INFINITY;
      mt = fmaxf(mt, s[m]);
    }
    mt = row_max8(mt);
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;  // a row with nothing allowed yet
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int m = 0; m < kGC / 8; ++m) {
      const float pr = __builtin_amdgcn_exp2f(s[m] - m_use);
      Ps[r * (kGC + 1) + c8 + 8 * m] = pr;
      rs += pr;
    }
    l_run = l_run * alpha + row_sum8(rs);
    m_run = m_new;
#pragma unroll
    for (int a = 0; a < kGNA; ++a) acc[a] *= alpha;
    __syncthreads();  // the row's probabilities are written
    for (int jj = 0; jj < kGC; ++jj) {
      const float pr = Ps[r * (kGC + 1) + jj];
      const float* vr = Vs + jj * d;
#pragma unroll
      for (int a = 0; a < kGNA; ++a) {
        const int c = c8 + 8 * a;
        if (c < d) acc[a] = fmaf(pr, vr[c], acc[a]);
      }
    }
  }

  if (row_ok) {
    const float inv = 1.f / l_run;
    const int64_t orow = qrow0 + my_i;
#pragma unroll
    for (int a = 0; a < kGNA; ++a) {
      const int c = c8 + 8 * a;
      if (c < d) {
        const float x = acc[a] * inv;
        if (p.obf16) ((uint16_t*)p.o)[orow * d + c] = (uint16_t)f32_to_bf16_rne(x);
        else ((float*)p.o)[orow * d + c] = x;
      }
    }
    if (p.lse && c8 == 0) p.lse[orow] = (m_run + __log2f(l_run)) * kLn2;
  }
}

}  // namespace

bool fwd_generic_supported(int d, int k) {
  return d >= 1 && d <= kGDmax && k >= 1 && k <= d && generic_lds_bytes(d, k) <= 160 * 1024;
}

hipError_t launch_attn_fwd_generic(const void* q_idx, const void* q_val, const void* k_idx,
                                   const void* k_val, const void* v, int B, int Hq, int Hkv,
                                   int n, int d, int k, int causal, int window, int n_global,
                                   float scale, int ifmt, int vfmt, int vbf16, int obf16, void* o,
                                   float* lse, hipStream_t stream) {
  GenParams p;
  p.q_idx = q_idx; p.q_val = q_val; p.k_idx = k_idx; p.k_val = k_val; p.v = v;
  p.o = o; p.lse = lse;
  p.Hq = Hq; p.Hkv = Hkv; p.n = n; p.d = d; p.k = k;
  p.causal = causal; p.window = window; p.n_global = n_global;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);
  p.ifmt = ifmt; p.vfmt = vfmt; p.vbf16 = vbf16; p.obf16 = obf16;
  p.nqb = (n + kGR - 1) / kGR;
  const size_t bytes = generic_lds_bytes(d, k);
  if (bytes > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)sfa_fwd_generic_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(sfa_fwd_generic_kernel, dim3(p.nqb, B * Hq), dim3(kGT), bytes, stream, p);
  return hipGetLastError();
}

}  // namespace sfa
