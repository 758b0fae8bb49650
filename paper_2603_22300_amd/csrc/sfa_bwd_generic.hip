// SFA backward with the straight-through estimator (Sec. 3.1, Eq. (6)) for
// head dimensions without the matrix-core kernels: any d <= 256 other than
// 64 and 128, float32 arithmetic, no workspace.
//
// With P_ij = exp2(s_ij log2(e) - LSE_i log2(e)) recomputed from the
// forward's LSE, D_i = dO_i . O_i and dS_ij = P_ij (dO_i . v_j - D_i):
//   dq_val[i][t] = scale sum_j dS_ij k~_j[q_idx[i][t]]
//   dk_val[j][t] = scale sum_i dS_ij q~_i[k_idx[j][t]]
//   dv[j]        = sum_i P_ij dO_i
// Two kernels, each output element owned by one thread (no atomics):
//   sfa_bwd_generic_dq_kernel:  16 query rows of one head; key tiles of 32
//     keys densified in LDS; 16 threads per row (2 keys each for the
//     scores, every 16th support slot for dq);
//   sfa_bwd_generic_dkv_kernel: 16 keys of one KV head; query tiles of 32
//     rows of each query head of the group densified in LDS; 16 threads per
//     key (2 queries each, every 16th dimension of dv, every 16th support
//     slot of dk).
// Scores are the overlap sums of one side's codes against the other side's
// densified rows: k lookups per pair.
#include "sfa_device.h"
#include "sfa_launch.h"

namespace sfa {
namespace {

constexpr int kBR = 16;   // rows (dq) or keys (dkv) per workgroup
constexpr int kBT = 32;   // partner tile: keys (dq) or query rows (dkv)
constexpr int kBThr = 256;
constexpr int kBDmax = 256;
constexpr int kBS = kBDmax / 16;  // slots / dimensions per thread, at most

struct GBwdParams {
  const void *q_idx, *q_val, *k_idx, *k_val, *v, *o, *dout;
  const float* lse;
  float *dq, *dk, *dv;
  int Hq, Hkv, n, d, k, G, causal, window, n_global;
  float scale, scale_log2;
  int ifmt, vfmt, vbf16, obf16;
};

__device__ __forceinline__ int gb_idx(const void* p, int64_t i, int ifmt, int d) {
  const int u = load_idx(p, i, ifmt, -1);
  return u < 0 ? 0 : (u >= d ? d - 1 : u);
}

__device__ __forceinline__ float gb_val16(const void* p, int64_t i, int bf16) {
  return bf16 ? bf16_bits_to_f32(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}

__device__ __forceinline__ float sum16(float x) {
  x += __shfl_xor(x, 1, 64);
  x += __shfl_xor(x, 2, 64);
  x += __shfl_xor(x, 4, 64);
  return x + __shfl_xor(x, 8, 64);
}

__device__ __forceinline__ bool gb_allowed(const GBwdParams& p, int i, int j) {
  return i < p.n && j < p.n && (!p.causal || j <= i) &&
         (p.window <= 0 || abs(i - j) < p.window || j < p.n_global || i < p.n_global);
}

// LDS sizes (floats): dq kernel: codes 2 [kBR][k], dO [kBR][d], K~ and V
// [kBT][d], dS [kBR][kBT + 1], L2 and D [kBR]
__host__ __device__ constexpr size_t gbq_floats(int d, int k) {
  return 2 * (size_t)kBR * k + (size_t)kBR * d + 2 * (size_t)kBT * d + kBR * (kBT + 1) + 2 * kBR;
}
// dkv kernel: codes 2 [kBR][k], V [kBR][d], Q~ and dO [kBT][d], P and dS
// [kBR][kBT + 1] each, L2 and D [kBT]
__host__ __device__ constexpr size_t gbk_floats(int d, int k) {
  return 2 * (size_t)kBR * k + (size_t)kBR * d + 2 * (size_t)kBT * d + 2 * kBR * (kBT + 1) +
         2 * kBT;
}

__global__ __launch_bounds__(kBThr) void sfa_bwd_generic_dq_kernel(GBwdParams p) {
  extern __shared__ __attribute__((aligned(16))) float gq[];
  const int d = p.d, k = p.k, n = p.n;
  int* Qi = (int*)gq;                       // [kBR][k]
  float* Qv = gq + kBR * k;                 // [kBR][k]
  float* dOs = Qv + kBR * k;                // [kBR][d]
  float* Kd = dOs + kBR * d;                // [kBT][d] densified key codes
  float* Vs = Kd + kBT * d;                 // [kBT][d]
  float* dS = Vs + kBT * d;                 // [kBR][kBT + 1]
  float* L2 = dS + kBR * (kBT + 1);         // [kBR]
  float* Dr = L2 + kBR;                     // [kBR]

  const int tid = threadIdx.x, r = tid >> 4, c16 = tid & 15;
  const int b = blockIdx.y / p.Hq, hq = blockIdx.y - b * p.Hq, hkv = hq / p.G;
  const int i0 = ((int)gridDim.x - 1 - (int)blockIdx.x) * kBR;  // longest causal blocks first
  const int64_t qrow0 = ((int64_t)b * p.Hq + hq) * n;
  const int64_t krow0 = ((int64_t)b * p.Hkv + hkv) * n;
  const int my_i = i0 + r;
  const bool row_ok = my_i < n;

  for (int e = tid; e < kBR * k; e += kBThr) {
    const int rr = e / k, i = i0 + rr;
    const int64_t gi = (qrow0 + min(i, n - 1)) * k + (e - rr * k);
    Qi[e] = gb_idx(p.q_idx, gi, p.ifmt, d);
    Qv[e] = i < n ? load_val(p.q_val, gi, p.vfmt) : 0.f;
  }
  for (int x = tid; x < kBR * d; x += kBThr) {
    const int i = i0 + x / d;
    dOs[x] = i < n ? gb_val16(p.dout, qrow0 * d + (int64_t)i0 * d + x, p.obf16) : 0.f;
  }
  __syncthreads();
  // D_i = dO_i . O_i by the row's 16 threads
  float dpart = 0.f;
  for (int c = c16; c < d; c += 16)
    if (row_ok) dpart = fmaf(dOs[r * d + c], gb_val16(p.o, (qrow0 + my_i) * d + c, p.obf16), dpart);
  dpart = sum16(dpart);
  if (c16 == 0) {
    Dr[r] = dpart;
    L2[r] = row_ok ? p.lse[qrow0 + my_i] * 1.4426950408889634f : INFINITY;
  }

  float dq[kBS];
#pragma unroll
  for (int m = 0; m < kBS; ++m) dq[m] = 0.f;
  const int last = min(n, i0 + kBR) - 1;
  const int kend = p.causal ? last + 1 : n;
  const bool win = p.window > 0;
  for (int j0 = 0; j0 < kend; j0 += kBT) {
    if (win && i0 >= p.n_global && j0 >= p.n_global &&
        (j0 + kBT - 1 <= i0 - p.window || j0 >= last + p.window))
      continue;  // a tile in the gap of the window: uniform per workgroup
    __syncthreads();  // previous tile's readers done
    for (int x = tid; x < kBT * d; x += kBThr) {
      Kd[x] = 0.f;
      const int j = j0 + x / d;
      Vs[x] = j < n ? gb_val16(p.v, (krow0 + j0) * d + x, p.vbf16) : 0.f;
    }
    __syncthreads();
    for (int e = tid; e < kBT * k; e += kBThr) {
      const int j = j0 + e / k;
      if (j < n) {
        const int64_t gi = (krow0 + j0) * k + e;
        Kd[(e / k) * d + gb_idx(p.k_idx, gi, p.ifmt, d)] = load_val(p.k_val, gi, p.vfmt);
      }
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < kBT / 16; ++m) {
      const int jj = c16 + 16 * m, j = j0 + jj;
      float ds = 0.f;
      if (row_ok && gb_allowed(p, my_i, j)) {
        float s = 0.f;
        for (int t = 0; t < k; ++t) s = fmaf(Qv[r * k + t], Kd[jj * d + Qi[r * k + t]], s);
        const float pr = __builtin_amdgcn_exp2f(s * p.scale_log2 - L2[r]);
        float dp = 0.f;
        for (int c = 0; c < d; ++c) dp = fmaf(dOs[r * d + c], Vs[jj * d + c], dp);
        ds = pr * (dp - Dr[r]);
      }
      dS[r * (kBT + 1) + jj] = ds;
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < kBS; ++m) {
      const int t = c16 + 16 * m;
      if (t < k) {
        const int u = Qi[r * k + t];
        float a = dq[m];
        for (int jj = 0; jj < kBT; ++jj) a = fmaf(dS[r * (kBT + 1) + jj], Kd[jj * d + u], a);
        dq[m] = a;
      }
    }
  }
  if (row_ok) {
#pragma unroll
    for (int m = 0; m < kBS; ++m) {
      const int t = c16 + 16 * m;
      if (t < k) p.dq[(qrow0 + my_i) * k + t] = p.scale * dq[m];
    }
  }
}

__global__ __launch_bounds__(kBThr) void sfa_bwd_generic_dkv_kernel(GBwdParams p) {
  extern __shared__ __attribute__((aligned(16))) float gk[];
  const int d = p.d, k = p.k, n = p.n;
  int* Ki = (int*)gk;                       // [kBR][k]
  float* Kv = gk + kBR * k;                 // [kBR][k]
  float* Vk = Kv + kBR * k;                 // [kBR][d] my keys' values
  float* Qd = Vk + kBR * d;                 // [kBT][d] densified query codes
  float* dOt = Qd + kBT * d;                // [kBT][d]
  float* Pt = dOt + kBT * d;                // [kBR][kBT + 1]
  float* dSt = Pt + kBR * (kBT + 1);        // [kBR][kBT + 1]
  float* L2 = dSt + kBR * (kBT + 1);        // [kBT]
  float* Dq = L2 + kBT;                     // [kBT]

  const int tid = threadIdx.x, jr = tid >> 4, c16 = tid & 15;
  const int b = blockIdx.y / p.Hkv, hkv = blockIdx.y - b * p.Hkv;
  const int j0 = blockIdx.x * kBR;
  const int64_t krow0 = ((int64_t)b * p.Hkv + hkv) * n;
  const int my_j = j0 + jr;
  const bool key_ok = my_j < n;

  for (int e = tid; e < kBR * k; e += kBThr) {
    const int rr = e / k, j = j0 + rr;
    const int64_t gi = (krow0 + min(j, n - 1)) * k + (e - rr * k);
    Ki[e] = gb_idx(p.k_idx, gi, p.ifmt, d);
    Kv[e] = j < n ? load_val(p.k_val, gi, p.vfmt) : 0.f;
  }
  for (int x = tid; x < kBR * d; x += kBThr) {
    const int j = j0 + x / d;
    Vk[x] = j < n ? gb_val16(p.v, (krow0 + j0) * d + x, p.vbf16) : 0.f;
  }

  float dv[kBS], dk[kBS];
#pragma unroll
  for (int m = 0; m < kBS; ++m) { dv[m] = 0.f; dk[m] = 0.f; }
  const int jlast = min(n, j0 + kBR) - 1;
  const bool win = p.window > 0;
  // query rows that can see a key of this block: i >= j0 when causal
  const int ibeg = p.causal ? (j0 / kBT) * kBT : 0;
  for (int h = 0; h < p.G; ++h) {
    const int hq = hkv * p.G + h;
    const int64_t qrow0 = ((int64_t)b * p.Hq + hq) * n;
    for (int i0 = ibeg; i0 < n; i0 += kBT) {
      const int ilast = min(n, i0 + kBT) - 1;
      // no query row of the tile sees a key of the block (window gap)
      if (win && j0 >= p.n_global && i0 >= p.n_global &&
          (i0 >= jlast + p.window || ilast <= j0 - p.window))
        continue;  // uniform per workgroup
      __syncthreads();  // previous tile's readers done
      for (int x = tid; x < kBT * d; x += kBThr) {
        Qd[x] = 0.f;
        const int i = i0 + x / d;
        dOt[x] = i < n ? gb_val16(p.dout, (qrow0 + i0) * d + x, p.obf16) : 0.f;
      }
      __syncthreads();
      for (int e = tid; e < kBT * k; e += kBThr) {
        const int i = i0 + e / k;
        if (i < n) {
          const int64_t gi = (qrow0 + i0) * k + e;
          Qd[(e / k) * d + gb_idx(p.q_idx, gi, p.ifmt, d)] = load_val(p.q_val, gi, p.vfmt);
        }
      }
      // D_i = dO_i . O_i and L2_i, 8 threads per query row
      {
        const int ii = tid >> 3, c8 = tid & 7, i = i0 + ii;
        float dpart = 0.f;
        if (i < n)
          for (int c = c8; c < d; c += 8)
            dpart = fmaf(dOt[ii * d + c], gb_val16(p.o, (qrow0 + i) * d + c, p.obf16), dpart);
        dpart += __shfl_xor(dpart, 1, 64);
        dpart += __shfl_xor(dpart, 2, 64);
        dpart += __shfl_xor(dpart, 4, 64);
        if (c8 == 0) {
          Dq[ii] = dpart;
          L2[ii] = i < n ? p.lse[qrow0 + i] * 1.4426950408889634f : INFINITY;
        }
      }
      __syncthreads();
#pragma unroll
      for (int m = 0; m < kBT / 16; ++m) {
        const int ii = c16 + 16 * m, i = i0 + ii;
        float pr = 0.f, ds = 0.f;
        if (key_ok && gb_allowed(p, i, my_j)) {
          float s = 0.f;
          for (int t = 0; t < k; ++t) s = fmaf(Kv[jr * k + t], Qd[ii * d + Ki[jr * k + t]], s);
          pr = __builtin_amdgcn_exp2f(s * p.scale_log2 - L2[ii]);
          float dp = 0.f;
          for (int c = 0; c < d; ++c) dp = fmaf(dOt[ii * d + c], Vk[jr * d + c], dp);
          ds = pr * (dp - Dq[ii]);
        }
        Pt[jr * (kBT + 1) + ii] = pr;
        dSt[jr * (kBT + 1) + ii] = ds;
      }
      __syncthreads();
#pragma unroll
      for (int m = 0; m < kBS; ++m) {
        const int c = c16 + 16 * m;
        if (c < d) {
          float a = dv[m];
          for (int ii = 0; ii < kBT; ++ii) a = fmaf(Pt[jr * (kBT + 1) + ii], dOt[ii * d + c], a);
          dv[m] = a;
        }
        if (c < k) {
          const int u = Ki[jr * k + c];
          float a = dk[m];
          for (int ii = 0; ii < kBT; ++ii) a = fmaf(dSt[jr * (kBT + 1) + ii], Qd[ii * d + u], a);
          dk[m] = a;
        }
      }
    }
  }
  if (key_ok) {
#pragma unroll
    for (int m = 0; m < kBS; ++m) {
      const int c = c16 + 16 * m;
      if (c < d) p.dv[(krow0 + my_j) * d + c] = dv[m];
      if (c < k) p.dk[(krow0 + my_j) * k + c] = p.scale * dk[m];
    }
  }
}

}  // namespace

bool bwd_generic_supported(int d, int k) {
  return d >= 1 && d <= kBDmax && k >= 1 && k <= d &&
         sizeof(float) * gbq_floats(d, k) <= 160 * 1024 &&
         sizeof(float) * gbk_floats(d, k) <= 160 * 1024;
}

hipError_t launch_attn_bwd_generic(const void* q_idx, const void* q_val, const void* k_idx,
                                   const void* k_val, const void* v, const void* o,
                                   const float* lse, const void* dout, int B, int Hq, int Hkv,
                                   int n, int d, int k, int causal, int window, int n_global,
                                   float scale, int ifmt, int vfmt, int vbf16, int obf16,
                                   float* dq, float* dk, float* dv, hipStream_t stream) {
  GBwdParams p;
  p.q_idx = q_idx; p.q_val = q_val; p.k_idx = k_idx; p.k_val = k_val; p.v = v; p.o = o;
  p.dout = dout; p.lse = lse; p.dq = dq; p.dk = dk; p.dv = dv;
  p.Hq = Hq; p.Hkv = Hkv; p.n = n; p.d = d; p.k = k; p.G = Hq / Hkv;
  p.causal = causal; p.window = window; p.n_global = n_global;
  p.scale = scale;
  p.scale_log2 = (float)((double)scale * 1.4426950408889634);
  p.ifmt = ifmt; p.vfmt = vfmt; p.vbf16 = vbf16; p.obf16 = obf16;
  const size_t bq = sizeof(float) * gbq_floats(d, k), bk = sizeof(float) * gbk_floats(d, k);
  if (bq > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)sfa_bwd_generic_dq_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bq);
    if (e != hipSuccess) return e;
  }
  if (bk > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)sfa_bwd_generic_dkv_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bk);
    if (e != hipSuccess) return e;
  }
  const int nb = (n + kBR - 1) / kBR;
  hipLaunchKernelGGL(sfa_bwd_generic_dq_kernel, dim3(nb, B * Hq), dim3(kBThr), bq, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sfa_bwd_generic_dkv_kernel, dim3(nb, B * Hkv), dim3(kBThr), bk, stream, p);
  return hipGetLastError();
}

}  // namespace sfa
