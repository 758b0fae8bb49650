// KV-cache maintenance for SFA decode (App. B: generation appends one coded
// key and its value per token to a cache of sparse key codes and dense V).
//
// sfa_kv_append_kernel: one wavefront per new (sequence, KV head, token) row
// at a time.
// The key row is coded with the same exact Top-k selection as the coding
// kernel (Sec. 3.1, Eqs. (3)-(4)) and written, with the value row, at the
// token's position seq_len[b] + t: in a contiguous cache [B, Hkv, P, ...] at
// row (b, h, position), in a paged one through the block table (page
// table[b][position / P], slot position % P).  Positions past the capacity
// and pages outside the pool are not written.
// sfa_kv_advance_kernel: seq_len[b] += appended count, clamped to the
// capacity; it runs after the append on the same stream, so every append
// wave reads the old length.
// 8-bit cache (SFA with 8-bit activations, App. E "SFA (quant)"): the kept
// code values and the value row are each quantised as one row, s = max|x| /
// 127 and q = round-half-even(x / s) in [-127, 127] (float32 divisions,
// correctly rounded), stored as int8 with s per row.
#include "sfa_device.h"
#include "sfa_launch.h"
#include "sfa_topk.h"

namespace sfa {

__device__ __forceinline__ int appended_count(const int32_t* n_new, int b, int T) {
  if (!n_new) return T;
  const int c = n_new[b];
  return c < 0 ? 0 : (c > T ? T : c);
}

// Grid: y strides over the B * Hkv (sequence, KV head) pairs, x over the
// pair's tokens, one wavefront per token row, the next row's key and value
// loads in flight while the current one is selected and stored.  Everything
// that depends only on the pair (its length, count, capacity) is read once;
// a token's page and slot are a shift and a mask (power-of-two pages).
// E: coordinates per lane (d <= 64 * E).  COMMON: int16 / bf16 codes, bf16
// values in and in the cache, as compile-time constants (the stores then
// carry no format dispatch); else the formats are read from the arguments.
// Q8: the 8-bit cache (index format from the arguments).
template <int E, bool COMMON, bool Q8 = false>
__global__ __launch_bounds__(256) void sfa_kv_append_kernel(AppendArgs a) {
  static_assert(!(COMMON && Q8), "the 8-bit cache has its own formats");
  const int lane = threadIdx.x & 63;
  const int ifmt = COMMON ? (int)kIdxI16 : a.ifmt, vfmt = COMMON ? (int)kValBF16 : a.vfmt;
  const bool vin_bf16 = COMMON || a.vin_bf16, vc_bf16 = COMMON || a.vc_bf16;
  const int tw = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tstride = gridDim.x * 4;
  const int64_t cap = a.table ? (int64_t)a.max_pages * a.page_size : a.page_size;
  for (int bh = blockIdx.y; bh < a.B * a.Hkv; bh += gridDim.y) {
    const int b = bh / a.Hkv, h = bh - b * a.Hkv;
    int64_t L0 = a.seq_len[b];
    L0 = L0 < 0 ? 0 : (L0 > cap ? cap : L0);
    // tokens written: t < count, and positions below the capacity
    const int tend = (int)min((int64_t)appended_count(a.n_new, b, a.T), cap - L0);
    if (tw >= tend) continue;  // uniform per wave
    const float* kbase = a.k_new + (int64_t)bh * a.T * a.d;
    const unsigned char* vbase =
        (const unsigned char*)a.v_new + (int64_t)bh * a.T * a.d * (vin_bf16 ? 2 : 4);

    // raw 32-bit words: key bits, and value bits (bf16 zero-extended or
    // float); and the row's page, loaded with them so that the wait for it
    // does not also wait for the next row's loads (loads retire in order)
    uint32_t nk[E], nv[E];
    int npage = 0;
    auto load_row = [&](int t) {
      if (a.table) npage = a.table[(int64_t)b * a.max_pages + ((L0 + t) >> a.log2P)];
      const int64_t o = (int64_t)t * a.d;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int c = min(lane + 64 * e, a.d - 1);
        nk[e] = __float_as_uint(kbase[o + c]);
        nv[e] = vin_bf16 ? (uint32_t)((const uint16_t*)vbase)[o + c]
                           : ((const uint32_t*)vbase)[o + c];
      }
    };
    load_row(tw);
    for (int t = tw; t < tend; t += tstride) {
      uint32_t bits[E], vb[E], key[E];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        bits[e] = nk[e];
        vb[e] = nv[e];
        key[e] = topk_key(bits[e], lane + 64 * e < a.d);
      }
      const int row_page = __builtin_amdgcn_readfirstlane(npage);
      if (t + tstride < tend) load_row(t + tstride);
      const int64_t pos = L0 + t;
      int64_t page = b, slot = pos;
      if (a.table) {
        page = row_page;
        slot = pos & (a.page_size - 1);
        if (page < 0 || page >= a.num_pages) continue;  // uniform per wave
      }
      const int64_t crow = (page * a.Hkv + h) * a.page_size + slot;

      bool sel[E];
      topk_select<E>(key, a.k, sel);
      int sl[E];
      topk_slots<E>(sel, sl);
      if constexpr (Q8) {
        // the kept values' largest magnitude is the row's largest: the
        // largest key, |bits| + 1
        uint32_t km = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) km = max(km, key[e]);
        const float ks = __uint_as_float(wave_umax(km) - 1u) / 127.f;
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (sel[e] && sl[e] < a.k) {
            const int64_t at = crow * a.k + sl[e];
            const int u = lane + 64 * e;
            if (ifmt == kIdxI16) ((int16_t*)a.kc_idx)[at] = (int16_t)u;
            else if (ifmt == kIdxU8) ((uint8_t*)a.kc_idx)[at] = (uint8_t)u;
            else ((int32_t*)a.kc_idx)[at] = u;
            const float qf = ks > 0.f ? rintf(__uint_as_float(bits[e]) / ks) : 0.f;
            ((int8_t*)a.kc_val)[at] = (int8_t)(int)fminf(fmaxf(qf, -127.f), 127.f);
          }
        if (lane == 0) a.kc_scale[crow] = ks;
        // the value row
        float vf[E];
        uint32_t vm = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const bool in = lane + 64 * e < a.d;
          vf[e] = in ? (vin_bf16 ? bf16_bits_to_f32(vb[e]) : __uint_as_float(vb[e])) : 0.f;
          vm = max(vm, __float_as_uint(vf[e]) & 0x7fffffffu);
        }
        const float vs = __uint_as_float(wave_umax(vm)) / 127.f;
        const int64_t vo = crow * a.d;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int c = lane + 64 * e;
          if (c < a.d) {
            const float qf = vs > 0.f ? rintf(vf[e] / vs) : 0.f;
            ((int8_t*)a.v_cache)[vo + c] = (int8_t)(int)fminf(fmaxf(qf, -127.f), 127.f);
          }
        }
        if (lane == 0) a.v_scale[crow] = vs;
        continue;
      }
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (sel[e] && sl[e] < a.k)
          store_code(a.kc_idx, a.kc_val, crow * a.k + sl[e], lane + 64 * e, bits[e], ifmt,
                     vfmt);
      // value row (bf16 cache from float32 values: round to nearest even)
      const int64_t vo = crow * a.d;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int c = lane + 64 * e;
        if (c < a.d) {
          if (vc_bf16)
            ((uint16_t*)a.v_cache)[vo + c] =
                vin_bf16 ? (uint16_t)vb[e] : (uint16_t)f32_to_bf16_rne(__uint_as_float(vb[e]));
          else
            ((uint32_t*)a.v_cache)[vo + c] = vin_bf16 ? vb[e] << 16 : vb[e];
        }
      }
    }
  }
}

__global__ void sfa_kv_advance_kernel(int32_t* seq_len, const int32_t* n_new, int B, int T,
                                      int64_t cap) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int64_t L = seq_len[b];
  L = L < 0 ? 0 : (L > cap ? cap : L);
  L += appended_count(n_new, b, T);
  seq_len[b] = (int32_t)(L > cap ? cap : L);
}

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t stream) {
  const int64_t rows = (int64_t)a.B * a.Hkv * a.T;
  if (rows > 0) {
    // about 2048 workgroups of 4 waves (8 per compute unit) over the pairs
    const int pairs = a.B * a.Hkv;
    const int gy = pairs < 65535 ? pairs : 65535;
    int gx = (2048 + gy - 1) / gy;
    const int gx_need = (a.T + 3) / 4;
    if (gx > gx_need) gx = gx_need;
    dim3 grid(gx, gy), block(256);
    const bool common =
        !a.q8 && a.ifmt == kIdxI16 && a.vfmt == kValBF16 && a.vin_bf16 && a.vc_bf16;
    auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, grid, block, 0, stream, a); };
    if (a.q8) {
      if (a.d <= 64) go(sfa_kv_append_kernel<1, false, true>);
      else if (a.d <= 128) go(sfa_kv_append_kernel<2, false, true>);
      else go(sfa_kv_append_kernel<4, false, true>);
    } else if (a.d <= 64) {
      common ? go(sfa_kv_append_kernel<1, true>) : go(sfa_kv_append_kernel<1, false>);
    } else if (a.d <= 128) {
      common ? go(sfa_kv_append_kernel<2, true>) : go(sfa_kv_append_kernel<2, false>);
    } else {
      common ? go(sfa_kv_append_kernel<4, true>) : go(sfa_kv_append_kernel<4, false>);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t cap = a.table ? (int64_t)a.max_pages * a.page_size : a.page_size;
  hipLaunchKernelGGL(sfa_kv_advance_kernel, dim3((a.B + 255) / 256), dim3(256), 0, stream,
                     a.seq_len, a.n_new, a.B, a.T, cap);
  return hipGetLastError();
}

}  // namespace sfa
