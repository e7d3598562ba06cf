// Fresh-token encoding and append for gfx950 (patch prefill and decode steps,
// Sec. 4.2, Eq. 6).  One block per token: the block reads the D/2 cos/sin of
// its position from the cache's rotary table (LDS), then its lanes turn every rotary pair of the
// token's query and key heads and store
//   - the key (rounded to storage) and the value into the cache slot of the
//     token's position in this layer,
//   - the query (rounded to storage) into the query workspace [Hkv][rows][D],
//     row rank * g + (hq % g) of kv head hq / g, where the attention kernels
//     read it.
#include "fcg_device.hpp"
#include "kernels.hpp"

namespace fcg {

template <typename T, int D>
__global__ void __launch_bounds__(256) rope_append_kernel(const TokenMeta* __restrict__ meta,
                                                          const T* __restrict__ q, const T* __restrict__ k,
                                                          const T* __restrict__ v, CacheView cv, int layer,
                                                          const float2* __restrict__ rope, int Hq,
                                                          int rows_ws, T* __restrict__ qws) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int HALF = D / 2;
  constexpr int KT = HALF / VEC;
  constexpr int VT = D / VEC;
  __shared__ float s_cos[HALF], s_sin[HALF];

  const int r = blockIdx.x;
  const int t = threadIdx.x;
  const TokenMeta m = meta[r];
  const int Hkv = cv.n_kv_heads;
  const int g = Hq / Hkv;
  T* ck = reinterpret_cast<T*>(cv.k);
  T* cvv = reinterpret_cast<T*>(cv.v);
  const int n_q = Hq * KT, n_k = Hkv * KT, n_v = Hkv * VT;
  const int total = n_q + n_k + n_v;
  // item i: a q or k rotary chunk (i < n_q + n_k) or a v chunk; the source of
  // each item (both halves of a rotary pair) is loaded before the rotary table
  // is built, so the two latencies overlap
  auto src_of = [&](int i, const T** p) -> bool {  // -> is a rotary item
    if (i < n_q + n_k) {
      const bool is_q = i < n_q;
      const int ii = is_q ? i : i - n_q;
      const int head = ii / KT, c = ii % KT;
      *p = (is_q ? q + ((int64_t)m.tok * Hq + head) * D : k + ((int64_t)m.tok * Hkv + head) * D) + c * VEC;
      return true;
    }
    const int ii = i - n_q - n_k;
    *p = v + ((int64_t)m.tok * Hkv + ii / VT) * D + (ii % VT) * VEC;
    return false;
  };
  auto finish = [&](int i, const uint4& a, const uint4& b) {
    if (i < n_q + n_k) {
      const bool is_q = i < n_q;
      const int ii = is_q ? i : i - n_q;
      const int head = ii / KT, c = ii % KT;
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Store<T>::unpack(a, x1);
      Store<T>::unpack(b, x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float cs = s_cos[c * VEC + e], sn = s_sin[c * VEC + e];
        y1[e] = fmaf(x1[e], cs, -x2[e] * sn);
        y2[e] = fmaf(x2[e], cs, x1[e] * sn);
      }
      T* dst = is_q ? qws + ((int64_t)(head / g) * rows_ws + (int64_t)r * g + head % g) * D
                    : ck + cache_offset(cv, layer, m.seq, head, m.pos);
      st16(dst + c * VEC, Store<T>::pack(y1));
      st16(dst + HALF + c * VEC, Store<T>::pack(y2));
    } else {
      const int ii = i - n_q - n_k;
      st16(cvv + cache_offset(cv, layer, m.seq, ii / VT, m.pos) + (ii % VT) * VEC, a);
    }
  };
  constexpr int PRE = 3;  // items per lane loaded up front (all of them up to 64 query heads at D 128)
  uint4 pa[PRE], pb[PRE];
#pragma unroll
  for (int p = 0; p < PRE; ++p) {
    const int i = t + p * 256;
    if (i < total) {
      const T* src;
      const bool rot = src_of(i, &src);
      pa[p] = ld16(src);
      pb[p] = rot ? ld16(src + HALF) : pa[p];
    }
  }
  const float2 cs = rope[(int64_t)m.pos * HALF + t % HALF];  // (cos, sin) of the token's position
  if (t < HALF) {
    s_cos[t] = cs.x;
    s_sin[t] = cs.y;
  }
  __syncthreads();
#pragma unroll
  for (int p = 0; p < PRE; ++p) {
    const int i = t + p * 256;
    if (i < total) finish(i, pa[p], pb[p]);
  }
  for (int i = t + PRE * 256; i < total; i += 256) {
    const T* src;
    const bool rot = src_of(i, &src);
    const uint4 a = ld16(src);
    finish(i, a, rot ? ld16(src + HALF) : a);
  }
}

int launch_rope_append(int dtype, const TokenMeta* meta, int n, const void* q, const void* k, const void* v,
                       const CacheView& cv, int layer, const float2* rope, int Hq, void* qws, hipStream_t s, KTime tm) {
  if (n == 0) return 0;
  const int rows_ws = n * (Hq / cv.n_kv_heads);
#define RA(T, DD)                                                                                          \
  hipExtLaunchKernelGGL((rope_append_kernel<T, DD>), dim3(n), dim3(256), 0, s, tm.start, tm.stop, 0, meta, (const T*)q, (const T*)k, \
                     (const T*)v, cv, layer, rope, Hq, rows_ws, (T*)qws)
  if (dtype == 0) { if (cv.head_dim == 64) RA(float, 64); else RA(float, 128); }
  else { if (cv.head_dim == 64) RA(bf16_t, 64); else RA(bf16_t, 128); }
#undef RA
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

// (cos, sin) of p * w_i for every position p < n_pos and pair i < half: the
// float64 angle and float64 cos/sin of the definition, rounded to fp32 (the
// same values a kernel computing them itself would use)
__global__ void __launch_bounds__(256) rope_table_kernel(const double* __restrict__ inv_freq, int half, int64_t n,
                                                         float2* __restrict__ tab) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= n) return;
  const int64_t p = idx / half;
  const int i = (int)(idx % half);
  float c, sn;
  rope_cs((double)p, inv_freq[i], &c, &sn);
  tab[idx] = make_float2(c, sn);
}

int launch_rope_table(const double* inv_freq, int half, int n_pos, float2* tab, hipStream_t s) {
  const int64_t n = (int64_t)n_pos * half;
  if (n == 0) return 0;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, inv_freq, half, n, tab);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
