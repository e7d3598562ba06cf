// Fresh-token encoding and append for gfx950 (patch prefill and decode steps,
// Sec. 4.2, Eq. 6).  One block per token: the block computes the D/2 cos/sin
// of its position once (LDS), then its lanes turn every rotary pair of the
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
                                                          const double* __restrict__ inv_freq, int Hq,
                                                          int rows_ws, T* __restrict__ qws) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int HALF = D / 2;
  constexpr int KT = HALF / VEC;
  constexpr int VT = D / VEC;
  __shared__ float s_cos[HALF], s_sin[HALF];

  const int r = blockIdx.x;
  const TokenMeta m = meta[r];
  const int Hkv = cv.n_kv_heads;
  const int g = Hq / Hkv;
  if (threadIdx.x < HALF) rope_cs((double)m.pos, inv_freq[threadIdx.x], &s_cos[threadIdx.x], &s_sin[threadIdx.x]);
  __syncthreads();

  T* ck = reinterpret_cast<T*>(cv.k);
  T* cvv = reinterpret_cast<T*>(cv.v);
  const int n_q = Hq * KT, n_k = Hkv * KT, n_v = Hkv * VT;
  for (int i = threadIdx.x; i < n_q + n_k + n_v; i += blockDim.x) {
    if (i < n_q + n_k) {
      const bool is_q = i < n_q;
      const int ii = is_q ? i : i - n_q;
      const int head = ii / KT, c = ii % KT;
      const T* src = is_q ? q + ((int64_t)m.tok * Hq + head) * D : k + ((int64_t)m.tok * Hkv + head) * D;
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Store<T>::unpack(ld16(src + c * VEC), x1);
      Store<T>::unpack(ld16(src + HALF + c * VEC), x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float cs = s_cos[c * VEC + e], sn = s_sin[c * VEC + e];
        y1[e] = fmaf(x1[e], cs, -x2[e] * sn);
        y2[e] = fmaf(x2[e], cs, x1[e] * sn);
      }
      T* dst;
      if (is_q) {
        const int hk = head / g, j = head % g;
        dst = qws + ((int64_t)hk * rows_ws + (int64_t)r * g + j) * D;
      } else {
        dst = ck + cache_offset(cv, layer, m.seq, head, m.pos);
      }
      st16(dst + c * VEC, Store<T>::pack(y1));
      st16(dst + HALF + c * VEC, Store<T>::pack(y2));
    } else {
      const int ii = i - n_q - n_k;
      const int head = ii / VT, c = ii % VT;
      const int64_t off = cache_offset(cv, layer, m.seq, head, m.pos);
      st16(cvv + off + c * VEC, ld16(v + ((int64_t)m.tok * Hkv + head) * D + c * VEC));
    }
  }
}

int launch_rope_append(int dtype, const TokenMeta* meta, int n, const void* q, const void* k, const void* v,
                       const CacheView& cv, int layer, const double* inv_freq, int Hq, void* qws, hipStream_t s, KTime tm) {
  if (n == 0) return 0;
  const int rows_ws = n * (Hq / cv.n_kv_heads);
#define RA(T, DD)                                                                                          \
  hipExtLaunchKernelGGL((rope_append_kernel<T, DD>), dim3(n), dim3(256), 0, s, tm.start, tm.stop, 0, meta, (const T*)q, (const T*)k, \
                     (const T*)v, cv, layer, inv_freq, Hq, rows_ws, (T*)qws)
  if (dtype == 0) { if (cv.head_dim == 64) RA(float, 64); else RA(float, 128); }
  else { if (cv.head_dim == 64) RA(bf16_t, 64); else RA(bf16_t, 128); }
#undef RA
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
