// One decode step at one layer for a batch of sequences, in a single launch
// (Sec. 4.2, Eq. 6: decoding over the reused, grafted KV states).
//
// Per sequence i the new token sits at position pos_i = its current length.
// Block (split s of sequence i, kv head h) attends the token's g query heads
// over key positions [s * split_keys, min(pos_i + 1, (s + 1) * split_keys)):
//   - it encodes the token's queries at pos_i (cos/sin of the position in
//     LDS, fp64 angle), rounds them to storage and pre-scales them by
//     log2(e) / sqrt(D) for a base-2 softmax;
//   - the block whose split holds pos_i also encodes the new key, stores key
//     and value into the cache slot and attends to them from registers; no
//     other block touches that slot;
//   - cached keys stream through 16-byte vector loads, LPK lanes per key,
//     U key steps (U * 256 / LPK keys) in flight per lane before any math;
//     scores are reduced across a key's lanes with DPP, and each lane keeps
//     an online softmax rescaled once per chunk of U steps;
//   - the block merges its key slots through LDS; a single-split sequence
//     writes its output, otherwise the block stores a partial (max, sum,
//     unnormalised output) that the combine kernel merges.  The merge is a
//     separate launch on purpose: merging in the last-arriving block needs a
//     device-scope release/acquire per block, which on gfx950 writes back
//     and invalidates the XCD's whole L2.
#include "fcg_device.hpp"
#include "kernels.hpp"

namespace fcg {

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

template <int LPK>
__device__ __forceinline__ float lanes_sum(float x) {
  if (LPK >= 2) x += dpp_f<0xB1>(x);   // quad_perm [1,0,3,2]
  if (LPK >= 4) x += dpp_f<0x4E>(x);   // quad_perm [2,3,0,1]
  if (LPK >= 8) x += dpp_f<0x141>(x);  // row_half_mirror
  if (LPK >= 16) x += dpp_f<0x140>(x); // row_mirror
  return x;
}

// Lane's rotated dims [d0, d0 + DPL) of a row x (storage T), encoded with the
// block's cos/sin table; rounded to storage and returned as fp32.
template <typename T, int D, int DPL>
__device__ __forceinline__ void encode_dims(const T* __restrict__ x, int d0, const float* s_cos, const float* s_sin,
                                            float* y) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int HALF = D / 2;
  float a[DPL], b[DPL];
  const int dp = d0 < HALF ? d0 + HALF : d0 - HALF;  // partner dims
#pragma unroll
  for (int nv = 0; nv < DPL / VEC; ++nv) {
    Store<T>::unpack(ld16(x + d0 + nv * VEC), a + nv * VEC);
    Store<T>::unpack(ld16(x + dp + nv * VEC), b + nv * VEC);
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) {
    const int i = (d0 + e) % HALF;
    const float c = s_cos[i], s = s_sin[i];
    // first half: x_i c - x_{i+D/2} s; second half: x_{i+D/2} c + x_i s
    const float r = d0 < HALF ? fmaf(a[e], c, -b[e] * s) : fmaf(a[e], c, b[e] * s);
    y[e] = Store<T>::round(r);
  }
}

template <typename T, int D, int G, bool PAGED>
__global__ void __launch_bounds__(256) decode_kernel(DecodeArgs args, const T* __restrict__ q,
                                                     const T* __restrict__ k, const T* __restrict__ v, CacheView cv,
                                                     int layer, const double* __restrict__ inv_freq,
                                                     T* __restrict__ out, float* __restrict__ part_o,
                                                     float* __restrict__ part_ml) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int NV = (D / VEC > 16) ? (D / VEC) / 16 : 1;
  constexpr int DPL = VEC * NV;
  constexpr int LPK = D / DPL;
  constexpr int SLOTS = 256 / LPK;
  constexpr int U = G >= 8 ? 4 : 8;
  constexpr int HALF = D / 2;
  __shared__ float s_cos[HALF], s_sin[HALF];
  __shared__ float s_m[SLOTS][G], s_l[SLOTS][G];
  __shared__ float s_o[SLOTS][DPL][LPK];
  __shared__ float s_M[G], s_L[G];

  // which sequence and split this block serves
  const int b = blockIdx.x;
  int i = 0;
  while (i + 1 < args.n && args.split0[i + 1] <= b) ++i;
  const int split = b - args.split0[i];
  const int nsplit = args.split0[i + 1] - args.split0[i];
  const int seq = args.seq[i], pos = args.pos[i];
  const int hk = blockIdx.y;
  const int Hkv = cv.n_kv_heads;
  const int Hq = Hkv * G;
  const int t = threadIdx.x;
  const int chunk = t % LPK, slot = t / LPK;
  const int d0 = chunk * DPL;
  const int k0 = split * args.split_keys;
  const int k1 = min(pos + 1, k0 + args.split_keys);
  const bool owns_new = k0 <= pos && pos < k1;

  if (t < HALF) rope_cs((double)pos, inv_freq[t], &s_cos[t], &s_sin[t]);
  __syncthreads();

  const float qscale = 1.4426950408889634f / sqrtf((float)D);
  float qf[G][DPL];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    encode_dims<T, D, DPL>(q + ((int64_t)i * Hq + hk * G + j) * D, d0, s_cos, s_sin, qf[j]);
#pragma unroll
    for (int e = 0; e < DPL; ++e) qf[j][e] *= qscale;
  }

  float mx[G], sm[G], o[G][DPL];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    mx[j] = -INFINITY;
    sm[j] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[j][e] = 0.f;
  }

  const T* ck = reinterpret_cast<const T*>(cv.k);
  const T* cvv = reinterpret_cast<const T*>(cv.v);
  const int kend = owns_new ? pos : k1;  // cached keys; the new one is handled below
  for (int base = k0; base < kend; base += U * SLOTS) {
    // raw 16-byte vectors, all U steps in flight before any math; keys past
    // the split re-read its last cached key (valid, scores masked)
    uint4 kr[U][NV], vr[U][NV];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int key = base + u * SLOTS + slot;
      ok[u] = key < kend;
      const int64_t off = kv_offset<PAGED>(cv, layer, seq, hk, min(key, kend - 1)) + d0;
#pragma unroll
      for (int nv = 0; nv < NV; ++nv) {
        kr[u][nv] = ld16(ck + off + nv * VEC);
        vr[u][nv] = ld16(cvv + off + nv * VEC);
      }
    }
    float s[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < G; ++j) {
        float kx[DPL];
#pragma unroll
        for (int nv = 0; nv < NV; ++nv) Store<T>::unpack(kr[u][nv], kx + nv * VEC);
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) a = fmaf(qf[j][e], kx[e], a);
        a = lanes_sum<LPK>(a);
        s[u][j] = ok[u] ? a : -INFINITY;
      }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      float cm = s[0][j];
#pragma unroll
      for (int u = 1; u < U; ++u) cm = fmaxf(cm, s[u][j]);
      const float mn = fmaxf(mx[j], cm);
      if (mn == -INFINITY) continue;  // nothing seen yet by this lane
      const float a = exp2f(mx[j] - mn);
      float acc_l = sm[j] * a;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] *= a;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = exp2f(s[u][j] - mn);  // 0 for masked keys (their values are finite)
        acc_l += p;
        float vx[DPL];
#pragma unroll
        for (int nv = 0; nv < NV; ++nv) Store<T>::unpack(vr[u][nv], vx + nv * VEC);
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(p, vx[e], o[j][e]);
      }
      sm[j] = acc_l;
      mx[j] = mn;
    }
  }
  if (owns_new && slot == 0) {
    // encode, store and attend the new token (lanes of slot 0)
    float kn[DPL], vn[DPL];
    encode_dims<T, D, DPL>(k + ((int64_t)i * Hkv + hk) * D, d0, s_cos, s_sin, kn);
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) Store<T>::unpack(ld16(v + ((int64_t)i * Hkv + hk) * D + d0 + nv * VEC), vn + nv * VEC);
    T* kdst = reinterpret_cast<T*>(cv.k) + kv_offset<PAGED>(cv, layer, seq, hk, pos) + d0;
    T* vdst = reinterpret_cast<T*>(cv.v) + kv_offset<PAGED>(cv, layer, seq, hk, pos) + d0;
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) {
      st16(kdst + nv * VEC, Store<T>::pack(kn + nv * VEC));
      st16(vdst + nv * VEC, Store<T>::pack(vn + nv * VEC));
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) a = fmaf(qf[j][e], kn[e], a);
      a = lanes_sum<LPK>(a);
      const float mn = fmaxf(mx[j], a);
      const float f = exp2f(mx[j] - mn), p = exp2f(a - mn);
      sm[j] = fmaf(sm[j], f, p);
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(o[j][e], f, p * vn[e]);
      mx[j] = mn;
    }
  }

  // merge the block's key slots
  if (chunk == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) { s_m[slot][j] = mx[j]; s_l[slot][j] = sm[j]; }
  }
  __syncthreads();
  if (t < G) {
    float M = -INFINITY;
    for (int s2 = 0; s2 < SLOTS; ++s2) M = fmaxf(M, s_m[s2][t]);
    float L = 0.f;
    if (M != -INFINITY)
      for (int s2 = 0; s2 < SLOTS; ++s2)
        if (s_m[s2][t] != -INFINITY) L += s_l[s2][t] * exp2f(s_m[s2][t] - M);
    s_M[t] = M;
    s_L[t] = L;
  }
  __syncthreads();
  // partial slot of this split in the combine layout [slot][Hkv][G][D] (+ [slot][Hkv][G][2])
  const int64_t prow = ((int64_t)(args.split0[i] + split) * Hkv + hk) * G;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const float M = s_M[j];
    const float f = (M == -INFINITY || mx[j] == -INFINITY) ? 0.f : exp2f(mx[j] - M);
#pragma unroll
    for (int e = 0; e < DPL; ++e) s_o[slot][e][chunk] = o[j][e] * f;
    __syncthreads();
    for (int d = t; d < D; d += 256) {
      const int c = d / DPL, e = d % DPL;
      float acc = 0.f;
      for (int s2 = 0; s2 < SLOTS; ++s2) acc += s_o[s2][e][c];
      if (nsplit == 1) {
        const float L = s_L[j];
        Store<T>::store1(out + ((int64_t)i * Hq + hk * G + j) * D + d, L > 0.f ? acc / L : 0.f);
      } else {
        part_o[(prow + j) * D + d] = acc;
        if (d == 0) {
          part_ml[(prow + j) * 2 + 0] = M;
          part_ml[(prow + j) * 2 + 1] = s_L[j];
        }
      }
    }
    __syncthreads();
  }
}

int launch_decode(int dtype, const DecodeArgs& args, const void* q, const void* k, const void* v, const CacheView& cv,
                  int layer, const double* inv_freq, int Hq, void* out, float* part_o, float* part_ml,
                  hipStream_t s) {
  if (args.n == 0) return 0;
  const int g = Hq / cv.n_kv_heads;
  dim3 grid(args.split0[args.n], cv.n_kv_heads);
#define DK(T, DD, GG)                                                                                       \
  if (cv.page_size)                                                                                         \
    hipLaunchKernelGGL((decode_kernel<T, DD, GG, true>), grid, dim3(256), 0, s, args, (const T*)q,          \
                       (const T*)k, (const T*)v, cv, layer, inv_freq, (T*)out, part_o, part_ml);             \
  else                                                                                                      \
    hipLaunchKernelGGL((decode_kernel<T, DD, GG, false>), grid, dim3(256), 0, s, args, (const T*)q,         \
                       (const T*)k, (const T*)v, cv, layer, inv_freq, (T*)out, part_o, part_ml)
#define DKG(T, DD)                                                                                          \
  switch (g) {                                                                                              \
    case 1: DK(T, DD, 1); break;                                                                            \
    case 2: DK(T, DD, 2); break;                                                                            \
    case 4: DK(T, DD, 4); break;                                                                            \
    case 8: DK(T, DD, 8); break;                                                                            \
    case 16: DK(T, DD, 16); break;                                                                          \
    default: return -1;                                                                                     \
  }
  if (dtype == 0) { if (cv.head_dim == 64) { DKG(float, 64) } else { DKG(float, 128) } }
  else { if (cv.head_dim == 64) { DKG(bf16_t, 64) } else { DKG(bf16_t, 128) } }
#undef DKG
#undef DK
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
