// Vector-ALU attention for gfx950: one query token (its g query heads sharing
// one kv head) per block, over one split [k0, k1) of its causal key range.
// Used for decode steps (one query per sequence: HBM-bound, about 4 FLOP per
// byte at g = 4, so matrix cores would idle) and for fp32 caches.
//
// Lane layout: a key row of D elements is split into 16-byte vectors; LPK =
// D / VEC lanes hold one key, so a wave covers 64 / LPK keys per step and
// every load is a coalesced 16-byte vector.  Scores are reduced across the LPK
// lanes of a key with DPP (quad_perm, row_half_mirror, row_mirror).  Each lane
// keeps its own running max / sum / output (online softmax in base 2: the
// query is pre-scaled by log2(e) / sqrt(D)); the 256 lanes are merged through
// LDS at the end of the block.  A block that covers the whole range writes the
// normalised output; otherwise it writes a partial (max, sum, unnormalised
// output) that the combine kernel merges.
#include "fcg_device.hpp"
#include "kernels.hpp"

namespace fcg {

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over groups of LPK consecutive lanes (LPK in 1, 2, 4, 8, 16); every lane gets the sum.
template <int LPK>
__device__ __forceinline__ float group_sum(float x) {
  if (LPK >= 2) x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  if (LPK >= 4) x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  if (LPK >= 8) x += dpp<0x141>(x);  // row_half_mirror
  if (LPK >= 16) x += dpp<0x140>(x); // row_mirror
  return x;
}

template <typename T, int D, int G>
__global__ void __launch_bounds__(256) attn_rows_kernel(const AttnItem* __restrict__ items,
                                                        const TokenMeta* __restrict__ meta,
                                                        const T* __restrict__ qws, int rows_ws, CacheView cv,
                                                        int layer, int Hq, T* __restrict__ out,
                                                        float* __restrict__ part_o, float* __restrict__ part_ml,
                                                        int part_stride_rows) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int NV = (D / VEC > 16) ? (D / VEC) / 16 : 1;  // 16-byte vectors per lane
  constexpr int DPL = VEC * NV;                              // dims per lane
  constexpr int LPK = D / DPL;                               // lanes per key (<= 16)
  constexpr int SLOTS = 256 / LPK;                           // keys per block step
  static_assert(LPK <= 16, "a key must fit one DPP row");
  __shared__ float s_m[SLOTS][G], s_l[SLOTS][G];
  __shared__ float s_o[SLOTS][DPL][LPK];
  __shared__ float s_M[G], s_L[G];

  const AttnItem it = items[blockIdx.x];
  const int hk = blockIdx.y;
  const int Hkv = cv.n_kv_heads;
  const TokenMeta m = meta[it.rank0];
  const int t = threadIdx.x;
  const int chunk = t % LPK;
  const int slot = t / LPK;
  const float qscale = 1.4426950408889634f / sqrtf((float)D);

  float q[G][DPL];
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) {
      float x[VEC];
      Store<T>::unpack(
          ld16(qws + ((int64_t)hk * rows_ws + (int64_t)it.rank0 * G + j) * D + chunk * DPL + nv * VEC), x);
#pragma unroll
      for (int e = 0; e < VEC; ++e) q[j][nv * VEC + e] = x[e] * qscale;
    }
  float mx[G], sum[G], o[G][DPL];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    mx[j] = -INFINITY;
    sum[j] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[j][e] = 0.f;
  }
  const T* ck = reinterpret_cast<const T*>(cv.k);
  const T* cvv = reinterpret_cast<const T*>(cv.v);
  const int end = min(it.k1, m.pos + 1);
  for (int base = it.k0; base < end; base += SLOTS) {
    const int key = base + slot;
    if (key < end) {  // uniform across the LPK lanes of a key, so DPP partners are active
      const int64_t off = cache_offset(cv, layer, m.seq, hk, key) + chunk * DPL;
      const T* vr = (cv.page_size ? v_row<true, T>(cv, layer, m.seq, hk, key) : cvv + off - chunk * DPL) + chunk * DPL;
      float kx[DPL], vx[DPL];
#pragma unroll
      for (int nv = 0; nv < NV; ++nv) {
        Store<T>::unpack(ld16(ck + off + nv * VEC), kx + nv * VEC);
        Store<T>::unpack(ld16(vr + nv * VEC), vx + nv * VEC);
      }
      float s[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) a = fmaf(q[j][e], kx[e], a);
        s[j] = group_sum<LPK>(a);
      }
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float mn = fmaxf(mx[j], s[j]);
        const float a = exp2f(mx[j] - mn);  // mx = -inf before the first key: a = 0
        const float p = exp2f(s[j] - mn);
        sum[j] = fmaf(sum[j], a, p);
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(o[j][e], a, p * vx[e]);
        mx[j] = mn;
      }
    }
  }
  // merge the SLOTS key slots of the block
  if (chunk == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) { s_m[slot][j] = mx[j]; s_l[slot][j] = sum[j]; }
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
      if (it.part < 0) {
        const float L = s_L[j];
        Store<T>::store1(out + ((int64_t)m.tok * Hq + hk * G + j) * D + d, L > 0.f ? acc / L : 0.f);
      } else {
        const int64_t row = ((int64_t)it.part * Hkv + hk) * part_stride_rows + j;
        part_o[row * D + d] = acc;
        if (d == 0) {
          part_ml[row * 2 + 0] = s_M[j];
          part_ml[row * 2 + 1] = s_L[j];
        }
      }
    }
    __syncthreads();
  }
}

// Merge split-KV partials: per row, M = max M_s, L = sum L_s 2^(M_s - M),
// O = sum O_s 2^(M_s - M) / L.  Block (row block, kv head, z) merges up to
// kCombRows rows, its item taken from the by-value plan.  Every load that
// does not depend on another is issued first: the (M_s, L_s) pairs into LDS,
// the rows' output tokens and, for the bf16 MFMA partials, the first
// PRE splits' partial outputs of the lane's 4-dim chunk; 32 lanes per
// row then form the scales 2^(M_s - M) / L with shuffles, and each 4-dim
// output chunk is summed over the splits (fp32 partials: LPC lanes per chunk
// taking interleaved splits, their sums added through LDS).
constexpr int kCombRows = 8;
constexpr int kCombMaxParts = 256;
// PRE: the smallest of 4, 16 and 32 that covers every row block of the
// launch (each preload past the last split re-reads it: 7B patch call -0.4 us
// with 16 against 32).
template <typename T, int D, bool MFMA_PART, int PRE>
__global__ void __launch_bounds__(256) combine_kernel(CombineArgs args, const TokenMeta* __restrict__ meta, int Hq,
                                                      int Hkv, const float* __restrict__ part_o,
                                                      const float* __restrict__ part_ml, int part_stride_rows,
                                                      T* __restrict__ out) {
  __shared__ float s_f[kCombRows][kCombMaxParts + 1];  // +1: rows start in different banks
  __shared__ float s_l[kCombRows][kCombMaxParts + 1];
  __shared__ float4 s_acc[256];
  const CombineItem it = args.item[blockIdx.x];
  const int hk = blockIdx.y;
  // every argument in one batch of scalar loads, before any arithmetic on
  // them (else the compiler issues part of the batch after the division)
  asm volatile("" ::"s"(it.rank0), "s"(it.n_rank), "s"(it.n_part), "s"(it.part0), "s"(it.tok0), "s"(meta), "s"(part_o),
               "s"(part_ml), "s"(out), "s"(Hq), "s"(Hkv), "s"(part_stride_rows));
  __builtin_amdgcn_sched_barrier(0);
  const int g = Hq / Hkv;
  const int t = threadIdx.x;
  const int r0 = blockIdx.z * kCombRows;
  const int nr = min(kCombRows, it.n_rank * g - r0);
  const int np = it.n_part;
  if (nr <= 0) return;
  auto prow = [&](int s, int r) { return ((int64_t)(it.part0 + s) * Hkv + hk) * part_stride_rows + r0 + r; };
  constexpr int CPR = D / 4;                  // 4-dim chunks per row
  const int nch = nr * CPR;
  const int lpc = max(1, 256 / nch);          // lanes per chunk (power of two: nr, CPR are)
  // chunk c -> (row, 4-dim chunk): neighbouring lanes read neighbouring bytes
  // (rows fastest in the MFMA fragment order, dims fastest in row-major order)
  auto chunk = [&](int c, int* r, int* c4) {
    *r = MFMA_PART ? c % nr : c / CPR;
    *c4 = MFMA_PART ? c / nr : c % CPR;
  };
  // bf16 partial output of split s, row r, chunk c4, in the MFMA accumulator
  // order of the prefill kernel: per 16-row tile and 16-dim tile, 64 lanes x
  // 4 dims, lane = row % 16 + 16 * (4-dim chunk % 4)
  auto mfma_part = [&](int s, int r, int c4) -> uint2 {
    const int rr = r0 + r;
    const int64_t off = ((int64_t)(it.part0 + s) * Hkv + hk) * part_stride_rows * D +
                        (((rr / 16) * (D / 16) + c4 / 4) * 64 + rr % 16 + 16 * (c4 % 4)) * 4;
    return *reinterpret_cast<const uint2*>(reinterpret_cast<const bf16_t*>(part_o) + off);
  };
  int my_r = 0, my_c4 = 0;
  const bool my_chunk = t / lpc < nch;
  chunk(my_chunk ? t / lpc : 0, &my_r, &my_c4);
  uint2 pre[MFMA_PART ? PRE : 1];
  if (MFMA_PART) {
    // lpc is 1 here (nch = 8 rows x D/4 chunks = 256 lanes for a full block)
#pragma unroll
    for (int u = 0; u < PRE; ++u) pre[u] = mfma_part(min(u, np - 1), my_r, my_c4);
  }
  const int out_tok = it.tok0 >= 0 ? it.tok0 + (r0 + my_r) / g : meta[it.rank0 + (r0 + my_r) / g].tok;
  for (int idx = t; idx < nr * np; idx += 256) {
    const int r = idx / np, s = idx % np;
    s_f[r][s] = part_ml[prow(s, r) * 2];
    s_l[r][s] = part_ml[prow(s, r) * 2 + 1];
  }
  __syncthreads();
  {
    // 32 lanes per row: M, L and the scales 2^(M_s - M) / L
    const int r = t / 32, l32 = t % 32;
    if (r < nr) {
      float M = -INFINITY;
      for (int s = l32; s < np; s += 32) M = fmaxf(M, s_f[r][s]);
      M = max_lanes32(M);
      float L = 0.f;
      for (int s = l32; s < np; s += 32) {
        const float ms = s_f[r][s];
        L = fmaf(s_l[r][s], ms == -INFINITY ? 0.f : exp2f(ms - M), L);
      }
      L = sum_lanes32(L);
      const float inv = L > 0.f ? 1.f / L : 0.f;
      for (int s = l32; s < np; s += 32) {
        const float ms = s_f[r][s];
        s_f[r][s] = ms == -INFINITY ? 0.f : exp2f(ms - M) * inv;
      }
    }
  }
  __syncthreads();
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  auto add = [&](float4 o, float f) {
    acc.x = fmaf(o.x, f, acc.x);
    acc.y = fmaf(o.y, f, acc.y);
    acc.z = fmaf(o.z, f, acc.z);
    acc.w = fmaf(o.w, f, acc.w);
  };
  auto bf4 = [](uint2 u) { return make_float4(lo_bf16(u.x), hi_bf16(u.x), lo_bf16(u.y), hi_bf16(u.y)); };
  if (MFMA_PART) {
    if (!my_chunk) return;
#pragma unroll
    for (int u = 0; u < PRE; ++u)
      if (u < np) add(bf4(pre[u]), s_f[my_r][u]);
#pragma unroll 8
    for (int s = PRE; s < np; ++s) add(bf4(mfma_part(s, my_r, my_c4)), s_f[my_r][s]);
  } else {
    if (my_chunk) {
#pragma unroll 8
      for (int s = t % lpc; s < np; s += lpc)
        add(*reinterpret_cast<const float4*>(part_o + prow(s, my_r) * D + my_c4 * 4), s_f[my_r][s]);
    }
    if (lpc > 1) {
      s_acc[t] = acc;
      __syncthreads();
      if (t % lpc || !my_chunk) return;
      for (int sub = 1; sub < lpc; ++sub) {
        const float4 a4 = s_acc[t + sub];
        acc.x += a4.x;
        acc.y += a4.y;
        acc.z += a4.z;
        acc.w += a4.w;
      }
    } else if (!my_chunk) {
      return;
    }
  }
  T* dst = out + ((int64_t)out_tok * Hq + hk * g + (r0 + my_r) % g) * D + my_c4 * 4;
  Store<T>::store1(dst + 0, acc.x);
  Store<T>::store1(dst + 1, acc.y);
  Store<T>::store1(dst + 2, acc.z);
  Store<T>::store1(dst + 3, acc.w);
}

int launch_attn_rows(int dtype, const AttnItem* items, int n_items, const TokenMeta* meta, const void* qws,
                     int rows_ws, const CacheView& cv, int layer, int Hq, void* out, float* part_o,
                     float* part_ml, int part_stride_rows, hipStream_t s, KTime tm) {
  if (n_items == 0) return 0;
  const int g = Hq / cv.n_kv_heads;
  dim3 grid(n_items, cv.n_kv_heads);
#define AR(T, DD, GG)                                                                                       \
  hipExtLaunchKernelGGL((attn_rows_kernel<T, DD, GG>), grid, dim3(256), 0, s, tm.start, tm.stop, 0, items, meta, (const T*)qws,      \
                     rows_ws, cv, layer, Hq, (T*)out, part_o, part_ml, part_stride_rows)
#define ARG(T, DD)                                                                                          \
  switch (g) {                                                                                              \
    case 1: AR(T, DD, 1); break;                                                                            \
    case 2: AR(T, DD, 2); break;                                                                            \
    case 4: AR(T, DD, 4); break;                                                                            \
    case 8: AR(T, DD, 8); break;                                                                            \
    case 16: AR(T, DD, 16); break;                                                                          \
    default: return -1;                                                                                     \
  }
  if (dtype == 0) { if (cv.head_dim == 64) { ARG(float, 64) } else { ARG(float, 128) } }
  else { if (cv.head_dim == 64) { ARG(bf16_t, 64) } else { ARG(bf16_t, 128) } }
#undef ARG
#undef AR
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

int launch_combine(int dtype, const CombineArgs& args, const TokenMeta* meta, int Hq, int Hkv, int D,
                   const float* part_o, const float* part_ml, int part_stride_rows, void* out, hipStream_t s,
                   bool mfma_part, KTime tm) {
  if (args.n_items == 0) return 0;
  dim3 grid(args.n_items, Hkv, (part_stride_rows + kCombRows - 1) / kCombRows);
  int max_np = 0;
  for (int i = 0; i < args.n_items; ++i) max_np = max(max_np, (int)args.item[i].n_part);
  const int pre = max_np <= 4 ? 4 : max_np <= 16 ? 16 : 32;
#define CBK(T, DD, MP, PR)                                                                                  \
  hipExtLaunchKernelGGL((combine_kernel<T, DD, MP, PR>), grid, dim3(256), 0, s, tm.start, tm.stop, 0, args,   \
                        meta, Hq, Hkv, part_o, part_ml, part_stride_rows, (T*)out)
#define CB(T, DD)                                                                                            \
  do {                                                                                                       \
    if (!mfma_part) CBK(T, DD, false, 16);                                                                   \
    else if (pre == 4) CBK(T, DD, true, 4);                                                                  \
    else if (pre == 16) CBK(T, DD, true, 16);                                                                \
    else CBK(T, DD, true, 32);                                                                               \
  } while (0)
  if (dtype == 0) { if (D == 64) CB(float, 64); else CB(float, 128); }
  else { if (D == 64) CB(bf16_t, 64); else CB(bf16_t, 128); }
#undef CB
#undef CBK
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
