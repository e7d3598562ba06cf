// One decode step at one layer for a batch of sequences (Sec. 4.2, Eq. 6:
// decoding over the reused, grafted KV states).
//
// Per sequence i the new token sits at position pos_i = its current length.
// Block (split s, sequence i, kv head h) attends the token's g query heads
// over key positions [s * split_keys, min(pos_i + 1, (s + 1) * split_keys)):
//   - before anything else it issues the loads of its first chunk of cached
//     keys and values, of the query rows, of the new token's key and value
//     and of the rotary frequencies, so the block pays one memory latency
//     before its first math; every load is unconditional (positions past the
//     range re-read its last key, scores masked), which keeps the compiler's
//     load counting exact;
//   - it encodes the queries at pos_i (cos/sin of the position in LDS, fp64
//     angle), rounds them to storage and pre-scales them by log2(e) / sqrt(D)
//     for a base-2 softmax;
//   - cached keys stream through 16-byte vector loads, LPK lanes per key, U
//     key steps per chunk, the next chunk in flight while one is reduced;
//     scores are summed across a key's lanes with DPP, and each lane keeps an
//     online softmax rescaled once per chunk;
//   - the block whose split holds pos_i also encodes the new key, stores key
//     and value into the cache slot and attends to them from registers; no
//     other block touches that slot;
//   - the block merges its key slots through LDS; a single-split sequence
//     writes its output, otherwise the block stores a partial (max, sum,
//     unnormalised output) with device-coherent stores, waits for them to
//     complete and counts itself in the (sequence, kv head) counter; the
//     block that arrives last combines every split's partial (read with
//     device-coherent loads, so no L2 write-back or invalidation is needed)
//     and writes the output, then sets the counter back to zero.
#include "decode_common.hpp"

namespace fcg {

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// a.lo * b.lo + a.hi * b.hi + c over bf16 pairs (v_dot2c_f32_bf16, fp32 accumulate)
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}

template <int LPK>
__device__ __forceinline__ float lanes_sum(float x) {
  if (LPK >= 2) x += dpp_f<0xB1>(x);   // quad_perm [1,0,3,2]
  if (LPK >= 4) x += dpp_f<0x4E>(x);   // quad_perm [2,3,0,1]
  if (LPK >= 8) x += dpp_f<0x141>(x);  // row_half_mirror
  if (LPK >= 16) x += dpp_f<0x140>(x); // row_mirror
  return x;
}

template <int W>  // sum over the lanes of a wave that are W, 2W, ... apart
__device__ __forceinline__ float lanes_sum_stride(float x) {
#pragma unroll
  for (int o = W; o < 64; o *= 2) x += __shfl_xor(x, o);
  return x;
}

template <typename T, int D, int G, bool PAGED>
__global__ void __launch_bounds__(256) decode_kernel(DecodeArgs args, const T* __restrict__ q,
                                                     const T* __restrict__ k, const T* __restrict__ v, CacheView cv,
                                                     const float2* __restrict__ rope, T* __restrict__ out,
                                                     float* __restrict__ part_o, float* __restrict__ part_ml,
                                                     int* __restrict__ count, int layer) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int NV = (D / VEC > 16) ? (D / VEC) / 16 : 1;
  constexpr int DPL = VEC * NV;    // dims per lane
  constexpr int LPK = D / DPL;     // lanes per key
  constexpr int SLOTS = 256 / LPK; // keys per step
  constexpr int U = G >= 8 ? 2 : 4;  // steps per chunk
  constexpr int CK = U * SLOTS;    // keys per chunk
  constexpr int HALF = D / 2;
  constexpr int JB = G < 4 ? G : 4;  // query heads per LDS merge round
  constexpr bool BF = sizeof(T) == 2;  // bf16: scores with v_dot2 on packed pairs
  constexpr int NW = DPL / 2;          // packed pairs per lane
  __shared__ float s_cos[HALF], s_sin[HALF];
  __shared__ float s_m[SLOTS][G], s_l[SLOTS][G];
  // slot outputs [SLOTS][JB][D]; in the cross-split merge, the split
  // lanes' outputs of a round of heads
  constexpr int NBUF = SLOTS * JB * D;
  __shared__ float s_buf[NBUF];
  __shared__ float s_L[G];
  __shared__ int s_last;

  const int split = blockIdx.x, i = blockIdx.y, hk = blockIdx.z;
  const int seq = args.seq[i], pos = args.pos[i], slot0 = args.split0[i];
  const int npage = PAGED ? args.new_page[i] : -1;  // a page this step maps, by value
  const int nsplit = args.split0[i + 1] - slot0;
  const int sk = args.split_keys;
  const T* ck = reinterpret_cast<const T*>(cv.k);
  const T* cvv = reinterpret_cast<const T*>(cv.v);
  // every kernel argument in one batch of scalar loads before the first branch.
  // The batch must not load a dword nothing reads: the compiler may reuse its
  // register for a later load of the batch, which then waits for the first
  // loads to land (a second round trip).  So `layer` comes last (no padding
  // after it) and the unused head_dim, which a merged load covers, is listed.
  asm volatile("" ::"s"(seq), "s"(pos), "s"(slot0), "s"(nsplit), "s"(sk), "s"(q), "s"(k), "s"(v), "s"(ck),
               "s"(cvv), "s"(cv.layer_stride), "s"(cv.max_tokens), "s"(cv.n_kv_heads), "s"(layer), "s"(rope),
               "s"(out), "s"(part_o), "s"(part_ml), "s"(count), "s"(cv.head_dim));
  if (PAGED)
    asm volatile("" ::"s"(cv.page_table), "s"(cv.n_lp), "s"(cv.v_alias), "s"(cv.lib_v), "s"(cv.lib_cap), "s"(npage));
  if (split >= nsplit) return;  // padding split of a shorter sequence

  const int Hkv = cv.n_kv_heads;
  const int Hq = Hkv * G;
  const int t = threadIdx.x;
  const int chunk = t % LPK, slot = t / LPK;
  const int d0 = chunk * DPL;
  const int dp = d0 < HALF ? d0 + HALF : d0 - HALF;  // rotary partner dims
  const int k0 = split * sk;
  const int k1 = min(pos + 1, k0 + sk);
  const bool owns_new = k1 == pos + 1;  // the last split holds the new token
  const int kend = owns_new ? pos : k1;  // cached keys [k0, kend)

  auto load_chunk = [&](int b, uint4 (&kk)[U][NV], uint4 (&vv)[U][NV]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int p = max(0, min(b + u * SLOTS + slot, kend - 1));
      const int64_t off = kv_offset<PAGED>(cv, layer, seq, hk, p) + d0;
      const T* vr = (PAGED ? v_row<true, T>(cv, layer, seq, hk, p) : cvv + off - d0) + d0;
#pragma unroll
      for (int nv = 0; nv < NV; ++nv) {
        kk[u][nv] = ld16(ck + off + nv * VEC);
        vv[u][nv] = ld16(vr + nv * VEC);
      }
    }
  };
  // loads in the order their data is needed (they complete in issue order):
  // rotary frequency, raw query rows, new key (dims and partner dims) and
  // value, then two chunks of cached keys (a chunk past the range re-reads
  // its last key: one row, cached)
  const float2 cs_pos = rope[(int64_t)pos * HALF + t % HALF];  // (cos, sin) of the position
  uint4 qa[G][NV], qb[G][NV], na[NV], nb[NV], nvv[NV];
#pragma unroll
  for (int j = 0; j < G; ++j)
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) {
      const T* row = q + ((int64_t)i * Hq + hk * G + j) * D;
      qa[j][nv] = ld16(row + d0 + nv * VEC);
      qb[j][nv] = ld16(row + dp + nv * VEC);
    }
  {
    const T* krow = k + ((int64_t)i * Hkv + hk) * D;
    const T* vrow = v + ((int64_t)i * Hkv + hk) * D;
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) {
      na[nv] = ld16(krow + d0 + nv * VEC);
      nb[nv] = ld16(krow + dp + nv * VEC);
      nvv[nv] = ld16(vrow + d0 + nv * VEC);
    }
  }
  uint4 kr0[U][NV], vr0[U][NV], kr1[U][NV], vr1[U][NV];
  __builtin_amdgcn_sched_barrier(0);  // the scheduler keeps that order (else the chunks go first)
  load_chunk(k0, kr0, vr0);
  load_chunk(k0 + CK, kr1, vr1);
  if (t < HALF) {
    s_cos[t] = cs_pos.x;
    s_sin[t] = cs_pos.y;
  }
  __syncthreads();

  // rotate lane dims [d0, d0 + DPL) of a row given as (own dims, partner dims)
  auto encode = [&](const uint4 (&xa)[NV], const uint4 (&xb)[NV], float* y) {
    float a[DPL], bb[DPL];
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) {
      Store<T>::unpack(xa[nv], a + nv * VEC);
      Store<T>::unpack(xb[nv], bb + nv * VEC);
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      const int ii = (d0 + e) % HALF;
      const float c = s_cos[ii], sn = s_sin[ii];
      // first half: x_i c - x_{i+D/2} s; second half: x_{i+D/2} c + x_i s
      const float r = d0 < HALF ? fmaf(a[e], c, -bb[e] * sn) : fmaf(a[e], c, bb[e] * sn);
      y[e] = Store<T>::round(r);
    }
  };
  const float qscale = 1.4426950408889634f / sqrtf((float)D);
  // encoded queries: fp32 pre-scaled (fp32 storage), or the rounded bf16
  // values packed in pairs, the score scaled after the dot product
  float qf[G][DPL];
  uint32_t qp[G][NW];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    encode(qa[j], qb[j], qf[j]);
#pragma unroll
    for (int e = 0; e < NW; ++e)
      qp[j][e] = (__float_as_uint(qf[j][2 * e]) >> 16) | (__float_as_uint(qf[j][2 * e + 1]) & 0xFFFF0000u);
#pragma unroll
    for (int e = 0; e < DPL; ++e) qf[j][e] *= qscale;
  }
  // scaled score of query head j against this lane's dims of a key
  auto score = [&](int j, const uint4 (&kw)[NV], const float* kx) -> float {
    float a = 0.f;
    if constexpr (BF) {
#pragma unroll
      for (int nv = 0; nv < NV; ++nv) {
        a = dot2_bf16(qp[j][4 * nv + 0], kw[nv].x, a);
        a = dot2_bf16(qp[j][4 * nv + 1], kw[nv].y, a);
        a = dot2_bf16(qp[j][4 * nv + 2], kw[nv].z, a);
        a = dot2_bf16(qp[j][4 * nv + 3], kw[nv].w, a);
      }
      return lanes_sum<LPK>(a) * qscale;
    } else {
#pragma unroll
      for (int e = 0; e < DPL; ++e) a = fmaf(qf[j][e], kx[e], a);
      return lanes_sum<LPK>(a);
    }
  };

  float mx[G], sm[G], o[G][DPL];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    mx[j] = -INFINITY;
    sm[j] = 0.f;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[j][e] = 0.f;
  }

  // online softmax over one chunk of keys [b, b + CK) held in registers
  auto reduce_chunk = [&](int b, const uint4 (&kk)[U][NV], const uint4 (&vv)[U][NV]) {
    float s[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool ok = b + u * SLOTS + slot < kend;
      float kx[DPL];
      if constexpr (!BF) {
#pragma unroll
        for (int nv = 0; nv < NV; ++nv) Store<T>::unpack(kk[u][nv], kx + nv * VEC);
      }
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float a = score(j, kk[u], kx);
        s[u][j] = ok ? a : -INFINITY;
      }
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      float cm = s[0][j];
#pragma unroll
      for (int u = 1; u < U; ++u) cm = fmaxf(cm, s[u][j]);
      const float mn = fmaxf(mx[j], cm);
      if (mn == -INFINITY) continue;  // nothing seen yet by this lane
      const float a = __builtin_amdgcn_exp2f(mx[j] - mn);  // v_exp_f32: -inf gives 0
      float acc_l = sm[j] * a;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] *= a;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = __builtin_amdgcn_exp2f(s[u][j] - mn);  // 0 for masked keys
        acc_l += p;
        float vx[DPL];
#pragma unroll
        for (int nv = 0; nv < NV; ++nv) Store<T>::unpack(vv[u][nv], vx + nv * VEC);
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(p, vx[e], o[j][e]);
      }
      sm[j] = acc_l;
      mx[j] = mn;
    }
  };
  // two register sets: the chunk after next is in flight while one is reduced
  for (int b = k0; b < kend; b += 2 * CK) {
    reduce_chunk(b, kr0, vr0);
    if (b + CK >= kend) break;
    load_chunk(b + 2 * CK, kr0, vr0);
    reduce_chunk(b + CK, kr1, vr1);
    load_chunk(b + 3 * CK, kr1, vr1);
  }

  if (PAGED && owns_new && hk == 0 && t == 0 && npage >= 0) enter_page(cv, seq, pos, npage);
  if (owns_new && slot == 0) {
    // encode, store and attend the new token (lanes of slot 0)
    float kn[DPL], vn[DPL];
    encode(na, nb, kn);
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) Store<T>::unpack(nvv[nv], vn + nv * VEC);
    const int64_t off = new_token_offset<PAGED>(cv, layer, seq, hk, pos, npage) + d0;
    T* kdst = reinterpret_cast<T*>(cv.k) + off;
    T* vdst = reinterpret_cast<T*>(cv.v) + off;
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) {
      st16(kdst + nv * VEC, Store<T>::pack(kn + nv * VEC));
      st16(vdst + nv * VEC, nvv[nv]);
    }
    uint4 knw[NV];  // the rounded key, packed again (exact: bf16 values)
#pragma unroll
    for (int nv = 0; nv < NV; ++nv) knw[nv] = Store<T>::pack(kn + nv * VEC);
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const float a = score(j, knw, kn);
      const float mn = fmaxf(mx[j], a);
      const float f = __builtin_amdgcn_exp2f(mx[j] - mn), p = __builtin_amdgcn_exp2f(a - mn);
      sm[j] = fmaf(sm[j], f, p);
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[j][e] = fmaf(o[j][e], f, p * vn[e]);
      mx[j] = mn;
    }
  }

  // merge the block's key slots: every lane finds each head's block max M
  // from the slots' maxima, scales its output by 2^(m - M) into LDS, and the
  // block sums the slots per output element
  if (chunk == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) { s_m[slot][j] = mx[j]; s_l[slot][j] = sm[j]; }
  }
  __syncthreads();
#pragma unroll
  for (int jb = 0; jb < G; jb += JB) {
    if (jb) __syncthreads();  // the previous round's sums are read
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      const int j = jb + jj;
      float M = -INFINITY;
#pragma unroll
      for (int s2 = 0; s2 < SLOTS; ++s2) M = fmaxf(M, s_m[s2][j]);
      const float f = (M == -INFINITY || mx[j] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mx[j] - M);
#pragma unroll
      for (int e = 0; e < DPL; e += 4)
        *reinterpret_cast<float4*>(&s_buf[(slot * JB + jj) * D + d0 + e]) =
            make_float4(o[j][e] * f, o[j][e + 1] * f, o[j][e + 2] * f, o[j][e + 3] * f);
    }
    if (jb == 0 && t < G) {  // block sums of the heads
      float M = -INFINITY, L = 0.f;
#pragma unroll
      for (int s2 = 0; s2 < SLOTS; ++s2) M = fmaxf(M, s_m[s2][t]);
      if (M != -INFINITY) {
#pragma unroll
        for (int s2 = 0; s2 < SLOTS; ++s2) L = fmaf(s_l[s2][t], __builtin_amdgcn_exp2f(s_m[s2][t] - M), L);
      }
      s_L[t] = L;
    }
    __syncthreads();
    // two adjacent output dims per lane
    for (int idx = t; idx < JB * D / 2; idx += 256) {
      const int jj = idx / (D / 2), d = 2 * (idx % (D / 2)), j = jb + jj;
      float a0 = 0.f, a1 = 0.f;
#pragma unroll 8
      for (int s2 = 0; s2 < SLOTS; ++s2) {
        const float2 x = *reinterpret_cast<const float2*>(&s_buf[(s2 * JB + jj) * D + d]);
        a0 += x.x;
        a1 += x.y;
      }
      float M = -INFINITY;
      if (d == 0 && nsplit > 1) {
#pragma unroll
        for (int s2 = 0; s2 < SLOTS; ++s2) M = fmaxf(M, s_m[s2][j]);
      }
      emit_pair<T, D>(nsplit, part_row(slot0 + split, Hkv, hk, G, j), out + ((int64_t)i * Hq + hk * G + j) * D,
                      part_o, part_ml, d, a0, a1, M, s_L[j]);
    }
  }
  if (nsplit == 1) return;
  static_assert(merge_lanes<T, D>() <= SLOTS, "split lanes use the slot tables");
  merge_splits<T, D, G, NBUF>(args, i, hk, slot0, nsplit, Hkv, Hq, out, part_o, part_ml, count, s_buf, &s_m[0][0],
                              &s_l[0][0], &s_last);
}

int launch_decode(int dtype, const DecodeArgs& args, const void* q, const void* k, const void* v, const CacheView& cv,
                  int layer, const float2* rope, int Hq, void* out, float* part_o, float* part_ml, int* count,
                  hipStream_t s, KTime tm) {
  if (args.n == 0) return 0;
  const int g = Hq / cv.n_kv_heads;
  dim3 grid(args.max_split, args.n, cv.n_kv_heads);
#define DK(T, DD, GG)                                                                                       \
  if (cv.page_size)                                                                                         \
    hipExtLaunchKernelGGL((decode_kernel<T, DD, GG, true>), grid, dim3(256), 0, s, tm.start, tm.stop, 0, args, (const T*)q,          \
                       (const T*)k, (const T*)v, cv, rope, (T*)out, part_o, part_ml, count, layer);             \
  else                                                                                                      \
    hipExtLaunchKernelGGL((decode_kernel<T, DD, GG, false>), grid, dim3(256), 0, s, tm.start, tm.stop, 0, args, (const T*)q,         \
                       (const T*)k, (const T*)v, cv, rope, (T*)out, part_o, part_ml, count, layer)
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
