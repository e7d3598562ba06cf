// Shared tail of the decode kernels (Sec. 4.2, Eq. 6: decode over the
// grafted KV states).  A block has attended one split of one (sequence, kv
// head) and holds, per query head j of the group, its max M_j, sum L_j and
// unnormalised output O_j (base-2 exponent scale).
//   - emit_pair writes two adjacent output dims: normalised into out when the
//     sequence has a single split, else into the split's partial slot with
//     device-coherent stores (bf16 rows for bf16 storage, fp32 otherwise).
//   - merge_splits makes the block count itself in the (sequence, kv head)
//     counter once its partial stores have completed; the block that arrives
//     last folds every split's partial (device-coherent buffer loads) and
//     writes the output, then sets the counter back to zero.  Every access
//     that crosses blocks is device-coherent, so no L2 write-back or
//     invalidation is needed.
#pragma once

#include "fcg_device.hpp"
#include "kernels.hpp"

namespace fcg {

// Element offset of the new token's row (layer, seq, head, pos).  A page the
// step maps comes by value (DecodeArgs::new_page): the device page table gets
// its entry from this launch (enter_page), so no block reads it there.
template <bool PAGED>
__device__ __forceinline__ int64_t new_token_offset(const CacheView& c, int layer, int seq, int head, int pos,
                                                    int new_page) {
  if (PAGED && new_page >= 0)
    return (int64_t)layer * c.layer_stride +
           (((int64_t)new_page * c.n_kv_heads + head) * 16 + (pos & 15)) * c.head_dim;
  return kv_offset<PAGED>(c, layer, seq, head, pos);
}

// The device page-table entries of a page a decode step maps: its physical
// page, and "values not read from the library" (written by one lane of the
// owning split's first kv-head block; later launches read them).
__device__ __forceinline__ void enter_page(const CacheView& c, int seq, int pos, int new_page) {
  int32_t* row = const_cast<int32_t*>(c.page_table) + (int64_t)seq * 2 * c.n_lp;
  row[pos >> 4] = new_page;
  row[c.n_lp + (pos >> 4)] = -1;
}

// partial slot row of (split slot, kv head, query head): [slot][Hkv][G]
__device__ __forceinline__ int64_t part_row(int slot, int Hkv, int hk, int G, int j) {
  return ((int64_t)slot * Hkv + hk) * G + j;
}

template <typename T, int D>
__device__ __forceinline__ void emit_pair(int nsplit, int64_t prow, T* out_row, float* part_o, float* part_ml,
                                          int d, float a0, float a1, float M, float L) {
  if (nsplit == 1) {
    Store<T>::store1(out_row + d, L > 0.f ? a0 / L : 0.f);
    Store<T>::store1(out_row + d + 1, L > 0.f ? a1 / L : 0.f);
    return;
  }
  if constexpr (sizeof(T) == 2) {
    st_dev_u32(reinterpret_cast<uint32_t*>(part_o) + (prow * D + d) / 2, pack_bf16x2(a0, a1));
  } else {
    st_dev(&part_o[prow * D + d], a0);
    st_dev(&part_o[prow * D + d + 1], a1);
  }
  if (d == 0) {
    st_dev(&part_ml[prow * 2 + 0], M);
    st_dev(&part_ml[prow * 2 + 1], L);
  }
}

// Called by all 256 lanes after their emit_pair calls, when nsplit > 1.
// LDS: s_buf NBUF floats, s_mt / s_lt [256 / (D / EPL)][G] floats, s_flag.
// Always inlined: called out of line (a choice the compiler made once more
// kernel instances called it) it made every decode launch ~2 us longer.
template <typename T, int D, int G, int NBUF>
__device__ __forceinline__ void merge_splits(const DecodeArgs& args, int i, int hk, int slot0, int nsplit, int Hkv,
                                             int Hq, T* __restrict__ out, const float* part_o,
                                             const float* part_ml, int* count, float* s_buf, float* s_mt,
                                             float* s_lt, int* s_flag) {
  constexpr bool BF = sizeof(T) == 2;
  const int t = threadIdx.x;
  // Ordering of the cross-block merge, stated in the hardware's terms (the
  // atomics are relaxed: release/acquire at agent scope writes back and
  // invalidates the L2 around the add; an earlier merge built on such fences,
  // with a serial merge loop, took 50 us per launch):
  //  1. every partial store is a device-scope (sc1) store, written through to
  //     the device coherence point; s_waitcnt vmcnt(0) returns only once this
  //     wave's stores are acknowledged there, and the barrier makes that hold
  //     for all four waves before the block's counter add is issued;
  //  2. the counter adds are atomic read-modify-writes at that same point, so
  //     the block that reads nsplit - 1 is ordered after every other block's
  //     add, hence after all their acknowledged stores;
  //  3. that block's partial loads are device-scope (sc1) buffer loads served
  //     by the coherence point, issued only after its add returned: they sit
  //     behind a branch on the returned count and two barriers (workgroup
  //     fences), which the compiler does not move memory accesses across.
  // The many-split and split-edge GPU tests exercise exactly this path.
  wait_vm0();        // this wave's partial stores have completed
  __syncthreads();   // ... and every wave's
  if (t == 0) {
    int* c = count + (i * Hkv + hk) * kCountStride;
    const int before = __hip_atomic_fetch_add(c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = before == nsplit - 1;
    if (before == nsplit - 1) __hip_atomic_store(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!*s_flag) return;

  // O = sum_s O_s 2^(M_s - M) / sum_s L_s 2^(M_s - M), M = max_s M_s, per
  // query head.  Lane (split lane sl, 16-byte chunk dc of a row) folds the
  // splits sl, sl + NSL, ... of its chunk into a running (max, sum, output)
  // per head, as in the key loop; the NSL split lanes of each chunk then meet
  // in LDS.  Loads of splits past the last one use an offset beyond the
  // buffer: they return zeros without a memory access.
  constexpr int EB = BF ? 2 : 4;            // bytes per partial element
  constexpr int EPL = 16 / EB;              // elements per 16-byte chunk
  constexpr int NDC = D / EPL, NSL = 256 / NDC;
  constexpr int PF = 16 / G;                     // splits per lane per batch of loads
  constexpr int NMLV = G >= 2 ? G / 2 : 1;       // 16-byte loads of a split's (max, sum) pairs
  constexpr int JR0 = NBUF / (NSL * D);
  constexpr int JR = JR0 < G ? JR0 : G;          // heads per LDS round
  static_assert(JR >= 1, "merge buffer");
  constexpr uint32_t kFar = 0x80000000u;         // past every partial buffer (< 2^31 bytes)
  const int dc = t % NDC, sl = t / NDC;
  const int64_t hg = (int64_t)Hkv * G;          // rows per partial slot
  const int64_t row0 = (int64_t)slot0 * hg + (int64_t)hk * G;
  const uint32_t rows_all = (uint32_t)(args.slots * hg);
  const __amdgpu_buffer_rsrc_t ro = buf_rsrc(part_o, rows_all * D * EB);
  const __amdgpu_buffer_rsrc_t rml = buf_rsrc(part_ml, rows_all * 8u);
  float acc[G][EPL], lm[G], ll[G];
#pragma unroll
  for (int j = 0; j < G; ++j) {
    lm[j] = -INFINITY;
    ll[j] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[j][e] = 0.f;
  }
  for (int sb = 0; sb < nsplit; sb += NSL * PF) {
    u32x4_t rv[PF][G], mv[PF][NMLV];
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int sp = sb + sl + p * NSL;
      const bool ok = sp < nsplit;
      const int64_t r = row0 + (int64_t)sp * hg;
#pragma unroll
      for (int h = 0; h < NMLV; ++h) {
        if constexpr (G >= 2) {
          mv[p][h] = ld16_dev(rml, ok ? (uint32_t)((r + 2 * h) * 8) : kFar);
        } else {
          const u32x2_t x = ld8_dev(rml, ok ? (uint32_t)(r * 8) : kFar);
          mv[p][h] = u32x4_t{x.x, x.y, 0u, 0u};
        }
      }
#pragma unroll
      for (int j = 0; j < G; ++j)
        rv[p][j] = ld16_dev(ro, ok ? (uint32_t)(((r + j) * D + dc * EPL) * EB) : kFar);
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      auto mval = [&](int p) { return __uint_as_float(j % 2 ? mv[p][j / 2].z : mv[p][j / 2].x); };
      auto lval = [&](int p) { return __uint_as_float(j % 2 ? mv[p][j / 2].w : mv[p][j / 2].y); };
      float bm = -INFINITY;
#pragma unroll
      for (int p = 0; p < PF; ++p)
        if (sb + sl + p * NSL < nsplit) bm = fmaxf(bm, mval(p));
      const float mn = fmaxf(lm[j], bm);
      if (mn == -INFINITY) continue;
      const float f = __builtin_amdgcn_exp2f(lm[j] - mn);  // 0 while nothing was folded
      ll[j] *= f;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[j][e] *= f;
#pragma unroll
      for (int p = 0; p < PF; ++p) {
        if (sb + sl + p * NSL >= nsplit) continue;
        const float wgt = __builtin_amdgcn_exp2f(mval(p) - mn);
        ll[j] = fmaf(lval(p), wgt, ll[j]);
        float x[EPL];
        if constexpr (BF) {
          Store<T>::unpack(make_uint4(rv[p][j].x, rv[p][j].y, rv[p][j].z, rv[p][j].w), x);
        } else {
          x[0] = __uint_as_float(rv[p][j].x);
          x[1] = __uint_as_float(rv[p][j].y);
          x[2] = __uint_as_float(rv[p][j].z);
          x[3] = __uint_as_float(rv[p][j].w);
        }
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[j][e] = fmaf(x[e], wgt, acc[j][e]);
      }
      lm[j] = mn;
    }
  }
  // merge the split lanes: per head, M over the lanes, each lane's output
  // and sum weighted by 2^(m - M)
  if (dc == 0) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      s_mt[sl * G + j] = lm[j];
      s_lt[sl * G + j] = ll[j];
    }
  }
#pragma unroll
  for (int jr = 0; jr < G; jr += JR) {
    if (jr) __syncthreads();  // the previous round's sums are read
#pragma unroll
    for (int jj = 0; jj < JR; ++jj)
#pragma unroll
      for (int e = 0; e < EPL; e += 4)
        *reinterpret_cast<float4*>(&s_buf[(sl * JR + jj) * D + dc * EPL + e]) =
            make_float4(acc[jr + jj][e], acc[jr + jj][e + 1], acc[jr + jj][e + 2], acc[jr + jj][e + 3]);
    __syncthreads();
    for (int idx = t; idx < JR * D / 2; idx += 256) {
      const int jj = idx / (D / 2), d = 2 * (idx % (D / 2)), j = jr + jj;
      float M = -INFINITY;
#pragma unroll
      for (int s2 = 0; s2 < NSL; ++s2) M = fmaxf(M, s_mt[s2 * G + j]);
      float L = 0.f, o0 = 0.f, o1 = 0.f;
      if (M != -INFINITY) {
#pragma unroll 8
        for (int s2 = 0; s2 < NSL; ++s2) {
          const float ms = s_mt[s2 * G + j];
          const float wgt = ms == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ms - M);
          const float2 x = *reinterpret_cast<const float2*>(&s_buf[(s2 * JR + jj) * D + d]);
          L = fmaf(s_lt[s2 * G + j], wgt, L);
          o0 = fmaf(x.x, wgt, o0);
          o1 = fmaf(x.y, wgt, o1);
        }
      }
      T* dst = out + ((int64_t)i * Hq + hk * G + j) * D + d;
      Store<T>::store1(dst, L > 0.f ? o0 / L : 0.f);
      Store<T>::store1(dst + 1, L > 0.f ? o1 / L : 0.f);
    }
  }
}

// split-lane table size of merge_splits for (T, D)
template <typename T, int D>
constexpr int merge_lanes() {
  return 256 / (D / (16 / (int)sizeof(T)));
}

}  // namespace fcg
