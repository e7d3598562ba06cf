// Cache-stitching kernels for gfx950 (Sec. 4.2, Eq. 4; App. B.1).
//
// graft: every grafted token's key is turned from its source position to its
// target position (a rotation by the segment's delta, rotate-half pairs
// (i, i + D/2), angle delta * theta^(-2i/D)) and its value is copied.  The
// kernel is a pure HBM stream: each lane moves whole 16-byte vectors, the two
// halves of a rotary pair are loaded by the same lane, all loads of a block are
// issued before its stores, and data never passes through LDS (LDS holds only
// the D/2 cos/sin values of the block's delta, computed once per block).  Which
// cache hints the reads and writes carry depends on the cache layout (ld_lib,
// st_cache below).
//
// ingest: copy a segment given token-major [L][len][Hkv][D] into the library's
// head-major slabs [L][Hkv][cap][D].
#include "fcg_device.hpp"
#include "kernels.hpp"

namespace fcg {

template <typename T, int D>
__global__ void __launch_bounds__(256) ingest_kernel(const T* __restrict__ k, const T* __restrict__ v,
                                                     T* __restrict__ lk, T* __restrict__ lv, int len, int Hkv,
                                                     int64_t cap, int64_t tok_off) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int VPR = D / VEC;  // vectors per (token, head) row
  const int l = blockIdx.y;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = (int64_t)len * Hkv * VPR;
  if (i >= n) return;
  const int c = (int)(i % VPR);
  const int64_t th = i / VPR;
  const int h = (int)(th % Hkv);
  const int64_t j = th / Hkv;
  const int64_t src = (((int64_t)l * len + j) * Hkv + h) * D + c * VEC;
  const int64_t dst = (((int64_t)l * Hkv + h) * cap + tok_off + j) * D + c * VEC;
  st16(lk + dst, ld16(k + src));
  st16(lv + dst, ld16(v + src));
}

// Library reads and cache writes of the graft.  Contiguous caches: reads with
// the nontemporal hint (read once), plain stores (the cache is read next).  Paged
// caches, whose runs land in 4 KB page pieces: plain reads, so that segments
// several tasks of a batch share are served from cache, and nontemporal stores
// (batched workload: 10.2 -> 6.7 ms per graft; the same choice on a contiguous
// cache was slower).
template <bool PAGED>
__device__ __forceinline__ uint4 ld_lib(const void* p) {
  return PAGED ? ld16(p) : ld16_nt(p);
}
template <bool PAGED>
__device__ __forceinline__ void st_cache(void* p, const uint4& v) {
  if (PAGED)
    __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4_t*>(p));
  else
    st16(p, v);
}

template <typename T, int D, bool PAGED>
__global__ void __launch_bounds__(256) graft_kernel(const GraftChunk* __restrict__ chunks,
                                                    const T* __restrict__ lib_k, const T* __restrict__ lib_v,
                                                    int64_t cap, CacheView cv, const double* __restrict__ inv_freq) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int HALF = D / 2;
  constexpr int KT = HALF / VEC;            // lanes per key row (each owns a pair of vectors)
  constexpr int KR = 256 / KT;              // key rows per pass
  constexpr int KP = (kGraftChunk + KR - 1) / KR;
  constexpr int VT = D / VEC;               // lanes per value row
  constexpr int VR = 256 / VT;
  constexpr int VP = (kGraftChunk + VR - 1) / VR;

  __shared__ float s_cos[HALF], s_sin[HALF];

  const GraftChunk ch = chunks[blockIdx.x];
  const int h = blockIdx.y;
  const int l = blockIdx.z;
  const int t = threadIdx.x;
  const int Hkv = cv.n_kv_heads;

  // paged caches: the page-table entries of the run's (at most five) logical
  // pages, loaded once with the data rather than once per stored row (a
  // lookup per row put a dependent load in front of every store)
  constexpr int NPG = PAGED ? (kGraftChunk + 15) / 16 + 1 : 1;
  int32_t pg[NPG];
  const int lp0 = ch.dst >> 4;
  if (PAGED) {
    const int32_t* prow = cv.page_table + (int64_t)ch.seq * 2 * cv.n_lp + lp0;
    const int last = ((ch.dst + ch.n - 1) >> 4) - lp0;
#pragma unroll
    for (int i = 0; i < NPG; ++i) pg[i] = prow[min(i, last)];
  }
  // element offset of (layer l, head h, position pos) in the cache
  auto dst_off = [&](int pos) -> int64_t {
    if (!PAGED) return kv_offset<false>(cv, l, ch.seq, h, pos);
    const int e = (pos >> 4) - lp0;
    int32_t page = pg[0];
#pragma unroll
    for (int i = 1; i < NPG; ++i) page = e == i ? pg[i] : page;
    return (int64_t)l * cv.layer_stride + (((int64_t)page * Hkv + h) * 16 + (pos & 15)) * D;
  };

  const int64_t src_base = (((int64_t)l * Hkv + h) * cap + ch.src_tok) * D;
  const T* sk = lib_k + src_base;
  const T* sv = lib_v + src_base;
  T* ck = reinterpret_cast<T*>(cv.k);
  T* cvv = reinterpret_cast<T*>(cv.v);

  // issue every load of the block first; rows past the run re-read its last
  // row (their stores are skipped), so the loads carry no branches
  uint4 klo[KP], khi[KP], vv[VP];
  const int kc = t % KT, kr = t / KT;
#pragma unroll
  for (int p = 0; p < KP; ++p) {
    const int j = min(p * KR + kr, ch.n - 1);
    klo[p] = ld_lib<PAGED>(sk + (int64_t)j * D + kc * VEC);
    khi[p] = ld_lib<PAGED>(sk + (int64_t)j * D + HALF + kc * VEC);
  }
  const int vc = t % VT, vr = t / VT;
  // values: not read or written on pages the segment covers entirely when
  // the cache maps those onto the library; a run made only of such pages
  // skips them altogether (a block-uniform branch)
  const bool alias = PAGED && cv.v_alias;
  const bool run_aliased = alias && (ch.dst & ~15) >= ch.seg_lo && ((ch.dst + ch.n - 1) & ~15) + 16 <= ch.seg_hi;
  if (!run_aliased) {
#pragma unroll
    for (int p = 0; p < VP; ++p) {
      const int j = min(p * VR + vr, ch.n - 1);
      vv[p] = ld_lib<PAGED>(sv + (int64_t)j * D + vc * VEC);
    }
  }
  // cos/sin of the run's delta, while the loads are in flight
  if (t < HALF) rope_cs((double)ch.delta, inv_freq[t], &s_cos[t], &s_sin[t]);
  __syncthreads();  // cos/sin ready

  float c[VEC], s[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    c[e] = s_cos[kc * VEC + e];
    s[e] = s_sin[kc * VEC + e];
  }
#pragma unroll
  for (int p = 0; p < KP; ++p) {
    const int j = p * KR + kr;
    if (j < ch.n) {
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Store<T>::unpack(klo[p], x1);
      Store<T>::unpack(khi[p], x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        y1[e] = fmaf(x1[e], c[e], -x2[e] * s[e]);
        y2[e] = fmaf(x2[e], c[e], x1[e] * s[e]);
      }
      const int64_t off = dst_off(ch.dst + j);
      st_cache<PAGED>(ck + off + kc * VEC, Store<T>::pack(y1));
      st_cache<PAGED>(ck + off + HALF + kc * VEC, Store<T>::pack(y2));
    }
  }
  if (run_aliased) return;
#pragma unroll
  for (int p = 0; p < VP; ++p) {
    const int j = p * VR + vr;
    const int pg0 = (ch.dst + j) & ~15;
    if (j < ch.n && !(alias && pg0 >= ch.seg_lo && pg0 + 16 <= ch.seg_hi)) {
      const int64_t off = dst_off(ch.dst + j);
      st_cache<PAGED>(cvv + off + vc * VEC, vv[p]);
    }
  }
}

// Copy the first rows of value pages from the library into the cache's own
// pages (pages that were mapped onto the library and that a truncation split,
// so that new tokens can follow the kept rows).  Grid (item, kv head, layer).
template <typename T, int D>
__global__ void __launch_bounds__(256) unalias_kernel(const UnaliasItem* __restrict__ items,
                                                      const T* __restrict__ lib_v, int64_t cap, CacheView cv) {
  constexpr int VEC = Store<T>::VEC;
  constexpr int VT = D / VEC;
  const UnaliasItem it = items[blockIdx.x];
  const int h = blockIdx.y, l = blockIdx.z;
  const int Hkv = cv.n_kv_heads;
  for (int idx = threadIdx.x; idx < it.rows * VT; idx += 256) {
    const int r = idx / VT, c = idx % VT;
    const T* src = lib_v + (((int64_t)l * Hkv + h) * cap + it.lib_tok + r) * D + c * VEC;
    T* dst = reinterpret_cast<T*>(cv.v) + (int64_t)l * cv.layer_stride + (((int64_t)it.page * Hkv + h) * 16 + r) * D +
             c * VEC;
    st16(dst, ld16(src));
  }
}

static int check(hipError_t e) { return e == hipSuccess ? 0 : (int)e; }

int launch_unalias(int dtype, const UnaliasItem* items, int n_items, const void* lib_v, int64_t cap,
                   const CacheView& cv, int L, hipStream_t s) {
  if (n_items == 0) return 0;
  dim3 grid(n_items, cv.n_kv_heads, L);
#define UA(T, DD) hipLaunchKernelGGL((unalias_kernel<T, DD>), grid, dim3(256), 0, s, items, (const T*)lib_v, cap, cv)
  if (dtype == 0) { if (cv.head_dim == 64) UA(float, 64); else UA(float, 128); }
  else { if (cv.head_dim == 64) UA(bf16_t, 64); else UA(bf16_t, 128); }
#undef UA
  return check(hipGetLastError());
}

int launch_lib_ingest(int dtype, const void* k, const void* v, void* lib_k, void* lib_v, int L, int len, int Hkv,
                      int D, int64_t cap, int64_t tok_off, hipStream_t s) {
  const int vec = dtype == 0 ? 4 : 8;
  const int64_t n = (int64_t)len * Hkv * (D / vec);
  if (n == 0) return 0;
  dim3 grid((unsigned)((n + 255) / 256), L);
#define ING(T, DD)                                                                                          \
  hipLaunchKernelGGL((ingest_kernel<T, DD>), grid, dim3(256), 0, s, (const T*)k, (const T*)v, (T*)lib_k,    \
                     (T*)lib_v, len, Hkv, cap, tok_off)
  if (dtype == 0) { if (D == 64) ING(float, 64); else ING(float, 128); }
  else { if (D == 64) ING(bf16_t, 64); else ING(bf16_t, 128); }
#undef ING
  return check(hipGetLastError());
}

int launch_graft(int dtype, const GraftChunk* chunks, int n_chunks, const void* lib_k, const void* lib_v,
                 int64_t cap, const CacheView& cv, const double* inv_freq, int L, hipStream_t s, KTime tm) {
  if (n_chunks == 0) return 0;
  dim3 grid(n_chunks, cv.n_kv_heads, L);
#define GR(T, DD, PG)                                                                                       \
  hipExtLaunchKernelGGL((graft_kernel<T, DD, PG>), grid, dim3(256), 0, s, tm.start, tm.stop, 0, chunks, (const T*)lib_k,             \
                     (const T*)lib_v, cap, cv, inv_freq)
#define GRD(T, PG) { if (cv.head_dim == 64) GR(T, 64, PG); else GR(T, 128, PG); }
  const bool paged = cv.page_size != 0;
  if (dtype == 0) { if (paged) GRD(float, true) else GRD(float, false) }
  else { if (paged) GRD(bf16_t, true) else GRD(bf16_t, false) }
#undef GRD
#undef GR
  return check(hipGetLastError());
}

}  // namespace fcg
