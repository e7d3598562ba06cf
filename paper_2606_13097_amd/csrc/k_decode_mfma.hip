// One decode step at one layer on gfx950 matrix cores, bf16 caches (Sec.
// 4.2, Eq. 6: decoding over the reused, grafted KV states).
//
// Per sequence i the new token sits at position pos_i = its current length.
// Block (split s, sequence i, kv head h) attends the token's g query heads
// (g <= 16) over key positions [s * split_keys, min(pos_i + 1, (s + 1) *
// split_keys)).  Its four waves take the split's 16-key tiles in turn
// (w, w + 4, ...); per tile and wave:
//   - S^T = K Q^T with v_mfma_f32_16x16x32_bf16: A = the tile's keys straight
//     from memory into registers (lane l: key l % 16, dims 32 ks + 8 (l / 16)
//     .. + 7), B = the encoded queries, column j = query head j (columns past
//     g are zero).  Lane l then holds the scores of query l % 16 for keys
//     4 (l / 16) .. + 3.
//   - online softmax in base 2 with one running max per query shared by its
//     four lanes, moved only when a score exceeds it by 2^8 (ballot), so the
//     lanes exchange maxima (two shuffles) only then;
//   - O^T += V^T P^T with v_mfma_f32_16x16x16_bf16: B = the lane's four
//     probabilities rounded to bf16 (exactly the B layout), A = V^T read from
//     a per-wave LDS tile that each lane fills with one 4-key x 8-dim block
//     of V transposed in registers (v_perm).
// The block holding pos_i encodes the new key, stores key and value into the
// cache slot and keeps them in LDS; after its tiles, one wave attends to them
// as a one-key tile.  The four
// waves merge through LDS; the split's result goes to the output or, for a
// sequence with several splits, to its partial slot, and the last block of
// the sequence to finish merges the splits (decode_common.hpp).
#include "decode_common.hpp"

namespace fcg {
namespace {

typedef __bf16 dm_bf16x8 __attribute__((ext_vector_type(8)));
typedef short dm_i16x4 __attribute__((ext_vector_type(4)));
typedef float dm_f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 dm_bf16x2 __attribute__((ext_vector_type(2)));
typedef float dm_f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ dm_f32x4 mma_qk(const uint4& a, const uint4& b, const dm_f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(dm_bf16x8, a), __builtin_bit_cast(dm_bf16x8, b),
                                                 c, 0, 0, 0);
}
__device__ __forceinline__ dm_f32x4 mma_pv(const uint2& a, const uint2& b, const dm_f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(dm_i16x4, a), __builtin_bit_cast(dm_i16x4, b),
                                                   c, 0, 0, 0);
}
// two fp32 -> packed bf16, round to nearest even
__device__ __forceinline__ uint32_t dm_cvt_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((dm_f32x2){lo, hi}, dm_bf16x2));
}

}  // namespace

template <int D, int G, bool PAGED>
__global__ void __launch_bounds__(256) decode_mfma_kernel(DecodeArgs args, const bf16_t* __restrict__ q,
                                                          const bf16_t* __restrict__ k,
                                                          const bf16_t* __restrict__ v, CacheView cv,
                                                          const float2* __restrict__ rope,
                                                          bf16_t* __restrict__ out, float* __restrict__ part_o,
                                                          float* __restrict__ part_ml, int* __restrict__ count,
                                                          int layer) {
  static_assert(G >= 1 && G <= 16, "query group");
  constexpr int KS = D / 32;       // 32-deep k steps of S^T
  constexpr int DT = D / 16;       // 16-dim tiles of O^T
  constexpr int HALF = D / 2;
  constexpr int NDG = D / 8;       // 8-dim groups of a row
  constexpr int VBL = 4 * NDG;     // 4-key x 8-dim blocks of a 16-key tile
  // V^T in LDS: row r (a dim, 16 keys = 32 bytes) at element (r + r / 8) * 16,
  // a 32-byte gap after every 8 rows.  The writes (rows 8 dg + e of one e,
  // four 8-byte key groups each) and the reads (rows 16 dt .. + 15, all four
  // groups) then spread over every bank, so that each 512-byte access takes
  // the minimum number of LDS passes; with plain 32-byte rows the 16 rows of
  // a write, 8 apart, fall on the same 8 banks.
  constexpr int VT_ROWS = D + D / 8;
  constexpr int NSL = merge_lanes<bf16_t, D>();
  constexpr int GR = G < 4 ? G : 4;
  constexpr int NBUF = 4 * G * D > GR * NSL * D ? 4 * G * D : GR * NSL * D;
  __shared__ float s_cos[HALF], s_sin[HALF];
  __shared__ __align__(16) bf16_t s_vt[4][VT_ROWS * 16];
  __shared__ __align__(16) float s_buf[NBUF];
  __shared__ float s_wm[4][16], s_wl[4][16];
  __shared__ float s_mt[NSL * G], s_lt[NSL * G];
  __shared__ __align__(16) bf16_t s_newk[D], s_newv[D];  // the new token's encoded key and value
  __shared__ int s_last;
  // paged caches: the split's page and value-alias entries, read into LDS once
  // (a table lookup per tile would put a dependent load before every tile's loads)
  constexpr int NPG = PAGED ? kPageWindow : 1;
  __shared__ int32_t s_pg[NPG], s_al[NPG];

  const int split = blockIdx.x, i = blockIdx.y, hk = blockIdx.z;
  const int seq = args.seq[i], pos = args.pos[i], slot0 = args.split0[i];
  const int npage = PAGED ? args.new_page[i] : -1;  // a page this step maps, by value
  const int nsplit = args.split0[i + 1] - slot0;
  const int sk = args.split_keys;
  const bf16_t* ck = reinterpret_cast<const bf16_t*>(cv.k);
  const bf16_t* cvv = reinterpret_cast<const bf16_t*>(cv.v);
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
  const int w = t >> 6, l = t & 63, lr = l & 15, lq = l >> 4;
  const int kg = (l % VBL) / NDG, dg = l % NDG;  // this lane's V block: keys 4 kg .. + 3, dims 8 dg .. + 7
  const int k0 = split * sk;
  const int k1 = min(pos + 1, k0 + sk);
  const bool owns_new = k1 == pos + 1;   // the last split holds the new token
  const int kend = owns_new ? pos : k1;  // cached keys [k0, kend)
  const int ntile = (kend - k0 + 15) >> 4;

  // pages holding [ka, kend), ka = the lowest position a (clamped) load reads
  const int ka = max(0, min(k0, kend - 1));
  const int lpa = ka >> 4;
  const int npg = PAGED ? (max(ka, kend - 1) >> 4) - lpa + 1 : 0;
  const bool window = PAGED && npg <= NPG;  // else: entries read from memory per load (block-uniform)
  if (window) {
    const int32_t* row = cv.page_table + (int64_t)seq * 2 * cv.n_lp + lpa;
    for (int e = t; e < npg; e += 256) {
      s_pg[e] = row[e];
      s_al[e] = cv.v_alias ? row[cv.n_lp + e] : -1;
    }
  }

  // ---- loads, in the order their data is needed
  const float2 cs_pos = rope[(int64_t)pos * HALF + t % HALF];  // (cos, sin) of the position
  uint4 qa[KS], qb[KS];  // query head lr (row g - 1 for columns past the group): dims and rotary partners
  {
    const bf16_t* row = q + ((int64_t)i * Hq + hk * G + min(lr, G - 1)) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int d = ks * 32 + lq * 8;
      qa[ks] = ld16(row + d);
      qb[ks] = ld16(row + (d < HALF ? d + HALF : d - HALF));
    }
  }
  // the new token's key (dims and rotary partners) and value: lane t < D / 8
  // holds dims 8t .. 8t + 7 (loaded by every block, used by the owner's)
  const int dn = (t % NDG) * 8;
  uint4 na, nb, nv;
  {
    const bf16_t* krow = k + ((int64_t)i * Hkv + hk) * D;
    const bf16_t* vrow = v + ((int64_t)i * Hkv + hk) * D;
    na = ld16(krow + dn);
    nb = ld16(krow + (dn < HALF ? dn + HALF : dn - HALF));
    nv = ld16(vrow + dn);
  }
  // key and value rows of cached position p (p in [ka, kend))
  auto k_ptr = [&](int p) -> const bf16_t* {
    if (window) {
      const int32_t page = s_pg[(p >> 4) - lpa];
      return ck + (int64_t)layer * cv.layer_stride + (((int64_t)page * Hkv + hk) * 16 + (p & 15)) * D;
    }
    return ck + kv_offset<PAGED>(cv, layer, seq, hk, p);
  };
  auto v_ptr = [&](int p) -> const bf16_t* {
    if (window) {
      const int e = (p >> 4) - lpa;
      const int32_t a = s_al[e];
      if (a >= 0)
        return reinterpret_cast<const bf16_t*>(cv.lib_v) +
               (((int64_t)layer * Hkv + hk) * cv.lib_cap + a + (p & 15)) * D;
      return cvv + (int64_t)layer * cv.layer_stride + (((int64_t)s_pg[e] * Hkv + hk) * 16 + (p & 15)) * D;
    }
    return v_row<PAGED, bf16_t>(cv, layer, seq, hk, p);
  };
  if (window) __syncthreads();  // the page window is in LDS (a block-uniform branch)
  // a tile's keys (A layout) and V block; keys past the range re-read the last key
  auto load_tile = [&](int ti, uint4 (&kk)[KS], uint4 (&vv)[4]) {
    const int kb = k0 + ti * 16;
    const bf16_t* kr = k_ptr(max(0, min(kb + lr, kend - 1))) + lq * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kk[ks] = ld16(kr + ks * 32);
#pragma unroll
    for (int r = 0; r < 4; ++r) vv[r] = ld16(v_ptr(max(0, min(kb + 4 * kg + r, kend - 1))) + dg * 8);
  };
  // The loads above go out first: the position's (cos, sin), which the
  // barrier below waits for, and the query.  Left to itself the scheduler
  // issues them after the tiles' loads, and that wait then drains the whole
  // split before the first tile is attended.  Only the wave's first tile
  // follows them before the encoding; its next two go out after it (below):
  // with every block's whole split requested at once, the query and the
  // rotary pair wait behind that burst (7B decode call 12.0 -> 11.5 us).
  __builtin_amdgcn_sched_barrier(0);
  uint4 kA[KS], vA[4], kB[KS], vB[4], kC[KS], vC[4];
  load_tile(w, kA, vA);
  if (t < HALF) {
    s_cos[t] = cs_pos.x;
    s_sin[t] = cs_pos.y;
  }
  __syncthreads();

  // rotate 8 dims d .. d + 7 given (own dims, partner dims), round to bf16
  auto encode8 = [&](int d, const uint4& xa, const uint4& xb) -> uint4 {
    float a[8], b[8], y[8];
    Store<bf16_t>::unpack(xa, a);
    Store<bf16_t>::unpack(xb, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ii = (d + e) % HALF;
      const float c = s_cos[ii], sn = s_sin[ii];
      y[e] = d < HALF ? fmaf(a[e], c, -b[e] * sn) : fmaf(a[e], c, b[e] * sn);
    }
    return Store<bf16_t>::pack(y);
  };
  uint4 qB[KS];  // Q^T operand: column lr
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const uint4 e = encode8(ks * 32 + lq * 8, qa[ks], qb[ks]);
    qB[ks] = lr < G ? e : make_uint4(0u, 0u, 0u, 0u);
  }
  if (PAGED && owns_new && hk == 0 && t == 0 && npage >= 0) enter_page(cv, seq, pos, npage);
  if (owns_new && t < NDG) {
    // encode the new key, store key and value into the token's cache slot and
    // keep both in LDS for the wave that attends to them
    const uint4 kn = encode8(dn, na, nb);
    const int64_t off = new_token_offset<PAGED>(cv, layer, seq, hk, pos, npage) + dn;
    st16(reinterpret_cast<bf16_t*>(cv.k) + off, kn);
    st16(reinterpret_cast<bf16_t*>(cv.v) + off, nv);
    st16(&s_newk[dn], kn);
    st16(&s_newv[dn], nv);
  }
  __builtin_amdgcn_sched_barrier(0);
  load_tile(w + 4, kB, vB);
  load_tile(w + 8, kC, vC);
  const float qscale = 1.4426950408889634f / sqrtf((float)D);

  float mref = -INFINITY, lsum = 0.f;  // running max (log2 units) of query lr, sum of this lane's keys
  dm_f32x4 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = dm_f32x4{0.f, 0.f, 0.f, 0.f};
  bf16_t* vt = s_vt[w];

  // attend one tile: keys kb .. kb + 15, the first nvalid of them real
  auto attend_tile = [&](const uint4 (&kk)[KS], const uint4 (&vv)[4], int kb, int nvalid) {
    // V^T block into LDS: row e of the block = V[4 kg .. 4 kg + 3][8 dg + e]
    if (l < VBL) {
      const uint32_t* x = reinterpret_cast<const uint32_t*>(vv);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t w01 = __builtin_amdgcn_perm(x[4 + e / 2], x[e / 2], sel);
        const uint32_t w23 = __builtin_amdgcn_perm(x[12 + e / 2], x[8 + e / 2], sel);
        *reinterpret_cast<uint2*>(&vt[(dg * 9 + e) * 16 + kg * 4]) = make_uint2(w01, w23);  // row 8 dg + e
      }
    }
    dm_f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) s = mma_qk(kk[ks], qB[ks], s);
    float x[4], lmax = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      x[r] = 4 * lq + r < nvalid ? s[r] * qscale : -INFINITY;
      lmax = fmaxf(lmax, x[r]);
    }
    if (__builtin_amdgcn_ballot_w64(lmax > mref + 8.f)) {
      // exact running max of each query over its four lanes
      const float mn = max_rows4(fmaxf(mref, lmax));
      const float f = __builtin_amdgcn_exp2f(mref - mn);  // 0 while nothing was seen
      lsum *= f;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[dt] *= f;
      mref = mn;
    }
    float p[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      p[r] = __builtin_amdgcn_exp2f(x[r] - mref);  // 0 for keys past the tile's real ones
      lsum += p[r];
    }
    const uint2 pb = make_uint2(dm_cvt_bf16x2(p[0], p[1]), dm_cvt_bf16x2(p[2], p[3]));
    asm volatile("" ::: "memory");  // the wave's V^T writes come before its reads (LDS is in order per wave)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int r = dt * 16 + lr;
      const uint2 a = *reinterpret_cast<const uint2*>(&vt[(r + (r >> 3)) * 16 + 4 * lq]);
      acc[dt] = mma_pv(a, pb, acc[dt]);
    }
    asm volatile("" ::: "memory");  // ... and before the next tile's writes
  };

  // three register sets: the wave's next two tiles are in flight while one
  // is attended (a 192-key split is requested entirely before its first
  // tile is attended)
  for (int ti = w; ti < ntile; ti += 12) {
    attend_tile(kA, vA, k0 + ti * 16, min(16, kend - k0 - ti * 16));
    load_tile(ti + 12, kA, vA);
    if (ti + 4 >= ntile) break;
    attend_tile(kB, vB, k0 + (ti + 4) * 16, min(16, kend - k0 - (ti + 4) * 16));
    load_tile(ti + 16, kB, vB);
    if (ti + 8 >= ntile) break;
    attend_tile(kC, vC, k0 + (ti + 8) * 16, min(16, kend - k0 - (ti + 8) * 16));
    load_tile(ti + 20, kC, vC);
  }

  if (owns_new) __syncthreads();  // the new token is in LDS (a block-uniform branch)
  if (owns_new && w == (ntile & 3)) {
    // the new token as a one-key tile: key row 0, V block of keys 0 .. 3
    uint4 kn[KS], vn[4];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kn[ks] = lr == 0 ? *reinterpret_cast<const uint4*>(&s_newk[ks * 32 + lq * 8]) : make_uint4(0u, 0u, 0u, 0u);
    vn[0] = kg == 0 ? *reinterpret_cast<const uint4*>(&s_newv[dg * 8]) : make_uint4(0u, 0u, 0u, 0u);
    vn[1] = vn[2] = vn[3] = make_uint4(0u, 0u, 0u, 0u);
    attend_tile(kn, vn, pos, 1);
  }

  // ---- merge the four waves: per query, M over the waves, each wave's
  // output and sum weighted by 2^(m - M)
  lsum = sum_rows4(lsum);
  if (lr < G) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<float4*>(&s_buf[(w * G + lr) * D + dt * 16 + 4 * lq]) =
          make_float4(acc[dt][0], acc[dt][1], acc[dt][2], acc[dt][3]);
    if (lq == 0) {
      s_wm[w][lr] = mref;
      s_wl[w][lr] = lsum;
    }
  }
  __syncthreads();
  for (int idx = t; idx < G * D / 2; idx += 256) {
    const int j = idx / (D / 2), d = 2 * (idx % (D / 2));
    float M = -INFINITY;
#pragma unroll
    for (int w2 = 0; w2 < 4; ++w2) M = fmaxf(M, s_wm[w2][j]);
    float L = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < 4; ++w2) {
      const float m = s_wm[w2][j];
      const float f = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
      const float2 o = *reinterpret_cast<const float2*>(&s_buf[(w2 * G + j) * D + d]);
      L = fmaf(s_wl[w2][j], f, L);
      a0 = fmaf(o.x, f, a0);
      a1 = fmaf(o.y, f, a1);
    }
    emit_pair<bf16_t, D>(nsplit, part_row(slot0 + split, Hkv, hk, G, j), out + ((int64_t)i * Hq + hk * G + j) * D,
                         part_o, part_ml, d, a0, a1, M, L);
  }
  if (nsplit == 1) return;
  merge_splits<bf16_t, D, G, NBUF>(args, i, hk, slot0, nsplit, Hkv, Hq, out, part_o, part_ml, count, s_buf, s_mt,
                                   s_lt, &s_last);
}

int launch_decode_mfma(const DecodeArgs& args, const void* q, const void* k, const void* v, const CacheView& cv,
                       int layer, const float2* rope, int Hq, void* out, float* part_o, float* part_ml,
                       int* count, hipStream_t s, KTime tm) {
  if (args.n == 0) return 0;
  const int g = Hq / cv.n_kv_heads;
  dim3 grid(args.max_split, args.n, cv.n_kv_heads);
#define DM1(DD, GG, PG)                                                                                       \
  hipExtLaunchKernelGGL((decode_mfma_kernel<DD, GG, PG>), grid, dim3(256), 0, s, tm.start, tm.stop, 0, args,   \
                        (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, cv, rope, (bf16_t*)out, part_o,   \
                        part_ml, count, layer)
#define DM(DD, GG)                                                                                            \
  if (cv.page_size) DM1(DD, GG, true);                                                                        \
  else DM1(DD, GG, false)
#define DMG(DD)                                                                                               \
  switch (g) {                                                                                                \
    case 1: DM(DD, 1); break;                                                                                 \
    case 2: DM(DD, 2); break;                                                                                 \
    case 4: DM(DD, 4); break;                                                                                 \
    case 8: DM(DD, 8); break;                                                                                 \
    case 16: DM(DD, 16); break;                                                                               \
    default: return -1;                                                                                       \
  }
  if (cv.head_dim == 64) { DMG(64) } else { DMG(128) }
#undef DMG
#undef DM
#undef DM1
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
