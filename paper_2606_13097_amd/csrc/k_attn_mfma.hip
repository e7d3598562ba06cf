// Patch-prefill attention on gfx950 matrix cores (Sec. 4.2, Eq. 6: the patch
// span attends over the reused prefix KV states).  bf16 operands, fp32
// accumulation, fp32 online softmax in base 2.
//
// Block: 256 lanes = 4 waves, 128 query rows of one kv head (the g query heads
// of up to 128 / g consecutive tokens of one sequence), one split [k0, k1) of
// the key positions.  Wave w owns rows 32w .. 32w + 31 as two 16-row tiles.
//
// Per tile of 64 keys:
//   - the block stages K as rows [key][D] and V transposed [d][key] in LDS;
//     every lane copies four K vectors and transposes one 4-key x 8-dim V
//     block in registers (v_perm), so LDS writes are 16- and 8-byte vectors.
//     The next tile's global loads are issued, unconditionally (positions
//     clamped inside the split), before the current tile's math.
//   - S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (A = K from LDS, B = Q^T held
//     in registers for the whole block).  In the accumulator layout lane l
//     holds keys 4(l/16) .. +3 of a 16-key tile for query row l % 16, so each
//     lane owns one query row: the running max needs only two cross-lane
//     exchanges (lanes l ^ 16, l ^ 32) and the running sum none until the end.
//   - O^T += V^T P^T (A = V^T from LDS, B = P^T straight from the S^T
//     registers rounded to bf16: the k index of the two 16-key tiles that
//     make one 32-deep step is the same permutation in A and B).
// The causal mask is by position: key p is visible to a row at position q iff
// p <= q.  A block covering a row block's whole range writes the normalised
// output; otherwise a partial (max, sum, unnormalised output) for the combine.
#include "fcg_device.hpp"
#include "kernels.hpp"

namespace fcg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8_t, u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));

// two fp32 -> packed bf16 with the gfx950 conversion instruction (round to nearest even)
__device__ __forceinline__ uint32_t cvt_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((float2_t){lo, hi}, bf16x2_t));
}

__device__ __forceinline__ floatx4 mfma16x16x32(const uint4& a, const uint4& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

constexpr int kBM = 128;  // query rows per block
constexpr int kBN = 64;   // keys per tile

template <int D>
struct PrefillSmem {
  static constexpr int KROW = D + 8;      // bf16 elements per staged K row (16-byte pad)
  static constexpr int VROW = kBN + 8;    // bf16 elements per staged V^T row
  bf16_t k[kBN * KROW];
  bf16_t vt[D * VROW];
};

template <int D, bool PAGED>
__global__ void __launch_bounds__(256) attn_prefill_mfma_kernel(
    const AttnItem* __restrict__ items, const TokenMeta* __restrict__ meta, const bf16_t* __restrict__ qws,
    int rows_ws, CacheView cv, int layer, int Hq, bf16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_ml, int part_stride_rows) {
  constexpr int KS = D / 32;                 // 32-deep k steps over the head dimension
  constexpr int DT = D / 16;                 // 16-wide output tiles over the head dimension
  constexpr int KPT = kBN * D / 8 / 256;     // 16-byte K vectors per lane
  constexpr int VBLK = (kBN / 4) * (D / 8);  // 4-key x 8-dim V blocks (lanes 0 .. VBLK - 1)
  using Sm = PrefillSmem<D>;
  __shared__ Sm sm;

  const AttnItem it = items[blockIdx.x];
  const int hk = blockIdx.y;
  const int Hkv = cv.n_kv_heads;
  const int g = Hq / Hkv;
  const int t = threadIdx.x;
  const int w = t >> 6, lane = t & 63;
  const int lr = lane & 15, lq = lane >> 4;
  const int rows = it.n_rank * g;
  const float qscale = 1.4426950408889634f / sqrtf((float)D);

  // ---- query rows of this lane: one per 16-row tile (rows past the block's
  // last one load row 0 and are never written)
  int rpos[2];
  uint4 qf[2][KS];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int r = 32 * w + 16 * rt + lr;
    const int rl = r < rows ? r : 0;
    rpos[rt] = r < rows ? meta[it.rank0 + rl / g].pos : -1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[rt][ks] = ld16(qws + ((int64_t)hk * rows_ws + (int64_t)it.rank0 * g + rl) * D + ks * 32 + lq * 8);
  }
  const int pmax = meta[it.rank0 + it.n_rank - 1].pos;
  const int rmin = meta[it.rank0].pos;  // ranks ascend in position within a block
  const int kend = min(it.k1, pmax + 1);

  const bf16_t* ck = reinterpret_cast<const bf16_t*>(cv.k);
  const bf16_t* cvv = reinterpret_cast<const bf16_t*>(cv.v);

  // ---- tile loads: every lane KPT K vectors and (lanes < VBLK) one 4x8 V
  // block; positions past the split are clamped to its last key, whose
  // scores are masked, so every load is unconditional
  uint4 kpre[KPT], vpre[4];
  const int vkg = t % 16, vdc = t / 16;  // V block: keys 4 vkg .. +3, dims 8 vdc .. +7
  // contiguous caches: one base per (layer, sequence, head), 32-bit offsets after
  const int64_t head_base = PAGED ? 0 : kv_offset<false>(cv, layer, it.seq, hk, 0);
  auto row_off = [&](int p) -> int64_t {
    return PAGED ? kv_offset<true>(cv, layer, it.seq, hk, p) : head_base + (int64_t)(p * D);
  };
  auto load_tile = [&](int kb) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int idx = i * 256 + t;
      const int key = idx / (D / 8), c = idx % (D / 8);
      const int p = min(kb + key, kend - 1);
      kpre[i] = ld16(ck + row_off(p) + c * 8);
    }
    if (VBLK == 256 || t < VBLK) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = min(kb + vkg * 4 + i, kend - 1);
        vpre[i] = ld16(cvv + row_off(p) + vdc * 8);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int idx = i * 256 + t;
      const int key = idx / (D / 8), c = idx % (D / 8);
      st16(&sm.k[key * Sm::KROW + c * 8], kpre[i]);
    }
    if (VBLK == 256 || t < VBLK) {
      // vpre[i] = V[key 4 vkg + i][dims 8 vdc .. +7]; row e of the transpose holds
      // V[4 vkg .. 4 vkg + 3][8 vdc + e]
      const uint32_t* x = reinterpret_cast<const uint32_t*>(vpre);  // x[4i + e/2], half e%2
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t w01 = __builtin_amdgcn_perm(x[4 + e / 2], x[e / 2], sel);
        const uint32_t w23 = __builtin_amdgcn_perm(x[12 + e / 2], x[8 + e / 2], sel);
        *reinterpret_cast<uint2*>(&sm.vt[(vdc * 8 + e) * Sm::VROW + vkg * 4]) = make_uint2(w01, w23);
      }
    }
  };

  // ---- running state (per lane: its row of each row tile)
  float mrow[2] = {-INFINITY, -INFINITY};
  float lsum[2] = {0.f, 0.f};
  floatx4 acc[2][DT];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[rt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};

  if (it.k0 < kend) load_tile(it.k0);
  for (int kb = it.k0; kb < kend; kb += kBN) {
    __syncthreads();
    store_tile();
    __syncthreads();
    load_tile(kb + kBN);  // past the end it re-reads the clamped last key: no branch, no stall
    // keep the next tile's loads issued here, ahead of this tile's math (the
    // compiler would otherwise sink them to their LDS stores and serialise
    // memory latency with the matrix work)
    __asm__ volatile("" ::: "memory");

    // S^T = K Q^T: four 16-key tiles x two 16-row tiles
    floatx4 st[2][4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      uint4 ka[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) ka[ks] = ld16(&sm.k[(kt * 16 + lr) * Sm::KROW + ks * 32 + lq * 8]);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        floatx4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) c = mfma16x16x32(ka[ks], qf[rt][ks], c);
        st[rt][kt] = c;
      }
    }
    // mask (only tiles that reach past a row's position or the split's end),
    // running max, probabilities
    const bool need_mask = kb + kBN > kend || kb + kBN - 1 > rmin;
    uint4 pb[2][2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float tmax = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float sv = st[rt][kt][e] * qscale;
          if (need_mask) {
            const int p = kb + kt * 16 + lq * 4 + e;
            sv = (p <= rpos[rt] && p < kend) ? sv : -INFINITY;
          }
          st[rt][kt][e] = sv;
          tmax = fmaxf(tmax, sv);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      // lazy rescale: the reference max moves only when a row's max grows by
      // more than 2^8 (or on its first visible key); until then
      // probabilities stay below 2^8, harmless in fp32 and in bf16
      const bool grow = tmax > mrow[rt] + 8.f;
      if (__builtin_amdgcn_ballot_w64(grow)) {  // wave-uniform: any row of the wave
        const float mnew = fmaxf(mrow[rt], tmax);
        const float mref = mnew == -INFINITY ? 0.f : mnew;
        const float alpha = mrow[rt] == -INFINITY ? 0.f : exp2f(mrow[rt] - mref);
        mrow[rt] = mnew;
        lsum[rt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[rt][dt] *= alpha;
      }
      const float mref = mrow[rt] == -INFINITY ? 0.f : mrow[rt];
      float ps = 0.f;
      float pv[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pv[kt][e] = __builtin_amdgcn_exp2f(st[rt][kt][e] - mref);  // v_exp_f32: -inf gives 0
          ps += pv[kt][e];
        }
      lsum[rt] += ps;
      // B operand of step s (keys 32s .. 32s+31): tiles 2s (elements 0-3) and 2s+1 (elements 4-7)
#pragma unroll
      for (int s = 0; s < 2; ++s)
        pb[rt][s] = make_uint4(cvt_bf16x2(pv[2 * s][0], pv[2 * s][1]), cvt_bf16x2(pv[2 * s][2], pv[2 * s][3]),
                               cvt_bf16x2(pv[2 * s + 1][0], pv[2 * s + 1][1]),
                               cvt_bf16x2(pv[2 * s + 1][2], pv[2 * s + 1][3]));
    }
    // O^T += V^T P^T
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16_t* row = &sm.vt[(dt * 16 + lr) * Sm::VROW + s * 32 + lq * 4];
        const uint2 lo = *reinterpret_cast<const uint2*>(row);
        const uint2 hi = *reinterpret_cast<const uint2*>(row + 16);
        const uint4 va = make_uint4(lo.x, lo.y, hi.x, hi.y);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) acc[rt][dt] = mfma16x16x32(va, pb[rt][s], acc[rt][dt]);
      }
    }
  }

  // ---- epilogue: lane holds O^T[d = 16 dt + 4 lq + e][row lr] of each row tile
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    float l = lsum[rt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int r = 32 * w + 16 * rt + lr;
    if (r >= rows) continue;
    if (it.part < 0) {
      const float inv = l > 0.f ? 1.f / l : 0.f;
      const int tok = meta[it.rank0 + r / g].tok;
      bf16_t* o = out + ((int64_t)tok * Hq + hk * g + r % g) * D + lq * 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const floatx4 a = acc[rt][dt];
        *reinterpret_cast<uint2*>(o + dt * 16) =
            make_uint2(cvt_bf16x2(a[0] * inv, a[1] * inv), cvt_bf16x2(a[2] * inv, a[3] * inv));
      }
    } else {
      const int64_t pr = ((int64_t)it.part * Hkv + hk) * part_stride_rows + r;
      float* o = part_o + pr * D + lq * 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const floatx4 a = acc[rt][dt];
        *reinterpret_cast<float4*>(o + dt * 16) = make_float4(a[0], a[1], a[2], a[3]);
      }
      if (lq == 0) {
        part_ml[pr * 2 + 0] = mrow[rt];
        part_ml[pr * 2 + 1] = l;
      }
    }
  }
}

int launch_attn_mfma(const AttnItem* items, int n_items, const TokenMeta* meta, const void* qws, int rows_ws,
                     const CacheView& cv, int layer, int Hq, void* out, float* part_o, float* part_ml,
                     int part_stride_rows, hipStream_t s) {
  if (n_items == 0) return 0;
  dim3 grid(n_items, cv.n_kv_heads);
#define PF(DD, PG)                                                                                         \
  hipLaunchKernelGGL((attn_prefill_mfma_kernel<DD, PG>), grid, dim3(256), 0, s, items, meta, (const bf16_t*)qws, \
                     rows_ws, cv, layer, Hq, (bf16_t*)out, part_o, part_ml, part_stride_rows)
  const bool paged = cv.page_size != 0;
  if (cv.head_dim == 128) { if (paged) PF(128, true); else PF(128, false); }
  else { if (paged) PF(64, true); else PF(64, false); }
#undef PF
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
