// Patch-prefill attention on gfx950 matrix cores (Sec. 4.2, Eq. 6: the patch
// span attends over the reused prefix KV states).  bf16 operands, fp32
// accumulation, fp32 online softmax in base 2.
//
// Block: 4 or 8 waves of one kv head (the g query heads of consecutive tokens
// of one sequence) and one split [k0, k1) of the key positions.  Wave w owns
// RT 16-row tiles of query rows, rows 16 RT w .. 16 RT (w + 1) - 1.  The host
// picks the shape per call: 128-row blocks of 4 waves x 32 rows sized to run
// two per CU (the two blocks' softmax and matrix phases overlap); the same
// rows as 8 waves x 16 rows, one block per CU, when short key splits make the
// call latency-bound; or, when 256-row blocks alone fill the chip twice, 8
// waves x 32 rows one per CU.
//
// Key tiles of 64 keys go from memory straight into LDS (global_load_lds:
// each instruction fills 1 KB, 16 bytes per lane), into a ring of two or four
// single-tile buffers, so up to three tiles are in flight while one is
// attended and staging costs no registers.  K and V keep their [key][D] rows; the 16-byte
// chunks of each row are XOR-swizzled so that the reads below meet no bank
// conflicts.  Then per tile:
//   - S^T = K Q^T with v_mfma_f32_16x16x32_bf16 (A = K from LDS, B = Q^T held
//     in registers for the whole block).  In the accumulator layout lane l
//     holds keys 4(l/16) .. +3 of a 16-key tile for query row l % 16, so each
//     lane owns one query row: the running max needs only two cross-lane
//     exchanges (lanes l ^ 16, l ^ 32) and the running sum none until the end.
//   - O^T += V^T P^T (A = V^T read from the V rows with the LDS transpose read
//     ds_read_b64_tr_b16, B = P^T straight from the S^T registers rounded to
//     bf16: the k index of the two 16-key tiles that make one 32-deep step is
//     the same permutation in A and B).
// The causal mask is by position: key p is visible to a row at position q iff
// p <= q.  A block covering a row block's whole range writes the normalised
// output; otherwise a partial (max, sum, unnormalised output) for the combine.
#include <type_traits>

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

constexpr int kBN = 64;    // keys per tile
constexpr int kXcds = 8;   // accelerator dies (XCDs) of the MI355X, each with its own L2

template <int D>
struct PrefillTile {
  // [key][D] rows, 16-byte chunk c of row r at chunk position c ^ swz(r):
  //  - K is read as MFMA A fragments, 16 bytes per lane from 16 rows x 4
  //    chunks: swz_k(r) = r % NC puts every 8 (and every 16) lanes' reads in
  //    distinct banks;
  //  - V is read with ds_read_b64_tr_b16, 8 bytes per lane from 4 rows x 2
  //    chunks per 16 lanes: swz_v(r) = 2 (r % (NC / 2)) does the same.
  static constexpr int NC = D / 8;  // 16-byte chunks per row
  bf16_t k[kBN * D];
  bf16_t v[kBN * D];
  __device__ static int swz_k(int r) { return r % NC; }
  __device__ static int swz_v(int r) { return 2 * (r % (NC / 2)); }
};

// LDS byte address of a pointer into a __shared__ array
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// global -> LDS, 16 bytes per lane: lane l's bytes land at lds + 16 l (lds
// wave-uniform).  Inline assembly, so that the compiler's own wait
// bookkeeping, which cannot tell the ring's buffers apart, adds no
// vmcnt(0) before each tile's LDS reads; the waits are explicit (wait_vm).
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}
// s_waitcnt vmcnt(N): at most N of this wave's vector memory operations remain
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// this wave's LDS reads have returned, then the workgroup barrier
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

typedef short i16x4_t __attribute__((ext_vector_type(4)));
// ds_read_b64_tr_b16: within each 16-lane group, lane j receives element j % 4
// of the 8 bytes addressed by lanes 4e + j / 4, e = 0..3
__device__ __forceinline__ uint2 ld_tr8(const bf16_t* p) {
  const i16x4_t x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4_t*)(const_cast<bf16_t*>(p)));
  return __builtin_bit_cast(uint2, x);
}

// grid (row block, key split, kv head).  Each wave attends RT 16-row tiles
// of the block's query rows (WAVES * RT * 16 rows).  NBUF tiles in the LDS
// ring: 4 (three in flight while one is attended) for 8-wave blocks of 32-row
// waves and 4-wave blocks of the plain one-per-CU plan, 2 (132 KB against
// 68 KB of LDS at D 128) for 4-wave blocks planned two per CU, whose phases
// then overlap (one block's softmax beside the other's matrix work), and for
// 128-row blocks of 8 waves x 16 rows planned one per CU (two waves per SIMD
// again, each with half the row tiles).  4-wave blocks aim at 256 registers
// per lane (two waves per SIMD); the four-tile ring at D 128 still needs more,
// and the compiler keeps its accumulators in AGPRs.
template <int D, bool PAGED, int WAVES, int NBUF, bool FUSED, int RT>
__global__ void __launch_bounds__(WAVES * 64, WAVES == 4 ? 2 : 1) attn_prefill_mfma_kernel(
    PrefillArgs args, const TokenMeta* __restrict__ meta, const bf16_t* __restrict__ qws, int rows_ws,
    CacheView cv, int layer, int Hq, bf16_t* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_ml, int part_stride_rows, const bf16_t* __restrict__ raw_q,
    const bf16_t* __restrict__ raw_k, const bf16_t* __restrict__ raw_v, const float2* __restrict__ rope) {
  constexpr int NT = WAVES * 64;                    // lanes per block
  constexpr int KS = D / 32;                        // 32-deep k steps over the head dimension
  constexpr int DT = D / 16;                        // 16-wide output tiles over the head dimension
  using Tile = PrefillTile<D>;
  constexpr int NC = Tile::NC;
  constexpr int HALF = D / 2;
  constexpr int DPT = 2 * NC / WAVES;               // LDS loads per wave per tile (1 KB each)
  static_assert(NC % WAVES == 0, "tile loads split evenly over the waves");
  constexpr int kNBuf = NBUF;
  __shared__ Tile tiles[kNBuf];
  // paged caches: the split's page and value-alias entries, read into LDS once
  // (a table lookup per row would put a dependent load before every tile's loads)
  constexpr int NPG = PAGED ? kPageWindow : 1;
  __shared__ int32_t s_pg[NPG], s_al[NPG];

  // Block order.  Plain: grid (row block, split, kv head).  XCD-grouped
  // (args.xcd_group): workgroups are dealt to the eight XCDs in turn by
  // linear id (x fastest), so the row blocks that read the same key tiles
  // (one group = one split of one kv head) get ids 8 apart and run on one XCD,
  // whose L2 then serves the tiles after the first read: blockIdx.x = 8 r + x
  // (row block r), blockIdx.y = q, group 8 q + x, numbered kv head fastest so
  // that every XCD gets all the splits of its heads (late splits, which the
  // causal mask leaves to fewer row blocks, spread over the XCDs).  Ids past
  // the last group exit.
  const int Hkv = cv.n_kv_heads;
  // Every kernel argument the block reads is fetched in one batch of scalar
  // loads before the first branch: left to the compiler, the loads are placed
  // next to their uses, and a load whose address depends on a loaded value
  // (the row block, indexed by an id that depends on the launch's order) waits
  // for a round trip of its own.  So both candidate row blocks are fetched
  // (indices from the block id alone, clamped into the array) and one is
  // chosen once the batch has landed.
  const PrefillRb rb_plain = args.rb[min((int)blockIdx.x, kPfMaxRb - 1)];
  const PrefillRb rb_xcd = args.rb[blockIdx.x / kXcds];
  const bf16_t* ck = reinterpret_cast<const bf16_t*>(cv.k);
  const bf16_t* cvv = reinterpret_cast<const bf16_t*>(cv.v);
  asm volatile("" ::"s"(rb_plain.rank0), "s"(rb_plain.n_rank), "s"(rb_plain.seq), "s"(rb_plain.rmin),
               "s"(rb_plain.pmax), "s"(rb_plain.part0), "s"(rb_xcd.rank0), "s"(rb_xcd.n_rank), "s"(rb_xcd.seq),
               "s"(rb_xcd.rmin), "s"(rb_xcd.pmax), "s"(rb_xcd.part0), "s"(args.n_rb), "s"(args.n_split),
               "s"(args.span), "s"(args.xcd_group));
  asm volatile("" ::"s"(meta), "s"(qws), "s"(rows_ws), "s"(ck), "s"(cvv), "s"(cv.layer_stride), "s"(cv.max_tokens),
               "s"(Hkv), "s"(layer), "s"(Hq), "s"(out), "s"(part_o), "s"(part_ml), "s"(part_stride_rows));
  if (PAGED) asm volatile("" ::"s"(cv.page_table), "s"(cv.n_lp), "s"(cv.v_alias), "s"(cv.lib_v), "s"(cv.lib_cap));
  if (FUSED)
    asm volatile("" ::"s"(rb_plain.f0), "s"(rb_plain.ftok0), "s"(rb_xcd.f0), "s"(rb_xcd.ftok0), "s"(raw_q), "s"(raw_k),
                 "s"(raw_v), "s"(rope));
  __builtin_amdgcn_sched_barrier(0);
  int split, hk;
  if (args.xcd_group) {
    const int grp = blockIdx.y * kXcds + blockIdx.x % kXcds;
    split = grp / Hkv;
    hk = grp % Hkv;
  } else {
    split = blockIdx.y;
    hk = blockIdx.z;
  }
  // chosen field by field: a select of the whole struct was lowered to a copy
  // of both candidates into scratch memory and a load at a computed offset
  const bool xg = args.xcd_group != 0;
  PrefillRb rb;
  rb.rank0 = xg ? rb_xcd.rank0 : rb_plain.rank0;
  rb.n_rank = xg ? rb_xcd.n_rank : rb_plain.n_rank;
  rb.seq = xg ? rb_xcd.seq : rb_plain.seq;
  rb.rmin = xg ? rb_xcd.rmin : rb_plain.rmin;
  rb.pmax = xg ? rb_xcd.pmax : rb_plain.pmax;
  rb.part0 = xg ? rb_xcd.part0 : rb_plain.part0;
  rb.f0 = xg ? rb_xcd.f0 : rb_plain.f0;
  rb.ftok0 = xg ? rb_xcd.ftok0 : rb_plain.ftok0;
  const int k0 = split * args.span;
  const int kend = min(rb.pmax + 1, k0 + args.span);
  const int part = rb.part0 < 0 ? -1 : rb.part0 + split;
  if (split >= args.n_split || k0 >= kend) return;  // past the last group; padding split of a shorter row block
  const int g = Hq / Hkv;
  const int t = threadIdx.x;
  const int lpa = k0 >> 4;
  const int npg = PAGED ? ((kend - 1) >> 4) - lpa + 1 : 0;
  const bool window = PAGED && npg <= NPG;  // else: entries read from memory per row (block-uniform)
  if (window) {
    const int32_t* row = cv.page_table + (int64_t)rb.seq * 2 * cv.n_lp + lpa;
    for (int e = t; e < npg; e += NT) {
      s_pg[e] = row[e];
      s_al[e] = cv.v_alias ? row[cv.n_lp + e] : -1;
    }
    __syncthreads();
  }
  const int w = t >> 6, lane = t & 63;
  const int wu = __builtin_amdgcn_readfirstlane(w);  // the wave index, in a scalar register
  const int lr = lane & 15, lq = lane >> 4;
  const int rows = rb.n_rank * g;
  const float qscale = 1.4426950408889634f / sqrtf((float)D);

  // contiguous caches address a head's rows from one base with 32-bit offsets
  const int64_t head_base = PAGED ? 0 : kv_offset<false>(cv, layer, rb.seq, hk, 0);
  const bf16_t* kbase = ck + head_base;
  const bf16_t* vbase = cvv + head_base;
  // rows of positions in [k0, kend)
  auto krow = [&](int p) -> const bf16_t* __attribute__((always_inline)) {
    if (!PAGED) return kbase + p * D;
    if (window)
      return ck + (int64_t)layer * cv.layer_stride +
             (((int64_t)s_pg[(p >> 4) - lpa] * Hkv + hk) * 16 + (p & 15)) * D;
    return ck + kv_offset<true>(cv, layer, rb.seq, hk, p);
  };
  auto vrow = [&](int p) -> const bf16_t* __attribute__((always_inline)) {
    if (!PAGED) return vbase + p * D;
    if (window) {
      const int e = (p >> 4) - lpa;
      const int32_t a = s_al[e];
      if (a >= 0)
        return reinterpret_cast<const bf16_t*>(cv.lib_v) +
               (((int64_t)layer * Hkv + hk) * cv.lib_cap + a + (p & 15)) * D;
      return cvv + (int64_t)layer * cv.layer_stride + (((int64_t)s_pg[e] * Hkv + hk) * 16 + (p & 15)) * D;
    }
    return v_row<true, bf16_t>(cv, layer, rb.seq, hk, p);
  };
  // the cache's own value row of position p (fresh tokens' pages are never read from the library)
  auto vown = [&](int p) -> const bf16_t* __attribute__((always_inline)) {
    if (!PAGED) return vbase + p * D;
    if (window)
      return cvv + (int64_t)layer * cv.layer_stride + (((int64_t)s_pg[(p >> 4) - lpa] * Hkv + hk) * 16 + (p & 15)) * D;
    return cvv + kv_offset<true>(cv, layer, rb.seq, hk, p);
  };
  // This wave's share of tile `tile` into its ring buffer: instruction j of
  // the tile (K: 0 .. NC - 1, V: NC .. 2 NC - 1) fills slots 64 j' .. 64 j' + 63
  // of the K or V rows, lane l the slot of row (64 j' + l) / NC at chunk
  // position (64 j' + l) % NC, so it loads the chunk that the swizzle puts
  // there.  Keys past the split read its last key (valid memory; masked).
  const int ntiles = (kend - k0 + kBN - 1) / kBN;
  auto issue_to = [&](int tile, Tile& B) __attribute__((always_inline)) {
    const int kb = k0 + tile * kBN;
#pragma unroll
    for (int u = 0; u < DPT; ++u) {
      const bool isv = WAVES * u >= NC;  // compile-time: instructions u < NC / WAVES are K
      const int jj = wu + WAVES * u - (isv ? NC : 0);
      const int slot = jj * 64 + lane;
      const int r = slot / NC, pos = slot % NC;
      const int p = min(kb + r, kend - 1);
      const int c = pos ^ (isv ? Tile::swz_v(r) : Tile::swz_k(r));
      const bf16_t* src;
      if (FUSED && p >= rb.f0)  // a fresh token: its raw row from the caller's input (keys turned below)
        src = (isv ? raw_v : raw_k) + ((int64_t)(rb.ftok0 + p - rb.f0) * Hkv + hk) * D + c * 8;
      else
        src = (isv ? vrow(p) : krow(p)) + c * 8;
      dma16(src, lds_addr(isv ? B.v : B.k) + jj * 1024);
    }
  };
  // Prologue.  Tile 0 goes in flight first, then the query rows (and the
  // metadata) are loaded, then the remaining kNBuf - 2 tiles.  The compiler
  // cannot see the tile loads (inline assembly), so its wait for the query
  // loads counts none of them and drains every load issued so far: issued in
  // this order, that wait covers tile 0 only, which step 0 needs anyway,
  // and leaves the later tiles in flight.
  // fused: the rotary table rows of the block's tokens (consecutive positions,
  // so one contiguous run of n_rank * D/2 (cos, sin) pairs) go first, into the
  // ring buffer that the prologue leaves free, when they fit; else each lane
  // reads its pairs from the table
  const int cs_bytes = FUSED ? rb.n_rank * HALF * 8 : 0;
  const bool stage_cs = FUSED && cs_bytes <= (int)sizeof(Tile);
  if (FUSED && stage_cs) {
    const int nchunk = cs_bytes / 16;  // 16-byte chunks, 64 per instruction
    const uint4* src = reinterpret_cast<const uint4*>(rope + (int64_t)rb.rmin * HALF);
    for (int j = wu; j * 64 < nchunk; j += WAVES)
      dma16(src + min(j * 64 + lane, nchunk - 1), lds_addr(&tiles[kNBuf - 1]) + j * 1024);
  }
  issue_to(0, tiles[0]);  // ntiles >= 1: the split is not empty
  // query rows of this lane: one per 16-row tile (rows past the block's last
  // one load row 0 and are never written)
  int rpos[RT], rtok[RT];  // position (of row 0 for rows past the block) and token of the lane's rows
  uint4 qf[RT][KS];
  // fused: the raw query dims of the lane, encoded once they and tile 0 have
  // landed.  The rotary partner of dims d (d +- D/2) is the lane's own k step
  // ks ^ (D / 64).
  uint4 qa[RT][FUSED ? KS : 1];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = 16 * (RT * w + rt) + lr;
    const int rl = r < rows ? r : 0;
    if constexpr (FUSED) {
      // the block's tokens are consecutive positions from rmin, consecutive caller indices
      const int tr = rl / g;
      rpos[rt] = rb.rmin + tr;
      rtok[rt] = rb.ftok0 + (rb.rmin - rb.f0) + tr;
      const bf16_t* row = raw_q + ((int64_t)rtok[rt] * Hq + hk * g + rl % g) * D;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qa[rt][ks] = ld16(row + ks * 32 + lq * 8);
    } else {
      const TokenMeta m = meta[rb.rank0 + rl / g];
      rpos[rt] = m.pos;
      rtok[rt] = m.tok;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[rt][ks] = ld16(qws + ((int64_t)hk * rows_ws + (int64_t)rb.rank0 * g + rl) * D + ks * 32 + lq * 8);
    }
  }
  if constexpr (FUSED) {
    // encode the queries at their positions (rotate-half pairs, fp32 turn,
    // rounded to bf16 by the conversion instruction: nearest even, as the
    // append kernel rounds)
    if (stage_cs) {
      wait_vm<0>();  // the table rows, tile 0 and the raw queries have landed
      lds_barrier();
    }
    const uint4* cs_lds = reinterpret_cast<const uint4*>(&tiles[kNBuf - 1]);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int d = ks * 32 + lq * 8;
        const int i0 = d % HALF;  // first pair index of the lane's 8 dims
        uint4 cw[4];
        if (stage_cs) {
          const uint4* c4 = cs_lds + (((rpos[rt] - rb.rmin) * HALF + i0) >> 1);
#pragma unroll
          for (int e = 0; e < 4; ++e) cw[e] = c4[e];
        } else {
          const uint4* c4 = reinterpret_cast<const uint4*>(rope + (int64_t)rpos[rt] * HALF + i0);
#pragma unroll
          for (int e = 0; e < 4; ++e) cw[e] = c4[e];
        }
        const float* cs = reinterpret_cast<const float*>(cw);  // (cos, sin) x 8
        float a[8], b[8], y[8];
        Store<bf16_t>::unpack(qa[rt][ks], a);
        Store<bf16_t>::unpack(qa[rt][ks ^ (HALF / 32)], b);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          y[e] = d < HALF ? fmaf(a[e], cs[2 * e], -b[e] * cs[2 * e + 1]) : fmaf(a[e], cs[2 * e], b[e] * cs[2 * e + 1]);
        qf[rt][ks] = make_uint4(cvt_bf16x2(y[0], y[1]), cvt_bf16x2(y[2], y[3]), cvt_bf16x2(y[4], y[5]),
                                cvt_bf16x2(y[6], y[7]));
      }
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" ::"v"(__builtin_bit_cast(u32x4_t, qf[rt][ks])));
    asm volatile("" ::"v"(rpos[rt]), "v"(rtok[rt]));
  }
#pragma unroll
  for (int i = 1; i < kNBuf - 1; ++i)
    if (i < ntiles) issue_to(i, tiles[i]);
  float mrow[RT], lsum[RT];
  floatx4 acc[RT][DT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    mrow[rt] = -INFINITY;
    lsum[rt] = 0.f;
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[rt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // One tile, in ring buffer `buf`, a std::integral_constant (each step of the
  // unrolled loop its own instantiation, every LDS address a constant offset
  // from a per-lane base).
  auto step = [&](int tile, auto buf) __attribute__((always_inline)) {
    const Tile& T = tiles[buf];
    // this wave's loads of the tile have landed (the later tiles in flight,
    // up to kNBuf - 2 of them, may still be pending) ...
    const int ahead = min(kNBuf - 2, ntiles - 1 - tile);
    if (ahead >= 2) wait_vm<2 * DPT>();
    else if (ahead == 1) wait_vm<DPT>();
    else wait_vm<0>();
    if constexpr (FUSED) {
      // keys of fresh tokens arrived raw: turn them in place.  Lane l's chunk c
      // of row r and its rotary partner c ^ NC/2 (lane l ^ NC/2, same
      // instruction) both came with this wave's loads; the wave reads both
      // chunks before it writes (LDS executes a wave's instructions in order).
      const int kb = k0 + tile * kBN;
      if (kb + kBN > rb.f0 && rb.f0 < kend) {  // the tile holds fresh keys (block-uniform)
        Tile& W = tiles[buf];
#pragma unroll
        for (int u = 0; u < NC / WAVES; ++u) {
          const int slot = (wu + WAVES * u) * 64 + lane;
          const int r = slot / NC, cpos = slot % NC;
          const int p = kb + r;
          if (p >= rb.f0 && p < kend) {
            const int c = cpos ^ Tile::swz_k(r);
            uint4* own = reinterpret_cast<uint4*>(&W.k[slot * 8]);
            const uint4* par = reinterpret_cast<const uint4*>(&W.k[(slot ^ (NC / 2)) * 8]);
            const uint4 xa = *own, xb = *par;
            const uint4* csp = reinterpret_cast<const uint4*>(rope + (int64_t)p * HALF + (c % (NC / 2)) * 8);
            float a[8], b[8];
            uint32_t yw[4];
            Store<bf16_t>::unpack(xa, a);
            Store<bf16_t>::unpack(xb, b);
#pragma unroll
            for (int h = 0; h < 2; ++h) {  // four dims at a time: (cos, sin) of pairs i0 + 4h .. + 3
              const uint4 c0 = csp[2 * h], c1 = csp[2 * h + 1];
              const float cs[8] = {__uint_as_float(c0.x), __uint_as_float(c0.y), __uint_as_float(c0.z),
                                   __uint_as_float(c0.w), __uint_as_float(c1.x), __uint_as_float(c1.y),
                                   __uint_as_float(c1.z), __uint_as_float(c1.w)};
              float y[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int de = 4 * h + e;
                y[e] = c < NC / 2 ? fmaf(a[de], cs[2 * e], -b[de] * cs[2 * e + 1])
                                  : fmaf(a[de], cs[2 * e], b[de] * cs[2 * e + 1]);
              }
              yw[2 * h] = cvt_bf16x2(y[0], y[1]);
              yw[2 * h + 1] = cvt_bf16x2(y[2], y[3]);
            }
            asm volatile("" ::: "memory");  // both chunks are read before the write
            const uint4 yk = make_uint4(yw[0], yw[1], yw[2], yw[3]);
            *own = yk;
            // the block's own token (exactly one block per fresh token and kv
            // head): its turned key also goes into the cache for later calls
            if (p >= rb.rmin) st16(const_cast<bf16_t*>(krow(p)) + c * 8, yk);
          }
        }
        // ... and its value, as it arrived
#pragma unroll
        for (int u = NC / WAVES; u < DPT; ++u) {
          const int slot = (wu + WAVES * u - NC) * 64 + lane;
          const int r = slot / NC, cpos = slot % NC;
          const int p = kb + r;
          if (p >= rb.rmin && p >= rb.f0 && p < kend) {
            const int c = cpos ^ Tile::swz_v(r);
            st16(const_cast<bf16_t*>(vown(p)) + c * 8, *reinterpret_cast<const uint4*>(&W.v[slot * 8]));
          }
        }
      }
    }
    // ... and every wave's; every wave is also done with the previous tile,
    // whose buffer the next load reuses
    lds_barrier();
    if (tile + kNBuf - 1 < ntiles) issue_to(tile + kNBuf - 1, tiles[(buf + kNBuf - 1) % kNBuf]);
    {
      const int kb = k0 + tile * kBN;
      // S^T = K Q^T: four 16-key tiles x two 16-row tiles
      floatx4 st[RT][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        uint4 ka[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const int r = kt * 16 + lr;
          ka[ks] = ld16(&T.k[(r * NC + ((ks * 4 + lq) ^ Tile::swz_k(r))) * 8]);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          floatx4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) c = mfma16x16x32(ka[ks], qf[rt][ks], c);
          st[rt][kt] = c;
        }
      }
      // causal / split-end mask, only on tiles that reach past the block's
      // first query position or the split's end (a block-uniform branch)
      if (kb + kBN > kend || kb + kBN - 1 > rb.rmin) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          // key kb + 16 kt + 4 lq + e is visible iff 16 kt + e <= lim.  The
          // empty asm keeps the compiler from hoisting this out of the loop,
          // which would wait for the metadata load before the first K/V load.
          int rp = rpos[rt];
          asm volatile("" : "+v"(rp));
          rp = 16 * (RT * w + rt) + lr < rows ? rp : -1;
          const int lim = min(rp, kend - 1) - kb - 4 * lq;
#pragma unroll
          for (int kt = 0; kt < 4; ++kt)
#pragma unroll
            for (int e = 0; e < 4; ++e) st[rt][kt][e] = (16 * kt + e <= lim) ? st[rt][kt][e] : -INFINITY;
        }
      }
      uint4 pb[RT][2];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        float tmax = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int e = 0; e < 4; ++e) tmax = fmaxf(tmax, st[rt][kt][e]);
        tmax = max_rows4(tmax);
        tmax *= qscale;  // scores are scaled inside the exponent below
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
            // v_exp_f32 of (s * scale - m): -inf gives 0
            pv[kt][e] = __builtin_amdgcn_exp2f(fmaf(st[rt][kt][e], qscale, -mref));
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
      // O^T += V^T P^T.  A fragment of step s, dims 16 dt ..: lane (lr, lq)
      // needs V[32 s + 4 lq + e][16 dt + lr] (e = 0..3) and the same 16 keys
      // later; in the transpose read, lane lr of group lq addresses row
      // 32 s + 4 lq + lr / 4 (+ 16), dims 16 dt + 4 (lr % 4) .. + 3.
      const int vr = 4 * lq + (lr >> 2);                 // row within a 32-key step
      const int vsw = Tile::swz_v(vr);                   // the same for rows vr + 16, + 32, + 48
      // fragment i = 2 dt + s; the next fragment's reads go out before the
      // current fragment's matrix ops, so that their latency is covered
      auto vfrag = [&](int i) -> uint4 {
        const int vc = (2 * (i >> 1) + ((lr & 3) >> 1)) ^ vsw;  // chunk position of dims 16 dt + 4 (lr % 4)
        const bf16_t* row = &T.v[((32 * (i & 1) + vr) * NC + vc) * 8 + (lr & 1) * 4];
        const uint2 lo = ld_tr8(row);
        const uint2 hi = ld_tr8(row + 16 * D);
        return make_uint4(lo.x, lo.y, hi.x, hi.y);
      };
      uint4 va = vfrag(0);
#pragma unroll
      for (int i = 0; i < 2 * DT; ++i) {
        const uint4 vn = i + 1 < 2 * DT ? vfrag(i + 1) : va;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[rt][i >> 1] = mfma16x16x32(va, pb[rt][i & 1], acc[rt][i >> 1]);
        va = vn;
      }
    }
  };
  // The loop is unrolled by the ring size, so each step's buffers are fixed and
  // every LDS address is a constant offset from a per-lane base (long-context
  // and 34B-shape prefill +4-7%).  The lambdas are forced inline: outlined, as
  // the compiler once chose for the paged instances, they kept a stack object
  // in scratch and those instances ran 6x slower.
  for (int t0 = 0; t0 < ntiles; t0 += kNBuf) {
    step(t0, std::integral_constant<int, 0>{});
    if (t0 + 1 >= ntiles) break;
    step(t0 + 1, std::integral_constant<int, 1>{});
    if constexpr (kNBuf == 4) {
      if (t0 + 2 >= ntiles) break;
      step(t0 + 2, std::integral_constant<int, 2 % kNBuf>{});
      if (t0 + 3 >= ntiles) break;
      step(t0 + 3, std::integral_constant<int, 3 % kNBuf>{});
    }
  }

  // epilogue: lane holds O^T[d = 16 dt + 4 lq + e][row lr] of each row tile
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const float l = sum_rows4(lsum[rt]);
    const int r = 16 * (RT * w + rt) + lr;
    if (r >= rows) continue;
    if (part < 0) {
      const float inv = l > 0.f ? 1.f / l : 0.f;
      bf16_t* o = out + ((int64_t)rtok[rt] * Hq + hk * g + r % g) * D + lq * 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const floatx4 a = acc[rt][dt];
        *reinterpret_cast<uint2*>(o + dt * 16) =
            make_uint2(cvt_bf16x2(a[0] * inv, a[1] * inv), cvt_bf16x2(a[2] * inv, a[3] * inv));
      }
    } else {
      // partial outputs in bf16 (the merge weights them in fp32; they end in
      // bf16), stored in accumulator order: per 16-row and 16-dim tile the 64
      // lanes' 4 values, so every store covers 512 contiguous bytes; streaming
      // stores, read once by the merge kernel
      const int64_t pr = ((int64_t)part * Hkv + hk) * part_stride_rows + r;
      bf16_t* o = reinterpret_cast<bf16_t*>(part_o) + ((int64_t)part * Hkv + hk) * part_stride_rows * D +
                  ((int64_t)(RT * w + rt) * DT * 64 + lane) * 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const floatx4 a = acc[rt][dt];
        st8_nt(o + dt * 256, cvt_bf16x2(a[0], a[1]), cvt_bf16x2(a[2], a[3]));
      }
      if (lq == 0) {
        part_ml[pr * 2 + 0] = mrow[rt];
        part_ml[pr * 2 + 1] = l;
      }
    }
  }
}

int launch_attn_mfma(const PrefillArgs& args, const TokenMeta* meta, const void* qws, int rows_ws,
                     const CacheView& cv, int layer, int Hq, void* out, float* part_o, float* part_ml,
                     int part_stride_rows, int nbuf, hipStream_t s, KTime tm, FusedIn fin, int wave_rows) {
  if (args.n_rb == 0 || args.n_split == 0) return 0;
  const int groups = args.n_split * cv.n_kv_heads;  // (split, kv head) pairs
  const dim3 grid = args.xcd_group ? dim3(kXcds * args.n_rb, (groups + kXcds - 1) / kXcds)
                                   : dim3(args.n_rb, args.n_split, cv.n_kv_heads);
  if (wave_rows != 16 && wave_rows != 32) return (int)hipErrorInvalidValue;
  const int waves = part_stride_rows / wave_rows;  // rows per block / rows per wave
  // instances: 128-row blocks of 4 waves (two-tile ring: two per CU; four-tile
  // ring: one per CU), 128-row blocks of 8 waves x 16 rows (two-tile ring, one
  // per CU), 256-row blocks of 8 waves (four-tile ring)
  const bool ok = wave_rows == 32 ? (waves == 4 && (nbuf == 2 || nbuf == 4)) || (waves == 8 && nbuf == 4)
                                  : waves == 8 && nbuf == 2;
  if (!ok) return (int)hipErrorInvalidValue;
  const bool fused = fin.q != nullptr;
#define PF(DD, PG, WV, NB, FU, RR)                                                                            \
  hipExtLaunchKernelGGL((attn_prefill_mfma_kernel<DD, PG, WV, NB, FU, RR>), grid, dim3(WV * 64), 0, s,         \
                        tm.start, tm.stop, 0, args, meta, (const bf16_t*)qws, rows_ws, cv, layer, Hq,           \
                        (bf16_t*)out, part_o, part_ml, part_stride_rows, (const bf16_t*)fin.q,                  \
                        (const bf16_t*)fin.k, (const bf16_t*)fin.v, fin.rope)
#define PFS(DD, PG, FU)                                                                                       \
  {                                                                                                           \
    if (wave_rows == 16) PF(DD, PG, 8, 2, FU, 1);                                                             \
    else if (nbuf == 2) PF(DD, PG, 4, 2, FU, 2);                                                              \
    else if (waves == 8) PF(DD, PG, 8, 4, FU, 2);                                                             \
    else PF(DD, PG, 4, 4, FU, 2);                                                                             \
  }
#define PFW(DD, PG) { if (fused) PFS(DD, PG, true) else PFS(DD, PG, false) }
  const bool paged = cv.page_size != 0;
  if (cv.head_dim == 128) { if (paged) PFW(128, true) else PFW(128, false) }
  else { if (paged) PFW(64, true) else PFW(64, false) }
#undef PFW
#undef PFS
#undef PF
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // namespace fcg
