// Launch interface between the host side of libfcg (api.cpp) and its gfx950
// kernels.  Plain structs and pointers only.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fcg {

// Optional events attached to a kernel's dispatch (hipExtLaunchKernelGGL):
// they take the kernel's own start and end times, with no extra stream work.
struct KTime {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// One run of up to kGraftChunk tokens of one grafted segment.
struct GraftChunk {
  int64_t src_tok;  // token index in the library slab of the first token
  int32_t dst;      // target position of the first token
  int32_t seq;      // target sequence
  int32_t delta;    // rotary turn of the keys (dst - src_pos0 of the segment)
  int32_t n;        // tokens in this run
  int32_t seg_lo, seg_hi;  // the whole segment's positions [seg_lo, seg_hi)
};
constexpr int kGraftChunk = 64;

// Device view of a composite cache (all layers).
struct CacheView {
  void* k;               // layer-0 base of K
  void* v;               // layer-0 base of V
  int64_t layer_stride;  // elements from one layer's region to the next
  // paged only: per sequence a row of 2 n_lp entries, the physical page of
  // each logical page, then (value aliasing) the library token of its first
  // position or -1
  const int32_t* page_table;
  const int32_t* v_alias;  // page_table + n_lp when values may be aliased, else null
  const void* lib_v;       // the aliased library's V slabs [L][Hkv][lib_cap][D]
  int64_t lib_cap;
  int32_t n_seqs, max_tokens, page_size, n_lp;
  int32_t n_kv_heads, head_dim;
};

// Offset (elements) of (layer, seq, head, pos) inside a cache; page_size is 0
// (contiguous) or a power of two.
__host__ __device__ inline int64_t cache_offset(const CacheView& c, int layer, int seq, int head, int pos) {
  int64_t base = (int64_t)layer * c.layer_stride;
  if (c.page_size == 0)
    return base + (((int64_t)seq * c.n_kv_heads + head) * c.max_tokens + pos) * c.head_dim;
  int32_t page = c.page_table[(int64_t)seq * 2 * c.n_lp + pos / c.page_size];
  return base + (((int64_t)page * c.n_kv_heads + head) * c.page_size + (pos % c.page_size)) * c.head_dim;
}

// Element offset of (layer, seq, head, pos) with the layout known at compile time.
template <bool PAGED>
__device__ __forceinline__ int64_t kv_offset(const CacheView& c, int layer, int seq, int head, int pos) {
  if (PAGED) {
    const int32_t page = c.page_table[(int64_t)seq * 2 * c.n_lp + (pos >> 4)];
    return (int64_t)layer * c.layer_stride + (((int64_t)page * c.n_kv_heads + head) * 16 + (pos & 15)) * c.head_dim;
  }
  return (int64_t)layer * c.layer_stride + (((int64_t)seq * c.n_kv_heads + head) * c.max_tokens + pos) * c.head_dim;
}

// Pages of a paged cache whose entries a block stages in LDS (the page window
// of its key range); a longer range reads the entries from memory.
constexpr int kPageWindow = 520;

// Value row (layer, seq, head, pos) to read: the cache's own row, or the
// library's row for a page whose values are mapped onto the library.
template <bool PAGED, typename T>
__device__ __forceinline__ const T* v_row(const CacheView& c, int layer, int seq, int head, int pos) {
  if (PAGED && c.v_alias) {
    const int32_t a = c.v_alias[(int64_t)seq * 2 * c.n_lp + (pos >> 4)];
    if (a >= 0)
      return reinterpret_cast<const T*>(c.lib_v) +
             (((int64_t)layer * c.n_kv_heads + head) * c.lib_cap + a + (pos & 15)) * c.head_dim;
  }
  return reinterpret_cast<const T*>(c.v) + kv_offset<PAGED>(c, layer, seq, head, pos);
}

// Per fresh (or decode) token, in attention order: tokens grouped by sequence,
// ascending position inside a sequence.  Query rows of kv head h for the token
// of rank r are r * g .. r * g + g - 1 of the query workspace.
struct TokenMeta {
  int32_t tok;  // index of the token in the caller's q/k/v/out arrays
  int32_t seq;
  int32_t pos;
  int32_t pad;
};

// A block of consecutive ranks (one sequence) attended over keys [k0, k1).
struct AttnItem {
  int32_t rank0, n_rank;  // token ranks of the row block
  int32_t seq;
  int32_t k0, k1;         // key positions of this split
  int32_t part;           // partial-result slot (-1: the only split, write the output directly)
  int32_t pad0, pad1;
};

// Row block -> its partial slots, for the split-KV combine.
struct CombineItem {
  int32_t rank0, n_rank;
  int32_t part0, n_part;  // partial slots part0 .. part0 + n_part - 1
  int32_t tok0;           // >= 0: the caller's index of rank0's token, the rest consecutive; -1: from meta
};
// By-value plan of one combine launch.
constexpr int kCombMaxItems = 128;
struct CombineArgs {
  int32_t n_items, pad0, pad1, pad2;
  CombineItem item[kCombMaxItems];
};

// By-value arguments of one fused decode launch (up to kMaxDecodeSeqs sequences).
constexpr int kMaxDecodeSeqs = 64;
struct DecodeArgs {
  int32_t n;           // sequences in this launch
  int32_t split_keys;  // key positions per split
  int32_t max_split;   // largest split count of the launch (grid x)
  int32_t slots;       // partial slots of the launch, split0[n] (a field of its own, at a fixed offset)
  int32_t seq[kMaxDecodeSeqs];
  int32_t pos[kMaxDecodeSeqs];         // the new token's position (= the sequence's length)
  int32_t split0[kMaxDecodeSeqs + 1];  // first partial slot of each sequence; split0[i + 1] - split0[i] splits
  // paged caches: the physical page this step maps for the new token's logical
  // page (its first position is the new token), or -1 when the page is mapped
  // already.  The kernel stores the new token there and enters the page (and
  // "values not read from the library") into the device page table.
  int32_t new_page[kMaxDecodeSeqs];
};

// Rotary table of a cache: for position p and pair i, (cos, sin) of the float64
// angle p * theta^(-2i/D), each rounded to fp32 -- the values every kernel that
// encodes a fresh or decoded token at p uses.  [n_pos][D/2] float2.
int launch_rope_table(const double* inv_freq, int half, int n_pos, float2* tab, hipStream_t s);

int launch_lib_ingest(int dtype, const void* k, const void* v, void* lib_k, void* lib_v, int L, int len,
                      int Hkv, int D, int64_t cap, int64_t tok_off, hipStream_t s);

int launch_graft(int dtype, const GraftChunk* chunks, int n_chunks, const void* lib_k, const void* lib_v,
                 int64_t cap, const CacheView& cv, const double* inv_freq, int L, hipStream_t s, KTime tm = {});

// A value page mapped onto the library that a truncation split: its first
// `rows` rows are copied from library token lib_tok .. into physical page `page`.
struct UnaliasItem {
  int64_t lib_tok;
  int32_t page, rows;
};
int launch_unalias(int dtype, const UnaliasItem* items, int n_items, const void* lib_v, int64_t cap,
                   const CacheView& cv, int L, hipStream_t s);

// Encode q and k of n tokens at their positions, store k and v in the cache
// (layer), write encoded q to qws [Hkv][n * g][D].
int launch_rope_append(int dtype, const TokenMeta* meta, int n, const void* q, const void* k, const void* v,
                       const CacheView& cv, int layer, const float2* rope, int Hq, void* qws,
                       hipStream_t s, KTime tm = {});

// By-value work list of one MFMA prefill launch: row blocks (up to 256 query
// rows of one sequence), each attended over n_split key splits of `span`
// positions (splits past a row block's last position are empty).  The grid is
// (row block, split, kv head), so a block finds its work without a memory
// round trip.
constexpr int kPfMaxRb = 96;
struct PrefillRb {
  int32_t rank0, n_rank, seq;
  int32_t rmin, pmax;  // smallest and largest query position of the block
  int32_t part0;       // first partial slot, -1 when the block has a single split
  // fused launches (fresh tokens encoded and appended by the attention kernel):
  // the sequence's first fresh position of the call and the caller's index of
  // that token.  Every position p >= f0 of the sequence up to its last query
  // is fresh, at caller index ftok0 + (p - f0); the block's own tokens are the
  // positions rmin .. pmax.
  int32_t f0, ftok0;
};
struct PrefillArgs {
  int32_t n_rb, n_split, span;
  int32_t xcd_group;  // 1: row blocks of one (split, kv head) on one XCD (see the kernel)
  PrefillRb rb[kPfMaxRb];
};

// bf16 MFMA attention of query-workspace rows over the cache.  Blocks of
// part_stride_rows / wave_rows waves (wave_rows 32, or 16: 128-row blocks of 8
// waves, two per SIMD, for blocks planned one per CU); nbuf: tiles of the LDS
// ring, 2 for 128-row blocks planned two per CU or of 16-row waves, else 4.
// Fused launches take the caller's fresh q [n][Hq][D], k, v [n][Hkv][D] and the
// cache's rotary table instead of the query workspace: queries are encoded in
// the kernel's prologue, fresh keys and values are read from the inputs (keys
// turned in LDS), and the block owning a fresh token stores its key and value
// into the cache.  q == nullptr: the workspace path (rope_append ran before).
struct FusedIn {
  const void* q = nullptr;
  const void* k = nullptr;
  const void* v = nullptr;
  const float2* rope = nullptr;
};
int launch_attn_mfma(const PrefillArgs& args, const TokenMeta* meta, const void* qws, int rows_ws,
                     const CacheView& cv, int layer, int Hq, void* out, float* part_o, float* part_ml,
                     int part_stride_rows, int nbuf, hipStream_t s, KTime tm = {}, FusedIn fin = {},
                     int wave_rows = 32);

// VALU attention, one token (g query rows) per item; any dtype.
int launch_attn_rows(int dtype, const AttnItem* items, int n_items, const TokenMeta* meta, const void* qws,
                     int rows_ws, const CacheView& cv, int layer, int Hq, void* out, float* part_o,
                     float* part_ml, int part_stride_rows, hipStream_t s, KTime tm = {});

// Decode step: encode + store the new token and split-KV attention over the
// cache.  q, k, v, out: [n][H][D] rows in the order of args.seq.  Grid
// (max_split, n, Hkv).  Splits of multi-split sequences leave partials in
// part_o [slot][Hkv][g][D] and part_ml [slot][Hkv][g][2], slot = split0[i] +
// split; the last block of each (sequence, kv head) to finish merges them.
// count: [kMaxDecodeSeqs][Hkv] arrival counters kCountStride ints apart (one
// per 128-byte line: atomics on one line serialise), zero before the launch
// and zero again after it.
constexpr int kCountStride = 32;
int launch_decode(int dtype, const DecodeArgs& args, const void* q, const void* k, const void* v, const CacheView& cv,
                  int layer, const float2* rope, int Hq, void* out, float* part_o, float* part_ml, int* count,
                  hipStream_t s, KTime tm = {});

// The same step on matrix cores for bf16 caches and query groups of up to 16
// heads (same arguments; -1 for a group size it has no instance for).
int launch_decode_mfma(const DecodeArgs& args, const void* q, const void* k, const void* v, const CacheView& cv,
                       int layer, const float2* rope, int Hq, void* out, float* part_o, float* part_ml,
                       int* count, hipStream_t s, KTime tm = {});

// Static scratch of the allocation-free decode entry point (noalloc.hip):
// arrival counters for kMaxDecodeSeqs sequences x kNoAllocMaxKvHeads kv heads,
// then the split partials.  noalloc_scratch returns its device address on the
// current device (taken, and the counters zeroed on stream s, at the first call
// on that device).
constexpr int kNoAllocMaxKvHeads = 64;
constexpr size_t kNoAllocCountBytes = (size_t)kMaxDecodeSeqs * kNoAllocMaxKvHeads * kCountStride * sizeof(int32_t);
constexpr size_t kNoAllocPartBytes = (size_t)8 << 20;
constexpr size_t kNoAllocScratchBytes = kNoAllocCountBytes + kNoAllocPartBytes;
int noalloc_scratch(hipStream_t s, void** base);

// Merge split partials into out: part_o fp32 rows, or (mfma_part) bf16 in the
// accumulator order of the MFMA prefill kernel.
int launch_combine(int dtype, const CombineArgs& args, const TokenMeta* meta, int Hq, int Hkv, int D,
                   const float* part_o, const float* part_ml, int part_stride_rows, void* out, hipStream_t s,
                   bool mfma_part = false, KTime tm = {});

}  // namespace fcg
