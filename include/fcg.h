/*
 * fcg.h - function-level KV cache grafting on one MI355X (gfx950).
 *
 * C ABI of libfcg.so.  The library holds a segment library of function-level
 * KV states (the two-tier code cache of Sec. 4.1, Eq. 2: every function entry
 * keeps the KV states of its interface and of its implementation), stitches
 * retrieved segments into a composite cache at new positions (cache-stitching,
 * Sec. 4.2, Eq. 4: the interface KV states are concatenated and injected as
 * context), prefills patch tokens over that cache and decodes (cache-patching,
 * Sec. 4.2, Eq. 6: the prefix KV states are reused and only the new span is
 * computed).  Text, tokenizer and model weights are outside this library; its
 * inputs are token-level K/V/Q tensors.
 *
 * Conventions
 *  - Every entry point returns an fcg_status; nothing aborts or throws across
 *    the ABI.  fcg_last_error() gives a thread-local message for the last
 *    failing call on the calling thread.
 *  - A call that returns an error changes no state (an EHIP failure of the
 *    runtime after a call's checks aside).
 *  - "device" pointers are HIP device memory on the current device; "host"
 *    pointers are ordinary host memory, read (or written) before the call
 *    returns.  The caller keeps ownership of everything it passes.
 *  - stream is a hipStream_t (NULL = the default stream).  Calls validate on
 *    the host, enqueue their kernels on the stream and return; results are
 *    ready when the stream reaches that point.  A handle (fcg_lib, fcg_cache)
 *    must not be used by two threads or two streams at the same time.
 *  - Device faults of earlier work surface as FCG_EHIP from a later call.
 *  - Storage dtype: FCG_F32 = IEEE binary32, FCG_BF16 = bfloat16 (raw 16-bit
 *    patterns).  Every narrowing rounds to nearest, ties to even.
 *
 * Tensor layouts (elements of the storage dtype, row-major, innermost last)
 *  - Segment input to fcg_lib_add_segment:   k, v  [L][len][Hkv][D]
 *  - Library slab of one layer:              [Hkv][capacity][D]
 *  - Contiguous cache, one layer:            [n_seqs][Hkv][max_tokens][D]
 *  - Paged cache, one layer:                 [n_pages][Hkv][page_size][D]
 *  - Fresh tokens of fcg_patch_prefill:      q [n][Hq][D], k, v [n][Hkv][D]
 *  - Decode tokens of fcg_decode:            q [n][Hq][D], k, v [n][Hkv][D]
 *  - Attention outputs:                      out [n][Hq][D]
 */
#ifndef FCG_H
#define FCG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FCG_OK = 0,
  FCG_EINVAL = 1,   /* malformed argument: null pointer, bad count, unsupported shape, mismatch */
  FCG_ERANGE = 2,   /* index out of range: layer, sequence, segment, position, span end */
  FCG_EOVERLAP = 3, /* a target position is given twice or is already written */
  FCG_EHOLE = 4,    /* attention would read a position that is not written */
  FCG_ENOMEM = 5,   /* device memory, library capacity, host tier or page pool exhausted */
  FCG_ESTATE = 6,   /* operation not valid in the current state (e.g. decode on an empty sequence) */
  FCG_EHIP = 7      /* the HIP runtime reported an error */
} fcg_status;

typedef enum { FCG_F32 = 0, FCG_BF16 = 1 } fcg_dtype;

/* Shape of the attention layers whose KV states are grafted.  Keys carry the
 * rotary position encoding in rotate-half layout: dimension i and i + D/2 turn
 * together by p * theta^(-2i/D) at position p (rope_style 0, the only one). */
typedef struct {
  int32_t n_layers;   /* L >= 1 */
  int32_t n_q_heads;  /* Hq, with Hq / Hkv one of 1, 2, 4, 8, 16 */
  int32_t n_kv_heads; /* Hkv >= 1 */
  int32_t head_dim;   /* D: 64 or 128 */
  double rope_theta;  /* theta > 1 */
  int32_t dtype;      /* fcg_dtype of every K, V, Q and output tensor */
  int32_t rope_style; /* 0 = rotate-half */
} fcg_model_desc;

typedef struct fcg_lib fcg_lib;
typedef struct fcg_cache fcg_cache;
typedef struct fcg_locality fcg_locality;

/* ---------------------------------------------------------------- library */

/* flags of fcg_lib_create and fcg_cache_create */
#define FCG_LAYOUT_ONLY 1u /* no device memory: only the index / layout is kept (planning and tests) */
/* fcg_cache_create, paged caches only: a logical page that one grafted
 * segment covers entirely reads its values from the library in place instead
 * of a copy (values are position-independent; keys are still turned and
 * copied).  The cache binds to the library of its first graft; the library
 * must outlive the cache. */
#define FCG_ALIAS_V 2u

/* Create an empty segment library (the KV side of the two-tier code cache,
 * Sec. 4.1, Eq. 2) holding up to capacity_tokens tokens in up to max_segments
 * segments.  Allocates L * Hkv * capacity_tokens * D elements for K and as
 * many for V (none with FCG_LAYOUT_ONLY: then only the segment index exists,
 * segments are added with k == v == NULL, and grafts into layout-only caches
 * are planned but move nothing).  FCG_ENOMEM if the device cannot hold them. */
fcg_status fcg_lib_create(const fcg_model_desc* desc, int64_t capacity_tokens,
                          int32_t max_segments, uint32_t flags, fcg_lib** out);

/* Append one segment of len tokens whose keys were encoded at source positions
 * src_pos0 .. src_pos0 + len - 1.  k, v: device [L][len][Hkv][D], copied into
 * the slabs on stream.  k == v == NULL reserves the space only (the caller
 * fills it through fcg_lib_device_ptrs).  *seg_id receives the new id
 * (ids are 0, 1, 2, ... in order of addition).  FCG_ENOMEM when capacity or
 * max_segments is exhausted. */
fcg_status fcg_lib_add_segment(fcg_lib* lib, int32_t len, int32_t src_pos0, const void* k,
                               const void* v, void* stream, int32_t* seg_id);

/* The update step of the cache management (Alg. 1; Sec. 4.1: low-scored
 * entries go to DRAM, high-scored ones stay on the GPU): with loc tracking one
 * function per library segment (function id = segment id), decide which
 * segments stay in device memory and move the others: segments read in place
 * by an FCG_ALIAS_V cache stay; then, in descending locality score (Eq. 3),
 * a segment stays while its bytes (len x K+V of all layers) fit in
 * budget_bytes; with ppl_threshold > 0 (the hyperparameter table's
 * perplexity-based eviction threshold, 15.0) segments whose perplexity is
 * below it are placed only after all others.  budget_bytes < 0 takes the
 * table's GPU memory threshold: 0.85 of the device memory less a 2 GB reserve
 * less what the rest of the process holds (at most the slabs).  Offloads are
 * issued first, then reloads, all on stream (a side stream is fine: grafts
 * wait for reloads, and reused ranges wait for earlier grafts).
 * *n_offloaded / *n_reloaded (host, may be NULL) receive the moves.
 * Errors: EINVAL (null arguments, loc's size differs from the segment count,
 * negative threshold), ESTATE (an offload without a host tier), ENOMEM (host
 * tier full, or no device range for a reload: the state stays consistent, the
 * moves made so far remain). */
fcg_status fcg_lib_update_residency(fcg_lib* lib, const fcg_locality* loc, int64_t budget_bytes,
                                    double ppl_threshold, void* stream, int32_t* n_offloaded,
                                    int32_t* n_reloaded);

/* Where segment seg_id sits: tokens tok_off .. tok_off + len - 1 of every
 * [Hkv][capacity][D] slab (tok_off = -1 while offloaded); keys encoded from
 * src_pos0.  Any output may be NULL. */
fcg_status fcg_lib_segment_info(const fcg_lib* lib, int32_t seg_id, int64_t* tok_off,
                                int32_t* len, int32_t* src_pos0);

/* Host tier of the library (the DRAM side of the code cache: low-scored
 * entries are offloaded and reloaded when needed; Sec. 4.1, App. C.5).
 * fcg_lib_host_reserve allocates pinned host slabs of host_tokens tokens
 * (layout as the device slabs); each segment gets a host copy on its first
 * offload, kept until the library is destroyed (segments never change).
 * Errors: EINVAL (host_tokens < 1), ESTATE (reserved already), ENOMEM, EHIP. */
fcg_status fcg_lib_host_reserve(fcg_lib* lib, int64_t host_tokens);

/* Move segment seg_id out of device memory: copy it to its host slot on
 * stream (first offload only) and free its device range for later segments
 * and reloads (first fit; a reused range is written only after the copy has
 * read it).  fcg_graft of an offloaded segment fails with ESTATE.  Async:
 * calls on one library are ordered by the caller (one stream, or events).
 * Errors: ERANGE (seg_id), ESTATE (not in device memory, no host tier, or an
 * FCG_ALIAS_V cache reads its values in place: reset those sequences first),
 * ENOMEM (host tier full), EHIP. */
fcg_status fcg_lib_offload(fcg_lib* lib, int32_t seg_id, void* stream);

/* Bring an offloaded segment back into device memory on stream, at the first
 * free device range that fits (fcg_lib_segment_info gives the new offset).
 * Errors: ERANGE, ESTATE (already in device memory), ENOMEM (no range fits), EHIP. */
fcg_status fcg_lib_reload(fcg_lib* lib, int32_t seg_id, void* stream);

/* *in_device = 1 iff seg_id is in device memory; *on_host = 1 iff it has a host
 * copy (either may be NULL).  Errors: EINVAL, ERANGE. */
fcg_status fcg_lib_segment_state(const fcg_lib* lib, int32_t seg_id, int32_t* in_device, int32_t* on_host);

/* Device base pointers of layer's K and V slab ([Hkv][capacity][D]). */
fcg_status fcg_lib_device_ptrs(const fcg_lib* lib, int32_t layer, void** k, void** v);

fcg_status fcg_lib_destroy(fcg_lib* lib);

/* ------------------------------------------------------------------ cache */

/* Create a composite cache for n_seqs sequences of up to max_tokens positions.
 * page_size == 0: contiguous, one [Hkv][max_tokens][D] region per sequence and
 * layer (n_pages ignored).  page_size == 16: a pool of n_pages pages per
 * layer, one page table per sequence shared by all layers; logical page
 * p / 16 of a sequence is mapped on first write to the lowest-numbered free
 * page, new pages of one call in ascending (sequence, logical page) order.
 * With FCG_LAYOUT_ONLY no device memory is allocated and graft, prefill
 * and decode only validate and record the layout (planning and tests);
 * FCG_ALIAS_V maps value pages onto the library (see the flag).
 * Errors: EINVAL (bad descriptor, n_seqs or max_tokens < 1, max_tokens *
 * head_dim >= 2^31, page_size not 0 or 16, unknown flags, FCG_ALIAS_V on a
 * contiguous cache), ENOMEM, EHIP. */
fcg_status fcg_cache_create(const fcg_model_desc* desc, int32_t n_seqs, int32_t max_tokens,
                            int32_t page_size, int32_t n_pages, uint32_t flags, fcg_cache** out);

/* Forget everything written in seq (all layers) and return its pages. */
fcg_status fcg_cache_reset(fcg_cache* cache, int32_t seq);

/* Cache-patching (Sec. 4.2, Eq. 6; the patch step of Alg. 1): keep only the
 * prefix [0, pos) of seq in every layer, so that the span after it can be
 * regenerated over the reused prefix states (fcg_patch_prefill of new tokens
 * at positions pos.., then fcg_decode).  The stale states past pos are never
 * read.  Pages holding no kept position return to the pool.  Host metadata
 * only, except with FCG_ALIAS_V when the cut splits a page whose values are
 * read from the library: its kept rows are copied into the cache's own page
 * on stream (new tokens will follow them).  pos = 0 empties the sequence;
 * pos = max_tokens keeps everything.  Errors: EINVAL (null cache), ERANGE
 * (seq outside [0, n_seqs), pos outside [0, max_tokens]), EHIP. */
fcg_status fcg_cache_truncate(fcg_cache* cache, int32_t seq, int32_t pos, void* stream);

/* Host copy of the layout of seq: page_table [ceil(max_tokens / page_size)]
 * physical page or -1 (paged caches only; may be NULL), *seq_len = 1 + the
 * highest written position of layer (0 if none; may be NULL), written
 * [max_tokens] bytes 1/0 per position of layer (may be NULL). */
fcg_status fcg_cache_export_layout(const fcg_cache* cache, int32_t seq, int32_t layer,
                                   int32_t* page_table, int32_t* seq_len, uint8_t* written);

/* FCG_ALIAS_V caches: v_alias [ceil(max_tokens / 16)] receives, per logical
 * page of seq, the library token (index into the [Hkv][capacity][D] slabs)
 * whose value row holds the page's first position, or -1 where the page holds
 * its own values.  -1 everywhere for other caches.  Errors: EINVAL (null
 * argument), ERANGE (seq). */
fcg_status fcg_cache_export_v_alias(const fcg_cache* cache, int32_t seq, int32_t* v_alias);

/* Device base pointers of layer's K and V region (layouts in the file header). */
fcg_status fcg_cache_device_ptrs(const fcg_cache* cache, int32_t layer, void** k, void** v);

fcg_status fcg_cache_destroy(fcg_cache* cache);

/* --------------------------------------------------------------- hot path */

/* Cache-stitching (Sec. 4.2, Eq. 4; App. B.1, module-level cache reuse):
 * for every item i, graft library segment seg[i] into sequence seq[i] at
 * positions dst[i] .. dst[i] + len - 1, in all layers, keeping its token
 * order.  Keys are turned by delta = dst[i] - src_pos0 (the rotary encoding of
 * a key at position p becomes that of p + delta) and rounded to the storage
 * dtype; values are copied bit for bit.  One launch covers every item and
 * layer.  seq, seg, dst: host arrays of n_items.
 * Errors: ERANGE (seq, seg, span outside [0, max_tokens)), EOVERLAP (spans
 * meet each other or written positions of any layer), ENOMEM (pages), EINVAL
 * (lib and cache shapes differ, null arrays, a layout-only library with a
 * cache that has device memory, an FCG_ALIAS_V cache bound to another
 * library), ESTATE (after all of the above pass: a segment is offloaded). */
fcg_status fcg_graft(fcg_cache* cache, const fcg_lib* lib, int32_t n_items, const int32_t* seq,
                     const int32_t* seg, const int32_t* dst, void* stream);

/* Patch prefill at one layer (Sec. 4.2, Eq. 6; App. B.1, cache-patching):
 * token t (host seq[t], pos[t]) gets its query and key encoded at pos[t]
 * (rounded to storage), its key and value stored at pos[t], and
 * out[t] = softmax(q k^T / sqrt(D)) v over every position <= pos[t] of its
 * sequence, query head h reading kv head h / (Hq / Hkv).  Tokens may belong to
 * several sequences and come in any order.  q, k, v, out: device.
 * Errors: ERANGE, EOVERLAP (position given twice or already written in this
 * layer), EHOLE (a position below a query's is unwritten after the call),
 * ENOMEM (pages). */
fcg_status fcg_patch_prefill(fcg_cache* cache, int32_t layer, int32_t n_tok, const int32_t* seq,
                             const int32_t* pos, const void* q, const void* k, const void* v,
                             void* out, void* stream);

/* One decode step at one layer for n_seqs distinct sequences (host seqs):
 * each appends its token at its current length in that layer and attends
 * over every position up to it, as in fcg_patch_prefill.  positions_out
 * (host, may be NULL) receives the positions used.
 * Errors: EINVAL (duplicate sequence), ERANGE (sequence full), ESTATE
 * (nothing written in this layer), EHOLE, ENOMEM. */
fcg_status fcg_decode(fcg_cache* cache, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                      const void* q, const void* k, const void* v, void* out,
                      int32_t* positions_out, void* stream);

/* fcg_decode for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, semantics, results and errors as fcg_decode; it calls no
 * hipMalloc / hipFree and uploads nothing.  Its split partials and arrival
 * counters live in a static device array of the library (8.5 MiB per GPU,
 * held until the process ends), not in memory of the cache; the cache itself
 * must exist already (fcg_cache_create allocates).  Every call on one GPU
 * shares that array: calls that overlap on one GPU (several streams or host
 * threads) race.  The first call on a device also launches a small kernel that
 * zeroes the counters.  Kernel timing (fcg_cache_timing) does not cover it.
 * Extra errors: EINVAL (more than 64 kv heads), ENOMEM (the step needs more
 * than 8 MiB of split partials: many long sequences at once; use fcg_decode). */
fcg_status fcg_decode_noalloc(fcg_cache* cache, int32_t layer, int32_t n_seqs, const int32_t* seqs,
                              const void* q, const void* k, const void* v, void* out,
                              int32_t* positions_out, void* stream);

/* ------------------------------------------------- code-cache management */

/* Locality score of the cache entries (Sec. 4.1, Eq. 3; App. B.1, Eq. 8-10;
 * the update step of Alg. 1), host only:
 *   l(f) = (1 - l_curr(f)) (alpha l_freq(f) + beta sum_j l_asso(j | f)
 *          + gamma l_sema(f)) + l_curr(f),
 *   l_freq(f) = count(f) / max_j count(j),
 *   l_asso(j | f) = cooccur(f, j) / count(f),
 *   l_sema(f) = PPL(f) / max_j PPL(j).
 * Functions are ids 0 .. n_funcs - 1 (a caller's map to library segments).
 * Statistics cover the last `window` recorded execution traces (one per task;
 * the paper uses 20); cooccur(f, j) counts calls of j that immediately follow
 * a call of f in one trace; l_curr(f) = 1 iff f occurs in the latest trace;
 * a component with a zero denominator is 0.  Weights: >= 0, summing to 1 (the
 * paper uses 0.4, 0.3, 0.3).
 * Errors: EINVAL (n_funcs or window < 1, bad weights, null output), ENOMEM. */
fcg_status fcg_locality_create(int32_t n_funcs, int32_t window, double alpha, double beta, double gamma,
                               fcg_locality** out);
/* Record one task's execution trace: func_ids[n] (host) in call order.
 * Errors: EINVAL (null handle, n < 0, null ids), ERANGE (an id). */
fcg_status fcg_locality_record(fcg_locality* loc, int32_t n, const int32_t* func_ids);
/* Perplexity of function func's implementation (>= 0; 0 until set).
 * Errors: EINVAL (null handle, negative or NaN ppl), ERANGE (func). */
fcg_status fcg_locality_set_ppl(fcg_locality* loc, int32_t func, double ppl);
/* scores[n_funcs] (host) receives l(f), each in [0, 1].  Errors: EINVAL. */
fcg_status fcg_locality_scores(const fcg_locality* loc, double* scores);
/* Which entries stay in device memory under a budget: in descending score
 * (ties: ascending id), an entry is kept when its cost[f] (host, >= 0, e.g.
 * bytes or tokens) still fits in what the kept ones leave of budget.
 * resident[n_funcs] (host) receives 1 / 0.  Errors: EINVAL (null arguments,
 * negative budget or cost). */
fcg_status fcg_locality_residency(const fcg_locality* loc, int64_t budget, const int64_t* cost, uint8_t* resident);
fcg_status fcg_locality_destroy(fcg_locality* loc);

/* ------------------------------------------------------------- diagnostics */

/* Kernel timing (measurement, not part of the method).  While enabled, every
 * call on this cache records HIP events on its stream around its kernels:
 *   FCG_TIME_GRAFT        the graft kernel of fcg_graft
 *   FCG_TIME_PREFILL_ATTN the attention kernel of fcg_patch_prefill
 *   FCG_TIME_PREFILL      all kernels of fcg_patch_prefill (append, attention, merge)
 *   FCG_TIME_DECODE       all kernels of fcg_decode (one per group of 64 sequences)
 *   FCG_TIME_DECODE_ATTN  the attention kernels of fcg_decode (the same kernels: the
 *                         split merge runs inside them)
 * Plan uploads and host work are outside the intervals.  fcg_cache_timing_read
 * waits for the recorded events, returns the number of intervals and their
 * summed duration in milliseconds for one kind (ERANGE for another value),
 * and forgets them.  enable = 0 stops recording (recorded intervals stay
 * readable). */
#define FCG_TIME_GRAFT 0
#define FCG_TIME_PREFILL_ATTN 1
#define FCG_TIME_PREFILL 2
#define FCG_TIME_DECODE 3
#define FCG_TIME_DECODE_ATTN 4
fcg_status fcg_cache_timing(fcg_cache* cache, int32_t enable);
fcg_status fcg_cache_timing_read(fcg_cache* cache, int32_t kind, int32_t* count, double* total_ms);

/* Name of a status code; the message of the calling thread's last failed
 * call (kept until its next failure; empty before any).  Both strings are
 * owned by the library. */
const char* fcg_status_string(fcg_status s);
const char* fcg_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FCG_H */
