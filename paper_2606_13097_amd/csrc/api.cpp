// libfcg C ABI (include/fcg.h): argument checks, the segment library and the
// composite cache objects, the upload of per-call plans, and kernel dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <deque>
#include <map>
#include <new>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "errors.hpp"
#include "fcg.h"
#include "kernels.hpp"
#include "locality.hpp"
#include "planner.hpp"

using namespace fcg;

namespace {

thread_local std::string g_err;

fcg_status fail(fcg_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

}  // namespace

fcg_status fcg::report(fcg_status s, const std::string& msg) { return fail(s, msg); }

namespace {

fcg_status hip_fail(hipError_t e, const char* what) {
  return fail(FCG_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                          \
  do {                                               \
    hipError_t e_ = (expr);                          \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

size_t esize(int32_t dtype) { return dtype == FCG_F32 ? 4 : 2; }

fcg_status check_desc(const fcg_model_desc* d) {
  if (!d) return fail(FCG_EINVAL, "null model descriptor");
  if (d->n_layers < 1 || d->n_layers > 255) return fail(FCG_EINVAL, "n_layers must be in [1, 255]");
  if (d->n_kv_heads < 1 || d->n_q_heads < d->n_kv_heads || d->n_q_heads % d->n_kv_heads)
    return fail(FCG_EINVAL, "n_q_heads must be a positive multiple of n_kv_heads");
  int g = d->n_q_heads / d->n_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8 && g != 16) return fail(FCG_EINVAL, "group size must be 1, 2, 4, 8 or 16");
  if (d->head_dim != 64 && d->head_dim != 128) return fail(FCG_EINVAL, "head_dim must be 64 or 128");
  if (!(d->rope_theta > 1.0) || !std::isfinite(d->rope_theta)) return fail(FCG_EINVAL, "rope_theta must be > 1");
  if (d->dtype != FCG_F32 && d->dtype != FCG_BF16) return fail(FCG_EINVAL, "unknown dtype");
  if (d->rope_style != 0) return fail(FCG_EINVAL, "only rope_style 0 (rotate-half) is supported");
  return FCG_OK;
}

bool same_shape(const fcg_model_desc& a, const fcg_model_desc& b) {
  return a.n_layers == b.n_layers && a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim &&
         a.dtype == b.dtype && a.rope_theta == b.rope_theta && a.rope_style == b.rope_style;
}

// float64 rotary frequencies w_i = theta^(-2i/D)
fcg_status upload_inv_freq(const fcg_model_desc& d, double** out) {
  std::vector<double> w(d.head_dim / 2);
  for (int i = 0; i < d.head_dim / 2; ++i) w[i] = std::pow(d.rope_theta, -2.0 * i / d.head_dim);
  HIP_TRY(hipMalloc(out, w.size() * sizeof(double)), "hipMalloc(inv_freq)");
  HIP_TRY(hipMemcpy(*out, w.data(), w.size() * sizeof(double), hipMemcpyHostToDevice), "hipMemcpy(inv_freq)");
  return FCG_OK;
}

// Staging of per-call plans: a pinned host ring mirrored by a device ring.  A
// call packs its arrays into one blob, copies it host-to-device on the call's
// stream and records an event; a region is reused only after its event.
struct Ring {
  char* host = nullptr;
  char* dev = nullptr;
  size_t cap = 0, head = 0;
  std::deque<std::tuple<size_t, size_t, hipEvent_t>> inflight;
  std::vector<hipEvent_t> spare;

  ~Ring() { release(); }
  void release() {
    for (auto& f : inflight) {
      hipEventSynchronize(std::get<2>(f));
      hipEventDestroy(std::get<2>(f));
    }
    inflight.clear();
    for (auto e : spare) hipEventDestroy(e);
    spare.clear();
    if (host) hipHostFree(host);
    if (dev) hipFree(dev);
    host = dev = nullptr;
    cap = head = 0;
  }
  fcg_status reserve(size_t n) {
    if (n <= cap) return FCG_OK;
    size_t nc = std::max<size_t>(cap * 2, std::max<size_t>(n, 1 << 20));
    release();
    HIP_TRY(hipHostMalloc((void**)&host, nc, hipHostMallocDefault), "hipHostMalloc(staging)");
    HIP_TRY(hipMalloc((void**)&dev, nc), "hipMalloc(staging)");
    cap = nc;
    return FCG_OK;
  }
  // Region [off, off + n) of both rings, free for writing.
  fcg_status acquire(size_t n, size_t* off) {
    fcg_status st = reserve(n);
    if (st) return st;
    if (head + n > cap) head = 0;
    const size_t a = head, b = head + n;
    for (auto it = inflight.begin(); it != inflight.end();) {
      if (std::get<1>(*it) <= a || std::get<0>(*it) >= b) {
        ++it;
        continue;
      }
      HIP_TRY(hipEventSynchronize(std::get<2>(*it)), "hipEventSynchronize(staging)");
      spare.push_back(std::get<2>(*it));
      it = inflight.erase(it);
    }
    head = b;
    *off = a;
    return FCG_OK;
  }
  fcg_status retire(size_t off, size_t n, hipStream_t s) {
    hipEvent_t e;
    if (!spare.empty()) {
      e = spare.back();
      spare.pop_back();
    } else {
      HIP_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate");
    }
    HIP_TRY(hipEventRecord(e, s), "hipEventRecord");
    inflight.emplace_back(off, off + n, e);
    return FCG_OK;
  }
};

// Packs host arrays into one blob with 256-byte aligned members.
struct Blob {
  std::vector<char> bytes;
  size_t add(const void* p, size_t n) {
    size_t off = (bytes.size() + 255) & ~size_t(255);
    bytes.resize(off + n);
    if (n) std::memcpy(bytes.data() + off, p, n);
    return off;
  }
};

}  // namespace

struct Segment {
  int64_t tok_off;  // first token in the device slabs, -1 while offloaded
  int32_t len, src_pos0;
  int64_t host_off = -1;  // first token in the pinned host slabs, -1 without a host copy
  mutable int32_t pins = 0;  // FCG_ALIAS_V caches reading this segment's values in place
};

struct fcg_lib {
  fcg_model_desc desc;
  int64_t cap = 0, used = 0;              // device slab tokens: capacity, high-water mark
  std::map<int64_t, int64_t> free_tok;    // device token ranges below `used` freed by offloads (start -> length)
  int32_t max_segments = 0;
  uint32_t flags = 0;
  std::vector<Segment> segs;
  void* k = nullptr;
  void* v = nullptr;
  int device = 0;
  // host tier (fcg_lib_host_reserve): pinned [L][Hkv][host_cap][D] slabs, filled once per segment
  int64_t host_cap = 0, host_used = 0;
  void* host_k = nullptr;
  void* host_v = nullptr;
  hipEvent_t freed = nullptr;  // after the copies that read the last freed device range
  // Ordering across streams (offload / reload on a side stream beside grafts):
  // a graft waits for the last reload; a reload or an ingest into a freed
  // range waits for the last graft (which may still read that range) and the
  // offload that freed it.
  mutable hipEvent_t graft_done = nullptr;
  hipEvent_t reload_done = nullptr;

  // first fit among freed ranges, else past the high-water mark; -1 if nothing fits
  int64_t alloc(int64_t len) {
    for (auto it = free_tok.begin(); it != free_tok.end(); ++it)
      if (it->second >= len) {
        const int64_t off = it->first, rest = it->second - len;
        free_tok.erase(it);
        if (rest) free_tok[off + len] = rest;
        return off;
      }
    if (used + len > cap) return -1;
    used += len;
    return used - len;
  }
  void release(int64_t off, int64_t len) {
    auto it = free_tok.emplace(off, len).first;
    auto nx = std::next(it);
    if (nx != free_tok.end() && it->first + it->second == nx->first) {
      it->second += nx->second;
      free_tok.erase(nx);
    }
    if (it != free_tok.begin()) {
      auto pv = std::prev(it);
      if (pv->first + pv->second == it->first) {
        pv->second += it->second;
        free_tok.erase(it);
        it = pv;
      }
    }
    if (it->first + it->second == used) {  // the top range returns to the high-water mark
      used = it->first;
      free_tok.erase(it);
    }
  }
};

struct fcg_cache {
  fcg_model_desc desc;
  int32_t n_seqs, max_tokens, page_size, n_pages;
  uint32_t flags;
  Planner plan;
  void* k = nullptr;
  void* v = nullptr;
  int64_t layer_stride = 0;
  int32_t* d_page_table = nullptr;
  double* d_inv_freq = nullptr;
  float2* d_rope = nullptr;   // (cos, sin) per position and rotary pair [max_tokens][D/2]
  int device = 0;
  Ring ring;
  // workspaces, grown on demand
  void* qws = nullptr;
  size_t qws_bytes = 0;
  float* part = nullptr;
  size_t part_bytes = 0;
  float* dpart = nullptr;     // decode split partials
  size_t dpart_bytes = 0;
  const fcg_lib* alias_lib = nullptr;  // FCG_ALIAS_V: the library value pages map onto (bound by the first graft)
  std::vector<std::vector<int32_t>> alias_segs;  // per sequence: segments it pins in alias_lib
  int32_t* d_count = nullptr; // decode merge arrival counters [kMaxDecodeSeqs][Hkv] (kCountStride apart), zero between launches
  // kernel timing (fcg_cache_timing): recorded (start, end) event pairs per kind
  bool timing = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> spans[5];
  std::vector<hipEvent_t> ev_pool;
  std::unordered_map<hipEvent_t, int> ev_refs;

  fcg_cache(const fcg_model_desc& d, int32_t ns, int32_t mt, int32_t ps, int32_t np, uint32_t fl)
      : desc(d), n_seqs(ns), max_tokens(mt), page_size(ps), n_pages(np), flags(fl),
        plan(d.n_layers, ns, mt, ps, np, (fl & FCG_ALIAS_V) != 0) {}
  bool layout_only() const { return flags & FCG_LAYOUT_ONLY; }

  CacheView view() const {
    CacheView c;
    c.k = k;
    c.v = v;
    c.layer_stride = layer_stride;
    c.page_table = d_page_table;
    c.v_alias = plan.alias_v() && d_page_table ? d_page_table + plan.n_logical_pages() : nullptr;
    c.lib_v = alias_lib ? alias_lib->v : nullptr;
    c.lib_cap = alias_lib ? alias_lib->cap : 0;
    c.n_seqs = n_seqs;
    c.max_tokens = max_tokens;
    c.page_size = page_size;
    c.n_lp = plan.n_logical_pages();
    c.n_kv_heads = desc.n_kv_heads;
    c.head_dim = desc.head_dim;
    return c;
  }
};

namespace {

// Kernel timing.  Events come from a per-cache pool and are attached to
// kernel dispatches (KTime); an event may close one interval and belong to
// another (the last kernel of a call ends both its own interval and the
// call's), so events carry a reference count and return to the pool at zero.
hipEvent_t timing_event(fcg_cache* c) {
  if (!c->timing) return nullptr;
  hipEvent_t e = nullptr;
  if (!c->ev_pool.empty()) {
    e = c->ev_pool.back();
    c->ev_pool.pop_back();
  } else if (hipEventCreate(&e) != hipSuccess) {
    return nullptr;
  }
  c->ev_refs[e] = 0;
  return e;
}

void event_put(fcg_cache* c, hipEvent_t e) {
  auto it = c->ev_refs.find(e);
  if (it == c->ev_refs.end()) return;
  if (--it->second <= 0) {
    c->ev_refs.erase(it);
    c->ev_pool.push_back(e);
  }
}

// Open an interval of `kind` at event e (the start event of a kernel).
void time_open(fcg_cache* c, int kind, hipEvent_t e) {
  if (!e) return;
  ++c->ev_refs[e];
  c->spans[kind].push_back({e, nullptr});
}

// Close the open interval of `kind` at event e (the stop event of a kernel).
void time_close(fcg_cache* c, int kind, hipEvent_t e) {
  if (!e || c->spans[kind].empty() || c->spans[kind].back().second) return;
  ++c->ev_refs[e];
  c->spans[kind].back().second = e;
}

// Unused events of a call (a kernel not launched) go back to the pool.
void time_drop(fcg_cache* c, hipEvent_t e) {
  auto it = c->ev_refs.find(e);
  if (it != c->ev_refs.end() && it->second == 0) {
    c->ev_refs.erase(it);
    c->ev_pool.push_back(e);
  }
}

fcg_status grow(void** p, size_t* have, size_t need, const char* what) {
  if (need <= *have) return FCG_OK;
  // at least twice the old size, so that a workload whose need creeps up (a
  // sequence crossing a split boundary every few decode steps) reallocates
  // rarely: each reallocation waits for the device
  const size_t n = std::max(need, *have * 2);
  if (*p) {
    HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize(grow)");
    hipFree(*p);
    *p = nullptr;
    *have = 0;
  }
  hipError_t e = hipMalloc(p, n);
  if (e != hipSuccess) return fail(FCG_ENOMEM, std::string("hipMalloc(") + what + ") failed");
  *have = n;
  return FCG_OK;
}

// After a planner check: map the new pages, and prepare the device copies of
// the touched page-table rows (appended to the blob).
// The device row of seq: its page row, then its value-alias row.
size_t stage_row(const fcg_cache* c, int32_t seq, Blob* blob) {
  const size_t nlp = c->plan.n_logical_pages();
  std::vector<int32_t> row(2 * nlp);
  std::memcpy(row.data(), c->plan.page_row(seq), nlp * sizeof(int32_t));
  std::memcpy(row.data() + nlp, c->plan.alias_row(seq), nlp * sizeof(int32_t));
  return blob->add(row.data(), row.size() * sizeof(int32_t));
}

void stage_pages(fcg_cache* c, const std::vector<std::pair<int32_t, int32_t>>& new_pages, Blob* blob,
                 std::vector<std::pair<int32_t, size_t>>* rows) {
  c->plan.map_pages(new_pages);
  std::vector<int32_t> seqs;
  for (auto& sl : new_pages) seqs.push_back(sl.first);
  std::sort(seqs.begin(), seqs.end());
  seqs.erase(std::unique(seqs.begin(), seqs.end()), seqs.end());
  for (int32_t s : seqs) rows->push_back({s, stage_row(c, s, blob)});
}

// Upload the blob; copy page rows into the device page table.  *dev receives
// the device address of the blob.
fcg_status upload(fcg_cache* c, const Blob& blob, const std::vector<std::pair<int32_t, size_t>>& rows,
                  hipStream_t s, char** dev, size_t* off_out) {
  size_t n = std::max<size_t>(blob.bytes.size(), 256), off;
  fcg_status st = c->ring.acquire(n, &off);
  if (st) return st;
  std::memcpy(c->ring.host + off, blob.bytes.data(), blob.bytes.size());
  HIP_TRY(hipMemcpyAsync(c->ring.dev + off, c->ring.host + off, blob.bytes.size(), hipMemcpyHostToDevice, s),
          "hipMemcpyAsync(plan)");
  const size_t nlp = c->plan.n_logical_pages();
  for (auto& r : rows)
    HIP_TRY(hipMemcpyAsync(c->d_page_table + (size_t)r.first * 2 * nlp, c->ring.dev + off + r.second,
                           2 * nlp * sizeof(int32_t), hipMemcpyDeviceToDevice, s),
            "hipMemcpyAsync(page table)");
  *dev = c->ring.dev + off;
  *off_out = off;
  return FCG_OK;
}

}  // namespace

extern "C" {

const char* fcg_status_string(fcg_status s) {
  switch (s) {
    case FCG_OK: return "FCG_OK";
    case FCG_EINVAL: return "FCG_EINVAL";
    case FCG_ERANGE: return "FCG_ERANGE";
    case FCG_EOVERLAP: return "FCG_EOVERLAP";
    case FCG_EHOLE: return "FCG_EHOLE";
    case FCG_ENOMEM: return "FCG_ENOMEM";
    case FCG_ESTATE: return "FCG_ESTATE";
    case FCG_EHIP: return "FCG_EHIP";
  }
  return "FCG_UNKNOWN";
}

const char* fcg_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------ library

fcg_status fcg_lib_create(const fcg_model_desc* desc, int64_t capacity_tokens, int32_t max_segments, uint32_t flags,
                          fcg_lib** out) {
  if (!out) return fail(FCG_EINVAL, "null output handle");
  if (fcg_status st = check_desc(desc)) return st;
  if (capacity_tokens < 1 || max_segments < 1) return fail(FCG_EINVAL, "capacity and max_segments must be >= 1");
  if (flags & ~FCG_LAYOUT_ONLY) return fail(FCG_EINVAL, "unknown flags");
  fcg_lib* lib = new (std::nothrow) fcg_lib();
  if (!lib) return fail(FCG_ENOMEM, "host allocation");
  lib->desc = *desc;
  lib->cap = capacity_tokens;
  lib->max_segments = max_segments;
  lib->flags = flags;
  if (flags & FCG_LAYOUT_ONLY) {
    *out = lib;
    return FCG_OK;
  }
  hipGetDevice(&lib->device);
  const size_t bytes = (size_t)desc->n_layers * desc->n_kv_heads * capacity_tokens * desc->head_dim * esize(desc->dtype);
  if (hipMalloc(&lib->k, bytes) != hipSuccess || hipMalloc(&lib->v, bytes) != hipSuccess) {
    if (lib->k) hipFree(lib->k);
    delete lib;
    return fail(FCG_ENOMEM, "library slabs do not fit in device memory");
  }
  if (hipEventCreateWithFlags(&lib->freed, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&lib->graft_done, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&lib->reload_done, hipEventDisableTiming) != hipSuccess) {
    fcg_lib_destroy(lib);
    return fail(FCG_EHIP, "hipEventCreate");
  }
  *out = lib;
  return FCG_OK;
}

fcg_status fcg_lib_add_segment(fcg_lib* lib, int32_t len, int32_t src_pos0, const void* k, const void* v,
                               void* stream, int32_t* seg_id) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (len < 1) return fail(FCG_EINVAL, "segment length must be >= 1");
  if (src_pos0 < 0) return fail(FCG_ERANGE, "negative source position");
  if ((k == nullptr) != (v == nullptr)) return fail(FCG_EINVAL, "k and v must both be given or both be null");
  if (k && (lib->flags & FCG_LAYOUT_ONLY)) return fail(FCG_EINVAL, "a layout-only library takes no data");
  if ((int32_t)lib->segs.size() >= lib->max_segments) return fail(FCG_ENOMEM, "max_segments reached");
  const bool reuse = !lib->free_tok.empty();
  const int64_t off = lib->alloc(len);
  if (off < 0) return fail(FCG_ENOMEM, "library capacity exhausted");
  const Segment sg{off, len, src_pos0};
  if (!(lib->flags & FCG_LAYOUT_ONLY)) {
    HIP_TRY(hipSetDevice(lib->device), "hipSetDevice");
    // a range an offload freed is written only after that offload has read it
    // and after the last graft (which may have read it) has run
    if (reuse) {
      HIP_TRY(hipStreamWaitEvent((hipStream_t)stream, lib->freed, 0), "hipStreamWaitEvent");
      HIP_TRY(hipStreamWaitEvent((hipStream_t)stream, lib->graft_done, 0), "hipStreamWaitEvent");
    }
  }
  if (k) {
    const fcg_model_desc& d = lib->desc;
    int rc = launch_lib_ingest(d.dtype, k, v, lib->k, lib->v, d.n_layers, len, d.n_kv_heads, d.head_dim, lib->cap,
                               sg.tok_off, (hipStream_t)stream);
    if (rc) {
      lib->release(off, len);
      return hip_fail((hipError_t)rc, "ingest launch");
    }
  }
  lib->segs.push_back(sg);
  if (seg_id) *seg_id = (int32_t)lib->segs.size() - 1;
  return FCG_OK;
}

fcg_status fcg_lib_host_reserve(fcg_lib* lib, int64_t host_tokens) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (host_tokens < 1) return fail(FCG_EINVAL, "host_tokens must be >= 1");
  if (lib->host_cap) return fail(FCG_ESTATE, "the host tier is already reserved");
  if (!(lib->flags & FCG_LAYOUT_ONLY)) {
    HIP_TRY(hipSetDevice(lib->device), "hipSetDevice");
    const fcg_model_desc& d = lib->desc;
    const size_t bytes = (size_t)d.n_layers * d.n_kv_heads * host_tokens * d.head_dim * esize(d.dtype);
    if (hipHostMalloc(&lib->host_k, bytes, hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc(&lib->host_v, bytes, hipHostMallocDefault) != hipSuccess) {
      if (lib->host_k) hipHostFree(lib->host_k);
      lib->host_k = nullptr;
      return fail(FCG_ENOMEM, "pinned host slabs");
    }
  }
  lib->host_cap = host_tokens;
  return FCG_OK;
}

namespace {

// Copy a segment between the device slabs and the host slabs: rows are the
// (layer, kv head) runs of len tokens, at the two slabs' own pitches.
fcg_status copy_segment(fcg_lib* lib, const Segment& sg, bool to_host, hipStream_t s) {
  const fcg_model_desc& d = lib->desc;
  const size_t es = esize(d.dtype), row = (size_t)d.head_dim * es;
  const size_t dpitch = (size_t)lib->cap * row, hpitch = (size_t)lib->host_cap * row;
  const size_t width = (size_t)sg.len * row, height = (size_t)d.n_layers * d.n_kv_heads;
  for (int kv = 0; kv < 2; ++kv) {
    char* dev = (char*)(kv ? lib->v : lib->k) + sg.tok_off * row;
    char* host = (char*)(kv ? lib->host_v : lib->host_k) + sg.host_off * row;
    const hipError_t e = to_host ? hipMemcpy2DAsync(host, hpitch, dev, dpitch, width, height, hipMemcpyDeviceToHost, s)
                                 : hipMemcpy2DAsync(dev, dpitch, host, hpitch, width, height, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy2DAsync(segment)");
  }
  return FCG_OK;
}

}  // namespace

fcg_status fcg_lib_offload(fcg_lib* lib, int32_t seg_id, void* stream) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (seg_id < 0 || seg_id >= (int32_t)lib->segs.size()) return fail(FCG_ERANGE, "segment id out of range");
  Segment& sg = lib->segs[seg_id];
  if (sg.tok_off < 0) return fail(FCG_ESTATE, "segment is not in device memory");
  if (sg.pins) return fail(FCG_ESTATE, "a cache reads this segment's values in place (FCG_ALIAS_V)");
  if (!lib->host_cap) return fail(FCG_ESTATE, "no host tier (fcg_lib_host_reserve)");
  const bool copy = sg.host_off < 0;
  if (copy && lib->host_used + sg.len > lib->host_cap) return fail(FCG_ENOMEM, "host tier full");
  hipStream_t s = (hipStream_t)stream;
  if (copy) {
    sg.host_off = lib->host_used;
    if (!(lib->flags & FCG_LAYOUT_ONLY)) {
      HIP_TRY(hipSetDevice(lib->device), "hipSetDevice");
      if (fcg_status st = copy_segment(lib, sg, true, s)) {
        sg.host_off = -1;
        return st;
      }
    }
    lib->host_used += sg.len;
  }
  if (!(lib->flags & FCG_LAYOUT_ONLY)) HIP_TRY(hipEventRecord(lib->freed, s), "hipEventRecord");
  lib->release(sg.tok_off, sg.len);
  sg.tok_off = -1;
  return FCG_OK;
}

fcg_status fcg_lib_reload(fcg_lib* lib, int32_t seg_id, void* stream) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (seg_id < 0 || seg_id >= (int32_t)lib->segs.size()) return fail(FCG_ERANGE, "segment id out of range");
  Segment& sg = lib->segs[seg_id];
  if (sg.tok_off >= 0) return fail(FCG_ESTATE, "segment is already in device memory");
  const int64_t off = lib->alloc(sg.len);
  if (off < 0) return fail(FCG_ENOMEM, "library capacity exhausted");
  sg.tok_off = off;
  if (!(lib->flags & FCG_LAYOUT_ONLY)) {
    HIP_TRY(hipSetDevice(lib->device), "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    fcg_status st = FCG_OK;
    if (hipStreamWaitEvent(s, lib->freed, 0) != hipSuccess || hipStreamWaitEvent(s, lib->graft_done, 0) != hipSuccess)
      st = fail(FCG_EHIP, "hipStreamWaitEvent");
    if (!st) st = copy_segment(lib, sg, false, s);
    if (!st && hipEventRecord(lib->reload_done, s) != hipSuccess) st = fail(FCG_EHIP, "hipEventRecord");
    if (st) {
      lib->release(off, sg.len);
      sg.tok_off = -1;
      return st;
    }
  }
  return FCG_OK;
}

fcg_status fcg_lib_segment_state(const fcg_lib* lib, int32_t seg_id, int32_t* in_device, int32_t* on_host) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (seg_id < 0 || seg_id >= (int32_t)lib->segs.size()) return fail(FCG_ERANGE, "segment id out of range");
  const Segment& sg = lib->segs[seg_id];
  if (in_device) *in_device = sg.tok_off >= 0;
  if (on_host) *on_host = sg.host_off >= 0;
  return FCG_OK;
}

fcg_status fcg_lib_update_residency(fcg_lib* lib, const fcg_locality* loc, int64_t budget_bytes, double ppl_threshold,
                                    void* stream, int32_t* n_offloaded, int32_t* n_reloaded) {
  if (!lib || !loc) return fail(FCG_EINVAL, "null library or scorer");
  const int32_t n = (int32_t)lib->segs.size();
  if (locality_size(loc) != n) return fail(FCG_EINVAL, "the scorer must track one function per library segment");
  if (!(ppl_threshold >= 0)) return fail(FCG_EINVAL, "the perplexity threshold must be >= 0");
  const fcg_model_desc& d = lib->desc;
  const int64_t b_tok = 2LL * d.n_layers * d.n_kv_heads * d.head_dim * (int64_t)esize(d.dtype);  // K+V, all layers
  if (budget_bytes < 0) {
    // the hyperparameter table's GPU memory threshold and reserve: 0.85 of the
    // device memory, less 2 GB, less what the rest of the process holds; never
    // more than the slabs
    budget_bytes = lib->cap * b_tok;
    if (!(lib->flags & FCG_LAYOUT_ONLY)) {
      HIP_TRY(hipSetDevice(lib->device), "hipSetDevice");
      size_t free_b = 0, total_b = 0;
      HIP_TRY(hipMemGetInfo(&free_b, &total_b), "hipMemGetInfo");
      const int64_t others = (int64_t)(total_b - free_b) - lib->cap * b_tok;
      const int64_t limit = (int64_t)(0.85 * (double)total_b) - (2LL << 30) - std::max<int64_t>(others, 0);
      budget_bytes = std::max<int64_t>(0, std::min(budget_bytes, limit));
    }
  }
  std::vector<int64_t> cost(n);
  std::vector<uint8_t> pinned(n), keep(n);
  for (int32_t f = 0; f < n; ++f) {
    cost[f] = lib->segs[f].len * b_tok;
    pinned[f] = lib->segs[f].pins > 0;
  }
  if (fcg_status st = locality_residency(loc, budget_bytes, cost.data(), ppl_threshold, pinned.data(), keep.data()))
    return st;
  int32_t n_off = 0, n_re = 0;
  // offloads first: they free the ranges the reloads may take
  for (int32_t f = 0; f < n; ++f)
    if (!keep[f] && lib->segs[f].tok_off >= 0) {
      if (fcg_status st = fcg_lib_offload(lib, f, stream)) return st;
      ++n_off;
    }
  for (int32_t f = 0; f < n; ++f)
    if (keep[f] && lib->segs[f].tok_off < 0) {
      if (fcg_status st = fcg_lib_reload(lib, f, stream)) return st;
      ++n_re;
    }
  if (n_offloaded) *n_offloaded = n_off;
  if (n_reloaded) *n_reloaded = n_re;
  return FCG_OK;
}

fcg_status fcg_lib_segment_info(const fcg_lib* lib, int32_t seg_id, int64_t* tok_off, int32_t* len,
                                int32_t* src_pos0) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (seg_id < 0 || seg_id >= (int32_t)lib->segs.size()) return fail(FCG_ERANGE, "segment id out of range");
  const Segment& s = lib->segs[seg_id];
  if (tok_off) *tok_off = s.tok_off;
  if (len) *len = s.len;
  if (src_pos0) *src_pos0 = s.src_pos0;
  return FCG_OK;
}

fcg_status fcg_lib_device_ptrs(const fcg_lib* lib, int32_t layer, void** k, void** v) {
  if (!lib) return fail(FCG_EINVAL, "null library");
  if (lib->flags & FCG_LAYOUT_ONLY) return fail(FCG_ESTATE, "layout-only library has no device memory");
  if (layer < 0 || layer >= lib->desc.n_layers) return fail(FCG_ERANGE, "layer out of range");
  const size_t off = (size_t)layer * lib->desc.n_kv_heads * lib->cap * lib->desc.head_dim * esize(lib->desc.dtype);
  if (k) *k = (char*)lib->k + off;
  if (v) *v = (char*)lib->v + off;
  return FCG_OK;
}

fcg_status fcg_lib_destroy(fcg_lib* lib) {
  if (!lib) return FCG_OK;
  if (lib->flags & FCG_LAYOUT_ONLY) {
    delete lib;
    return FCG_OK;
  }
  hipSetDevice(lib->device);
  hipDeviceSynchronize();
  if (lib->k) hipFree(lib->k);
  if (lib->v) hipFree(lib->v);
  if (lib->host_k) hipHostFree(lib->host_k);
  if (lib->host_v) hipHostFree(lib->host_v);
  if (lib->freed) hipEventDestroy(lib->freed);
  if (lib->graft_done) hipEventDestroy(lib->graft_done);
  if (lib->reload_done) hipEventDestroy(lib->reload_done);
  delete lib;
  return FCG_OK;
}

// -------------------------------------------------------------------- cache

fcg_status fcg_cache_create(const fcg_model_desc* desc, int32_t n_seqs, int32_t max_tokens, int32_t page_size,
                            int32_t n_pages, uint32_t flags, fcg_cache** out) {
  if (!out) return fail(FCG_EINVAL, "null output handle");
  if (fcg_status st = check_desc(desc)) return st;
  if (n_seqs < 1 || max_tokens < 1) return fail(FCG_EINVAL, "n_seqs and max_tokens must be >= 1");
  if ((int64_t)max_tokens * desc->head_dim >= ((int64_t)1 << 31))
    return fail(FCG_EINVAL, "max_tokens * head_dim must stay below 2^31");
  if (page_size != 0 && page_size != 16) return fail(FCG_EINVAL, "page_size must be 0 (contiguous) or 16");
  if (page_size && n_pages < 1) return fail(FCG_EINVAL, "a paged cache needs n_pages >= 1");
  if (flags & ~(FCG_LAYOUT_ONLY | FCG_ALIAS_V)) return fail(FCG_EINVAL, "unknown flags");
  if ((flags & FCG_ALIAS_V) && !page_size) return fail(FCG_EINVAL, "FCG_ALIAS_V needs a paged cache");
  fcg_cache* c = new (std::nothrow) fcg_cache(*desc, n_seqs, max_tokens, page_size, page_size ? n_pages : 0, flags);
  if (!c) return fail(FCG_ENOMEM, "host allocation");
  if (!c->layout_only()) {
    hipGetDevice(&c->device);
    const int64_t per_layer = page_size ? (int64_t)n_pages * desc->n_kv_heads * page_size * desc->head_dim
                                        : (int64_t)n_seqs * desc->n_kv_heads * max_tokens * desc->head_dim;
    c->layer_stride = per_layer;
    const size_t bytes = (size_t)per_layer * desc->n_layers * esize(desc->dtype);
    bool ok = hipMalloc(&c->k, bytes) == hipSuccess && hipMalloc(&c->v, bytes) == hipSuccess;
    if (ok && page_size) {
      const size_t pt = (size_t)n_seqs * 2 * c->plan.n_logical_pages() * sizeof(int32_t);
      ok = hipMalloc((void**)&c->d_page_table, pt) == hipSuccess && hipMemset(c->d_page_table, 0xFF, pt) == hipSuccess;
    }
    if (ok) {
      const size_t nc = (size_t)kMaxDecodeSeqs * desc->n_kv_heads * kCountStride * sizeof(int32_t);
      ok = hipMalloc((void**)&c->d_count, nc) == hipSuccess && hipMemset(c->d_count, 0, nc) == hipSuccess;
    }
    if (!ok) {
      fcg_cache_destroy(c);
      return fail(FCG_ENOMEM, "cache does not fit in device memory");
    }
    if (fcg_status st = upload_inv_freq(*desc, &c->d_inv_freq)) {
      fcg_cache_destroy(c);
      return st;
    }
    // rotary table of every position the cache can hold, computed once here
    const int half = desc->head_dim / 2;
    if (hipMalloc((void**)&c->d_rope, (size_t)max_tokens * half * sizeof(float2)) != hipSuccess) {
      fcg_cache_destroy(c);
      return fail(FCG_ENOMEM, "rotary table does not fit in device memory");
    }
    int rc = launch_rope_table(c->d_inv_freq, half, max_tokens, c->d_rope, nullptr);
    if (rc == 0) rc = (int)hipStreamSynchronize(nullptr);
    if (rc) {
      fcg_cache_destroy(c);
      return hip_fail((hipError_t)rc, "rotary table");
    }

  }
  *out = c;
  return FCG_OK;
}

fcg_status fcg_cache_reset(fcg_cache* c, int32_t seq) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (seq < 0 || seq >= c->n_seqs) return fail(FCG_ERANGE, "sequence out of range");
  c->plan.reset(seq);
  if (!c->alias_segs.empty()) {
    for (int32_t g : c->alias_segs[seq]) --c->alias_lib->segs[g].pins;
    c->alias_segs[seq].clear();
  }
  // the device page-table row is rewritten on the next mapping of this
  // sequence; stale entries are never read because unwritten positions are
  // never read
  return FCG_OK;
}

fcg_status fcg_cache_truncate(fcg_cache* c, int32_t seq, int32_t pos, void* stream) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (seq < 0 || seq >= c->n_seqs) return fail(FCG_ERANGE, "sequence out of range");
  if (pos < 0 || pos > c->max_tokens) return fail(FCG_ERANGE, "position out of range");
  std::vector<Unalias> un;
  c->plan.truncate(seq, pos, &un);  // freed page-table rows: as for fcg_cache_reset
  if (un.empty() || c->layout_only()) return FCG_OK;
  // a value page mapped onto the library and split by the cut: copy its kept
  // rows into the page and upload the sequence's row without the alias
  HIP_TRY(hipSetDevice(c->device), "hipSetDevice");
  hipStream_t s = (hipStream_t)stream;
  Blob blob;
  std::vector<std::pair<int32_t, size_t>> rows{{seq, stage_row(c, seq, &blob)}};
  std::vector<UnaliasItem> items;
  for (const Unalias& u : un) items.push_back(UnaliasItem{u.lib_tok, u.page, u.rows});
  const size_t o_items = blob.add(items.data(), items.size() * sizeof(UnaliasItem));
  char* dev;
  size_t off;
  if (fcg_status st = upload(c, blob, rows, s, &dev, &off)) return st;
  int rc = launch_unalias(c->desc.dtype, (const UnaliasItem*)(dev + o_items), (int)items.size(), c->alias_lib->v,
                          c->alias_lib->cap, c->view(), c->desc.n_layers, s);
  if (rc) return hip_fail((hipError_t)rc, "unalias launch");
  return c->ring.retire(off, blob.bytes.size(), s);
}

fcg_status fcg_cache_export_v_alias(const fcg_cache* c, int32_t seq, int32_t* v_alias) {
  if (!c || !v_alias) return fail(FCG_EINVAL, "null cache or output");
  if (seq < 0 || seq >= c->n_seqs) return fail(FCG_ERANGE, "sequence out of range");
  std::memcpy(v_alias, c->plan.alias_row(seq), sizeof(int32_t) * c->plan.n_logical_pages());
  return FCG_OK;
}

fcg_status fcg_cache_export_layout(const fcg_cache* c, int32_t seq, int32_t layer, int32_t* page_table,
                                   int32_t* seq_len, uint8_t* written) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (seq < 0 || seq >= c->n_seqs) return fail(FCG_ERANGE, "sequence out of range");
  if (layer < 0 || layer >= c->desc.n_layers) return fail(FCG_ERANGE, "layer out of range");
  if (page_table && c->page_size)
    std::memcpy(page_table, c->plan.page_row(seq), sizeof(int32_t) * c->plan.n_logical_pages());
  if (seq_len) *seq_len = c->plan.seq_len(seq, layer);
  if (written)
    for (int32_t p = 0; p < c->max_tokens; ++p) written[p] = c->plan.written(seq, layer, p) ? 1 : 0;
  return FCG_OK;
}

fcg_status fcg_cache_device_ptrs(const fcg_cache* c, int32_t layer, void** k, void** v) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (c->layout_only()) return fail(FCG_ESTATE, "layout-only cache has no device memory");
  if (layer < 0 || layer >= c->desc.n_layers) return fail(FCG_ERANGE, "layer out of range");
  const size_t off = (size_t)layer * c->layer_stride * esize(c->desc.dtype);
  if (k) *k = (char*)c->k + off;
  if (v) *v = (char*)c->v + off;
  return FCG_OK;
}

fcg_status fcg_cache_timing(fcg_cache* c, int32_t enable) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  c->timing = enable != 0;
  return FCG_OK;
}

fcg_status fcg_cache_timing_read(fcg_cache* c, int32_t kind, int32_t* count, double* total_ms) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (kind < 0 || kind > FCG_TIME_DECODE_ATTN) return fail(FCG_ERANGE, "unknown timing kind");
  double ms = 0.0;
  int32_t n = 0;
  for (auto& sp : c->spans[kind]) {
    if (sp.second) {
      HIP_TRY(hipEventSynchronize(sp.second), "hipEventSynchronize(timing)");
      float t = 0.f;
      HIP_TRY(hipEventElapsedTime(&t, sp.first, sp.second), "hipEventElapsedTime");
      ms += t;
      ++n;
      event_put(c, sp.second);
    }
    event_put(c, sp.first);
  }
  c->spans[kind].clear();
  if (count) *count = n;
  if (total_ms) *total_ms = ms;
  return FCG_OK;
}

fcg_status fcg_cache_destroy(fcg_cache* c) {
  if (!c) return FCG_OK;
  for (auto& v : c->alias_segs)
    for (int32_t g : v) --c->alias_lib->segs[g].pins;
  if (!c->layout_only()) {
    hipSetDevice(c->device);
    hipDeviceSynchronize();
    c->ring.release();
    if (c->k) hipFree(c->k);
    if (c->v) hipFree(c->v);
    if (c->d_page_table) hipFree(c->d_page_table);
    if (c->d_inv_freq) hipFree(c->d_inv_freq);
    if (c->d_rope) hipFree(c->d_rope);
    if (c->qws) hipFree(c->qws);
    if (c->part) hipFree(c->part);
    if (c->dpart) hipFree(c->dpart);
    if (c->d_count) hipFree(c->d_count);
    for (auto& v : c->spans)
      for (auto& sp : v) {
        if (sp.first) hipEventDestroy(sp.first);
        if (sp.second) hipEventDestroy(sp.second);
      }
    for (auto e : c->ev_pool) hipEventDestroy(e);

  }
  delete c;
  return FCG_OK;
}

// ----------------------------------------------------------------- hot path

fcg_status fcg_graft(fcg_cache* c, const fcg_lib* lib, int32_t n_items, const int32_t* seq, const int32_t* seg,
                     const int32_t* dst, void* stream) {
  if (!c || !lib) return fail(FCG_EINVAL, "null cache or library");
  if (n_items < 0) return fail(FCG_EINVAL, "negative item count");
  if (n_items > 0 && (!seq || !seg || !dst)) return fail(FCG_EINVAL, "null item array");
  if (!same_shape(c->desc, lib->desc)) return fail(FCG_EINVAL, "library and cache shapes differ");
  if ((lib->flags & FCG_LAYOUT_ONLY) && !c->layout_only())
    return fail(FCG_EINVAL, "a layout-only library can only feed a layout-only cache");
  std::vector<Span> spans(n_items);
  for (int32_t i = 0; i < n_items; ++i) {
    if (seg[i] < 0 || seg[i] >= (int32_t)lib->segs.size()) return fail(FCG_ERANGE, "segment id out of range");
    const Segment& sg = lib->segs[seg[i]];
    spans[i] = Span{seq[i], seg[i], dst[i], sg.len, dst[i] - sg.src_pos0};
  }
  std::vector<std::pair<int32_t, int32_t>> new_pages;
  std::string msg;
  if (fcg_status st = c->plan.check_graft(spans, &new_pages, &msg)) return fail(st, msg);
  if (n_items == 0) return FCG_OK;
  if (c->plan.alias_v() && c->alias_lib && c->alias_lib != lib)
    return fail(FCG_EINVAL, "a cache with FCG_ALIAS_V grafts from one library only");
  for (auto& sp : spans)
    if (lib->segs[sp.seg].tok_off < 0) return fail(FCG_ESTATE, "segment is not in device memory (fcg_lib_reload)");
  if (c->plan.alias_v()) {
    c->alias_lib = lib;
    if (c->alias_segs.empty()) c->alias_segs.resize(c->n_seqs);
    for (auto& sp : spans) {
      c->plan.alias_pages(sp.seq, sp.dst, sp.len, lib->segs[sp.seg].tok_off);
      ++lib->segs[sp.seg].pins;  // its values may now be read in place: no offload until the sequence is reset
      c->alias_segs[sp.seq].push_back(sp.seg);
    }
  }
  if (c->layout_only()) {
    c->plan.map_pages(new_pages);
    for (auto& s : spans) c->plan.mark_all_layers(s.seq, s.dst, s.len);
    return FCG_OK;
  }
  HIP_TRY(hipSetDevice(c->device), "hipSetDevice");
  hipStream_t s = (hipStream_t)stream;
  Blob blob;
  std::vector<std::pair<int32_t, size_t>> rows;
  stage_pages(c, new_pages, &blob, &rows);
  std::vector<GraftChunk> chunks;
  for (auto& sp : spans) {
    const Segment& sg = lib->segs[sp.seg];
    for (int32_t j = 0; j < sp.len; j += kGraftChunk)
      chunks.push_back(GraftChunk{sg.tok_off + j, sp.dst + j, sp.seq, sp.delta, std::min(kGraftChunk, sp.len - j),
                                  sp.dst, sp.dst + sp.len});
  }
  const size_t o_chunks = blob.add(chunks.data(), chunks.size() * sizeof(GraftChunk));
  char* dev;
  size_t off;
  if (fcg_status st = upload(c, blob, rows, s, &dev, &off)) return st;
  if (!(lib->flags & FCG_LAYOUT_ONLY))  // segments reloaded on another stream are in place first
    HIP_TRY(hipStreamWaitEvent(s, lib->reload_done, 0), "hipStreamWaitEvent");
  const KTime tg{timing_event(c), timing_event(c)};
  int rc = launch_graft(c->desc.dtype, (const GraftChunk*)(dev + o_chunks), (int)chunks.size(), lib->k, lib->v,
                        lib->cap, c->view(), c->d_inv_freq, c->desc.n_layers, s, tg);
  time_open(c, FCG_TIME_GRAFT, tg.start);
  time_close(c, FCG_TIME_GRAFT, tg.stop);
  if (rc) return hip_fail((hipError_t)rc, "graft launch");
  if (!(lib->flags & FCG_LAYOUT_ONLY)) HIP_TRY(hipEventRecord(lib->graft_done, s), "hipEventRecord");
  if (fcg_status st = c->ring.retire(off, blob.bytes.size(), s)) return st;
  for (auto& sp : spans) c->plan.mark_all_layers(sp.seq, sp.dst, sp.len);
  return FCG_OK;
}

namespace {

// Attention over the cache for tokens already sorted into TokenMeta ranks.
// Builds the split plan, uploads it with the page rows, then runs
// rope_append -> attention -> (combine).
fcg_status run_attention(fcg_cache* c, int32_t layer, const std::vector<TokenMeta>& meta,
                         const void* q, const void* k, const void* v, void* out,
                         const std::vector<std::pair<int32_t, int32_t>>& new_pages, hipStream_t s) {
  const fcg_model_desc& d = c->desc;
  const int n = (int)meta.size();
  const int g = d.n_q_heads / d.n_kv_heads;
  const bool mfma = d.dtype == FCG_BF16;
  // row blocks: consecutive ranks of one sequence, at most 256 (or 128) query
  // rows (MFMA) or one token
  auto row_blocks = [&](int max_rank) {
    std::vector<std::pair<int, int>> rb;  // (rank0, n_rank)
    for (int r = 0; r < n;) {
      int u = r;
      while (u < n && meta[u].seq == meta[r].seq && u - r < max_rank) ++u;
      rb.push_back({r, u - r});
      r = u;
    }
    return rb;
  };
  // bf16 calls whose tokens form, per sequence, one run of consecutive
  // positions given at consecutive caller indices (a patch span following its
  // context) run as one fused kernel: it encodes the queries itself, reads the
  // fresh keys and values from the caller's arrays and stores them into the
  // cache.  Other calls encode and append first (rope_append).
  std::vector<std::pair<int32_t, int32_t>> seq_first(d.dtype == FCG_BF16 ? n : 0);  // per rank: (f0, ftok0)
  bool fused = mfma;
  for (int r0 = 0; fused && r0 < n;) {
    int r1 = r0;
    while (r1 < n && meta[r1].seq == meta[r0].seq) {
      if (meta[r1].pos != meta[r0].pos + (r1 - r0) || meta[r1].tok != meta[r0].tok + (r1 - r0)) fused = false;
      seq_first[r1] = {meta[r0].pos, meta[r0].tok};
      ++r1;
    }
    r0 = r1;
  }
  std::vector<std::pair<int, int>> rblocks = row_blocks(mfma ? std::max(1, 256 / g) : 1);
  // MFMA: unless 256-row blocks alone fill the chip twice, use 128-row blocks
  // of 4 waves sized to run two per CU (one block's softmax beside the other's
  // matrix work), with the key splits planned for 512 blocks
  const bool pair = mfma && (int64_t)rblocks.size() * d.n_kv_heads < 512;
  if (pair) rblocks = row_blocks(std::max(1, 128 / g));
  // split the key range of each row block so that the grid covers the chip
  // once: one split length (in tiles) for the call, the smallest whose blocks
  // fit one per CU (two in pair mode); at most 256 splits per row block (the
  // merge table)
  const int tile = mfma ? 64 : 256;
  std::vector<int64_t> rb_tiles;
  int64_t total_tiles = 0, max_tiles = 0;
  for (auto& rb : rblocks) {
    rb_tiles.push_back((meta[rb.first + rb.second - 1].pos + tile) / tile);
    total_tiles += rb_tiles.back();
    max_tiles = std::max(max_tiles, rb_tiles.back());
  }
  const int min_tiles = mfma ? 2 : 1;
  auto split_tiles = [&](int64_t target) {
    int64_t per = std::max<int64_t>({(int64_t)min_tiles, (total_tiles * d.n_kv_heads + target - 1) / target,
                                     (max_tiles + 255) / 256});
    for (;;) {
      int64_t blocks = 0;
      for (int64_t nt : rb_tiles) blocks += (nt + per - 1) / per;
      if (blocks * d.n_kv_heads <= target || per >= max_tiles) break;
      ++per;
    }
    return per;
  };
  int64_t per = split_tiles(pair ? 512 : 256);
  // pair mode with splits under 8 tiles: the call is bound by latency, not by
  // the matrix work, and planning for one block per CU halves the splits the
  // combine merges (7B patch: call 35 -> 31 us, the attention kernel unchanged).
  // The 128-row blocks run as 8 waves of 16 rows (two waves per SIMD, each
  // with one row tile; 4 waves of 32 rows left one wave per SIMD: attention
  // kernel 16.0 -> 15.0 us) and keep the two-tile ring (the four-tile ring
  // measured no faster).
  bool pair_one = false;
  if (pair && per < 8) {
    per = split_tiles(256);
    pair_one = true;
  }
  const int nbuf = pair ? 2 : 4;
  const int64_t span = per * tile;
  std::vector<AttnItem> items;                 // VALU path: one item per (row block, split)
  std::vector<PrefillRb> pf_rb;                // MFMA path: row blocks, items built per launch
  std::vector<int> pf_nsplit;
  std::vector<CombineItem> comb;
  int n_part = 0;
  for (auto& rb : rblocks) {
    const int kend = meta[rb.first + rb.second - 1].pos + 1;
    const int nsplit = (int)((kend + span - 1) / span);
    const int part0 = nsplit > 1 ? n_part : -1;
    // fused calls: the output tokens follow from by-value fields, nothing is read from meta
    const int tok0 = fused ? seq_first[rb.first].second + (meta[rb.first].pos - seq_first[rb.first].first) : -1;
    if (nsplit > 1) comb.push_back(CombineItem{rb.first, rb.second, n_part, nsplit, tok0});
    pf_rb.push_back(PrefillRb{rb.first, rb.second, meta[rb.first].seq, meta[rb.first].pos, kend - 1, part0,
                              mfma ? seq_first[rb.first].first : 0, mfma ? seq_first[rb.first].second : 0});
    pf_nsplit.push_back(nsplit);
    for (int sidx = 0; sidx < nsplit; ++sidx)
      items.push_back(AttnItem{rb.first, rb.second, meta[rb.first].seq, (int)(sidx * span),
                               (int)std::min<int64_t>(kend, (sidx + 1) * span), nsplit > 1 ? n_part + sidx : -1, 0, 0});
    if (nsplit > 1) n_part += nsplit;
  }
  // MFMA launches: up to kPfMaxRb row blocks each, every row block given the
  // launch's largest split count (the extra splits are empty blocks)
  std::vector<PrefillArgs> pf_launch;
  if (mfma) {
    for (size_t b0 = 0; b0 < pf_rb.size();) {
      PrefillArgs a{};
      a.span = (int32_t)span;
      const size_t b1 = std::min(pf_rb.size(), b0 + (size_t)kPfMaxRb);
      a.n_rb = (int32_t)(b1 - b0);
      // blocks of a split grouped on one XCD (shared L2) once four or more row
      // blocks read its key tiles; with two, the pair ran in lockstep on
      // neighbouring CUs and the call was 8% slower
      a.xcd_group = a.n_rb >= 4;
      for (size_t b = b0; b < b1; ++b) {
        a.rb[b - b0] = pf_rb[b];
        a.n_split = std::max(a.n_split, pf_nsplit[b]);
      }
      pf_launch.push_back(a);
      b0 = b1;
    }
  }
  // MFMA blocks of 8 waves (256 rows) when some row block needs more than 4 waves
  int max_rows = 0;
  for (auto& rb : rblocks) max_rows = std::max(max_rows, rb.second * g);
  const int stride_rows = mfma ? (max_rows > 128 ? 256 : 128) : g;  // pair: max_rows <= 128
  // workspaces first: a failure here leaves the layout untouched
  const size_t qbytes = (size_t)d.n_kv_heads * n * g * d.head_dim * esize(d.dtype);
  if (!fused)
    if (fcg_status st = grow(&c->qws, &c->qws_bytes, qbytes, "query workspace")) return st;
  const size_t po = (size_t)n_part * d.n_kv_heads * stride_rows * d.head_dim;
  const size_t pml = (size_t)n_part * d.n_kv_heads * stride_rows * 2;
  if (n_part)
    if (fcg_status st = grow((void**)&c->part, &c->part_bytes, (po + pml) * sizeof(float), "split partials")) return st;
  Blob blob;
  std::vector<std::pair<int32_t, size_t>> rows;
  stage_pages(c, new_pages, &blob, &rows);
  // fused calls take their whole plan by value: an upload (one more copy
  // before the kernel) only when the call maps new pages
  const bool upload_plan = !fused || !rows.empty();
  const size_t o_meta = fused ? 0 : blob.add(meta.data(), meta.size() * sizeof(TokenMeta));
  const size_t o_items = mfma ? 0 : blob.add(items.data(), items.size() * sizeof(AttnItem));
  char* dev = nullptr;
  size_t off = 0;
  if (upload_plan)
    if (fcg_status st = upload(c, blob, rows, s, &dev, &off)) return st;
  const TokenMeta* dmeta = fused ? nullptr : (const TokenMeta*)(dev + o_meta);
  const CacheView cv = c->view();
  // timing: the append kernel opens the call's interval, the attention
  // launches bracket their own, the last kernel closes the call's
  const hipEvent_t e_attn0 = timing_event(c), e_attn1 = timing_event(c);
  const hipEvent_t e_call0 = fused ? e_attn0 : timing_event(c);
  const hipEvent_t e_call1 = comb.empty() ? e_attn1 : timing_event(c);
  int rc = 0;
  if (!fused) {
    rc = launch_rope_append(d.dtype, dmeta, n, q, k, v, cv, layer, c->d_rope, d.n_q_heads, c->qws, s,
                            KTime{e_call0, nullptr});
    if (rc) return hip_fail((hipError_t)rc, "append launch");
  }
  FusedIn fin;
  if (fused) fin = FusedIn{q, k, v, c->d_rope};
  float* part_o = c->part;
  float* part_ml = c->part ? c->part + po : nullptr;
  if (mfma) {
    for (size_t li = 0; li < pf_launch.size(); ++li) {
      const KTime tm{li == 0 ? e_attn0 : nullptr, li + 1 == pf_launch.size() ? e_attn1 : nullptr};
      rc = launch_attn_mfma(pf_launch[li], dmeta, c->qws, n * g, cv, layer, d.n_q_heads, out, part_o, part_ml,
                            stride_rows, nbuf, s, tm, fin, pair_one ? 16 : 32);
      if (rc) break;
    }
  } else
    rc = launch_attn_rows(d.dtype, (const AttnItem*)(dev + o_items), (int)items.size(), dmeta, c->qws, n * g, cv,
                          layer, d.n_q_heads, out, part_o, part_ml, stride_rows, s, KTime{e_attn0, e_attn1});
  if (rc) return hip_fail((hipError_t)rc, "attention launch");
  for (size_t c0 = 0; c0 < comb.size(); c0 += kCombMaxItems) {  // merge plans by value
    CombineArgs ca{};
    ca.n_items = (int32_t)std::min<size_t>(kCombMaxItems, comb.size() - c0);
    std::copy(comb.begin() + c0, comb.begin() + c0 + ca.n_items, ca.item);
    const bool last = c0 + kCombMaxItems >= comb.size();
    rc = launch_combine(d.dtype, ca, dmeta, d.n_q_heads, d.n_kv_heads, d.head_dim, part_o, part_ml, stride_rows,
                        out, s, mfma, KTime{nullptr, last ? e_call1 : nullptr});
    if (rc) return hip_fail((hipError_t)rc, "combine launch");
  }
  if (mfma && pf_launch.empty()) {  // nothing attended: no attention interval
    time_drop(c, e_attn0);
    if (e_call1 != e_attn1) time_drop(c, e_attn1);
  } else {
    time_open(c, FCG_TIME_PREFILL_ATTN, e_attn0);
    time_close(c, FCG_TIME_PREFILL_ATTN, e_attn1);
  }
  time_open(c, FCG_TIME_PREFILL, e_call0);
  time_close(c, FCG_TIME_PREFILL, e_call1);
  return upload_plan ? c->ring.retire(off, blob.bytes.size(), s) : FCG_OK;
}

// Split plan of one decode call: split length in keys and the largest number
// of partial slots any launch group needs.
struct DecodePlan {
  int64_t split_keys = 0;
  int max_slots = 0;
  size_t part_o = 0, part_ml = 0;  // floats of the partial outputs and of the (max, sum) pairs
};

DecodePlan plan_decode(const fcg_model_desc& d, int32_t n, const std::vector<int32_t>& pos) {
  const int g = d.n_q_heads / d.n_kv_heads;
  int64_t total = 0;
  int32_t pmax = 0;
  for (int32_t i = 0; i < n; ++i) {
    total += pos[i] + 1;
    pmax = std::max(pmax, pos[i]);
  }
  // split length: the smallest (from 64 keys up) whose blocks fit in one
  // wave of the grid -- one block per compute unit while that leaves at most
  // 256 keys per block (fewer partials for the merge in each (sequence, kv
  // head)'s last block), two per compute unit for more keys (shorter key
  // loops) -- rounded up to whole 64-key chunks; at most 256 splits per
  // sequence, and at most 32 when planning two blocks per compute unit: past
  // that the last block's fold of the partials costs more than the shorter
  // key loops save (16.7K-token context at batch 1: 53 splits 20.4 us per
  // call, 30 splits 19.1 us)
  const bool two_per_cu = total * d.n_kv_heads > 256 * 256;
  const int64_t target_blocks = two_per_cu ? 512 : 256;
  const int64_t max_splits = two_per_cu ? 32 : 256;
  int64_t sk = std::max<int64_t>(64, (total * d.n_kv_heads + target_blocks - 1) / target_blocks);
  sk = std::max<int64_t>(sk, (pmax + 1 + max_splits - 1) / max_splits);
  for (;;) {
    int64_t blocks = 0;
    for (int32_t i = 0; i < n; ++i) blocks += (pos[i] + sk) / sk;
    if (blocks * d.n_kv_heads <= target_blocks || blocks <= n) break;
    sk += (sk + 31) / 32;  // about 3% longer
  }
  sk = (sk + 63) / 64 * 64;
  DecodePlan p;
  p.split_keys = sk;
  // partial slots: one per split of every multi-split sequence of a launch group
  for (int32_t i0 = 0; i0 < n; i0 += kMaxDecodeSeqs) {
    int slots = 0;
    for (int32_t i = i0; i < std::min<int32_t>(n, i0 + kMaxDecodeSeqs); ++i) slots += (int)((pos[i] + sk) / sk);
    p.max_slots = std::max(p.max_slots, slots);
  }
  p.part_o = (size_t)p.max_slots * d.n_kv_heads * g * d.head_dim;
  p.part_ml = (size_t)p.max_slots * d.n_kv_heads * g * 2;
  return p;
}

// One decode launch per group of up to kMaxDecodeSeqs sequences; the launch
// merges the splits of each sequence itself and takes its plan by value
// (pages the step maps included), so a decode step uploads nothing.
// part_o / part_ml / count: the partial and counter buffers (the cache's own,
// or the static scratch of the allocation-free entry point).
fcg_status launch_decode_groups(fcg_cache* c, int32_t layer, int32_t n, const int32_t* seqs,
                                const std::vector<int32_t>& pos, const std::vector<int32_t>& new_page,
                                const DecodePlan& plan, const void* q, const void* k, const void* v, void* out,
                                float* part_o, float* part_ml, int32_t* count, bool timing, hipStream_t s) {
  const fcg_model_desc& d = c->desc;
  const CacheView cv = c->view();
  const size_t es = esize(d.dtype);
  const int64_t sk = plan.split_keys;
  for (int32_t i0 = 0; i0 < n; i0 += kMaxDecodeSeqs) {
    DecodeArgs a{};
    a.n = std::min<int32_t>(kMaxDecodeSeqs, n - i0);
    a.split_keys = (int32_t)sk;
    a.split0[0] = 0;
    for (int32_t i = 0; i < a.n; ++i) {
      a.seq[i] = seqs[i0 + i];
      a.pos[i] = pos[i0 + i];
      a.new_page[i] = new_page[i0 + i];
      const int32_t ns = (int32_t)((pos[i0 + i] + sk) / sk);
      a.split0[i + 1] = a.split0[i] + ns;
      a.max_split = std::max(a.max_split, ns);
    }
    a.slots = a.split0[a.n];
    const size_t qoff = (size_t)i0 * d.n_q_heads * d.head_dim * es, koff = (size_t)i0 * d.n_kv_heads * d.head_dim * es;
    // timing: one kernel, both intervals
    const hipEvent_t e0 = timing ? timing_event(c) : nullptr, e1 = timing ? timing_event(c) : nullptr;
    // bf16: matrix-core kernel; fp32: the vector-ALU kernel
    int rc = d.dtype == FCG_BF16
                 ? launch_decode_mfma(a, (const char*)q + qoff, (const char*)k + koff, (const char*)v + koff, cv,
                                      layer, c->d_rope, d.n_q_heads, (char*)out + qoff, part_o, part_ml, count, s,
                                      KTime{e0, e1})
                 : launch_decode(d.dtype, a, (const char*)q + qoff, (const char*)k + koff, (const char*)v + koff, cv,
                                 layer, c->d_rope, d.n_q_heads, (char*)out + qoff, part_o, part_ml, count, s,
                                 KTime{e0, e1});
    if (rc) return hip_fail((hipError_t)rc, "decode launch");
    if (timing) {
      time_open(c, FCG_TIME_DECODE_ATTN, e0);
      time_close(c, FCG_TIME_DECODE_ATTN, e1);
      time_open(c, FCG_TIME_DECODE, e0);
      time_close(c, FCG_TIME_DECODE, e1);
    }
  }
  return FCG_OK;
}

// The physical page each sequence's new token lands on when this step maps
// its page (the planner's mapping, already committed), else -1.
std::vector<int32_t> decode_new_pages(const fcg_cache* c, int32_t n, const int32_t* seqs, const std::vector<int32_t>& pos,
                                      const std::vector<std::pair<int32_t, int32_t>>& new_pages) {
  std::vector<int32_t> np(n, -1);
  if (new_pages.empty()) return np;
  for (int32_t i = 0; i < n; ++i)
    for (auto& sl : new_pages)
      if (sl.first == seqs[i] && sl.second == pos[i] / c->page_size) np[i] = c->plan.page_of(seqs[i], pos[i]);
  return np;
}

fcg_status run_decode(fcg_cache* c, int32_t layer, int32_t n, const int32_t* seqs, const std::vector<int32_t>& pos,
                      const void* q, const void* k, const void* v, void* out,
                      const std::vector<std::pair<int32_t, int32_t>>& new_pages, hipStream_t s) {
  const DecodePlan plan = plan_decode(c->desc, n, pos);
  if (fcg_status st = grow((void**)&c->dpart, &c->dpart_bytes, (plan.part_o + plan.part_ml) * sizeof(float),
                           "decode partials"))
    return st;
  c->plan.map_pages(new_pages);
  const std::vector<int32_t> np = decode_new_pages(c, n, seqs, pos, new_pages);
  return launch_decode_groups(c, layer, n, seqs, pos, np, plan, q, k, v, out, c->dpart, c->dpart + plan.part_o,
                              c->d_count, c->timing, s);
}

}  // namespace

fcg_status fcg_patch_prefill(fcg_cache* c, int32_t layer, int32_t n_tok, const int32_t* seq, const int32_t* pos,
                             const void* q, const void* k, const void* v, void* out, void* stream) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (n_tok < 0) return fail(FCG_EINVAL, "negative token count");
  if (n_tok > 0 && (!seq || !pos)) return fail(FCG_EINVAL, "null token array");
  if (n_tok > 0 && !c->layout_only() && (!q || !k || !v || !out)) return fail(FCG_EINVAL, "null tensor");
  std::vector<std::pair<int32_t, int32_t>> new_pages;
  std::string msg;
  if (fcg_status st = c->plan.check_append(layer, n_tok, seq, pos, &new_pages, &msg)) return fail(st, msg);
  if (n_tok == 0) return FCG_OK;
  if (c->layout_only()) {
    c->plan.map_pages(new_pages);
    for (int32_t t = 0; t < n_tok; ++t) c->plan.mark(seq[t], layer, pos[t]);
    return FCG_OK;
  }
  HIP_TRY(hipSetDevice(c->device), "hipSetDevice");
  std::vector<TokenMeta> meta(n_tok);
  for (int32_t t = 0; t < n_tok; ++t) meta[t] = TokenMeta{t, seq[t], pos[t], 0};
  std::sort(meta.begin(), meta.end(), [](const TokenMeta& a, const TokenMeta& b) {
    return a.seq != b.seq ? a.seq < b.seq : a.pos < b.pos;
  });
  if (fcg_status st = run_attention(c, layer, meta, q, k, v, out, new_pages, (hipStream_t)stream)) return st;
  for (int32_t t = 0; t < n_tok; ++t) c->plan.mark(seq[t], layer, pos[t]);
  return FCG_OK;
}

fcg_status fcg_decode(fcg_cache* c, int32_t layer, int32_t n_seqs, const int32_t* seqs, const void* q,
                      const void* k, const void* v, void* out, int32_t* positions_out, void* stream) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (n_seqs < 0) return fail(FCG_EINVAL, "negative sequence count");
  if (n_seqs > 0 && !seqs) return fail(FCG_EINVAL, "null sequence array");
  if (n_seqs > 0 && !c->layout_only() && (!q || !k || !v || !out)) return fail(FCG_EINVAL, "null tensor");
  std::vector<int32_t> pos;
  std::vector<std::pair<int32_t, int32_t>> new_pages;
  std::string msg;
  if (fcg_status st = c->plan.check_decode(layer, n_seqs, seqs, &pos, &new_pages, &msg)) return fail(st, msg);
  if (n_seqs == 0) return FCG_OK;
  if (!c->layout_only()) {
    HIP_TRY(hipSetDevice(c->device), "hipSetDevice");
    if (fcg_status st = run_decode(c, layer, n_seqs, seqs, pos, q, k, v, out, new_pages, (hipStream_t)stream))
      return st;
  } else {
    c->plan.map_pages(new_pages);
  }
  for (int32_t i = 0; i < n_seqs; ++i) {
    c->plan.mark(seqs[i], layer, pos[i]);
    if (positions_out) positions_out[i] = pos[i];
  }
  return FCG_OK;
}

fcg_status fcg_decode_noalloc(fcg_cache* c, int32_t layer, int32_t n_seqs, const int32_t* seqs, const void* q,
                              const void* k, const void* v, void* out, int32_t* positions_out, void* stream) {
  if (!c) return fail(FCG_EINVAL, "null cache");
  if (n_seqs < 0) return fail(FCG_EINVAL, "negative sequence count");
  if (n_seqs > 0 && !seqs) return fail(FCG_EINVAL, "null sequence array");
  if (n_seqs > 0 && !c->layout_only() && (!q || !k || !v || !out)) return fail(FCG_EINVAL, "null tensor");
  if (c->desc.n_kv_heads > kNoAllocMaxKvHeads)
    return fail(FCG_EINVAL, "fcg_decode_noalloc supports at most " + std::to_string(kNoAllocMaxKvHeads) + " kv heads");
  std::vector<int32_t> pos;
  std::vector<std::pair<int32_t, int32_t>> new_pages;
  std::string msg;
  if (fcg_status st = c->plan.check_decode(layer, n_seqs, seqs, &pos, &new_pages, &msg)) return fail(st, msg);
  if (n_seqs == 0) return FCG_OK;
  const DecodePlan plan = plan_decode(c->desc, n_seqs, pos);
  const size_t need = (plan.part_o + plan.part_ml) * sizeof(float);
  if (need > kNoAllocPartBytes)
    return fail(FCG_ENOMEM, "this step needs " + std::to_string(need) + " bytes of split partials; the static scratch of "
                                "fcg_decode_noalloc holds " + std::to_string(kNoAllocPartBytes) + " (use fcg_decode)");
  if (!c->layout_only()) {
    HIP_TRY(hipSetDevice(c->device), "hipSetDevice");
    hipStream_t s = (hipStream_t)stream;
    void* base = nullptr;
    if (int rc = noalloc_scratch(s, &base)) return hip_fail((hipError_t)rc, "static scratch");
    c->plan.map_pages(new_pages);
    const std::vector<int32_t> np = decode_new_pages(c, n_seqs, seqs, pos, new_pages);
    float* po = reinterpret_cast<float*>(static_cast<char*>(base) + kNoAllocCountBytes);
    if (fcg_status st = launch_decode_groups(c, layer, n_seqs, seqs, pos, np, plan, q, k, v, out, po,
                                             po + plan.part_o, static_cast<int32_t*>(base), false, s))
      return st;
  } else {
    c->plan.map_pages(new_pages);
  }
  for (int32_t i = 0; i < n_seqs; ++i) {
    c->plan.mark(seqs[i], layer, pos[i]);
    if (positions_out) positions_out[i] = pos[i];
  }
  return FCG_OK;
}

}  // extern "C"
