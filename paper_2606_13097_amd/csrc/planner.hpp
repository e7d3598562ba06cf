// Host-side layout planner of the composite cache: which positions of which
// sequence and layer are written, the page map of paged caches, and the
// validation of graft / prefill / decode requests.  Pure host code (no HIP):
// it decides, the kernels only move and compute.
//
// Placement follows module-level reuse (App. B.1; App. C.7): a grafted
// segment is a contiguous, order-preserving run of positions; fresh patch
// tokens take the positions the caller names (Sec. 4.2, Eq. 6).
#pragma once

#include <cstdint>
#include <set>
#include <string>
#include <utility>
#include <vector>

#include "fcg.h"

namespace fcg {

struct Span {
  int32_t seq, seg, dst, len, delta;
};

// A page whose values were mapped onto the library and that a truncation
// splits: its first `rows` rows must be copied from library token lib_tok ..
// into the cache page before new tokens follow them.
struct Unalias {
  int32_t seq, page, rows;
  int64_t lib_tok;
};

class Planner {
 public:
  // alias_v: pages that one grafted segment covers entirely read their values
  // from the library (paged caches only)
  Planner(int32_t n_layers, int32_t n_seqs, int32_t max_tokens, int32_t page_size, int32_t n_pages,
          bool alias_v = false);

  int32_t n_layers() const { return L_; }
  int32_t n_seqs() const { return S_; }
  int32_t max_tokens() const { return T_; }
  int32_t page_size() const { return P_; }
  int32_t n_pages() const { return NP_; }
  int32_t n_logical_pages() const { return NLP_; }
  bool alias_v() const { return AV_; }

  // Validation.  On success the returned status is FCG_OK and *new_pages holds
  // the (seq, logical page) pairs the call maps, in mapping order; on failure
  // *msg says why and nothing changes.
  fcg_status check_graft(const std::vector<Span>& spans, std::vector<std::pair<int32_t, int32_t>>* new_pages,
                         std::string* msg) const;
  fcg_status check_append(int32_t layer, int32_t n, const int32_t* seq, const int32_t* pos,
                          std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const;
  fcg_status check_decode(int32_t layer, int32_t n, const int32_t* seq, std::vector<int32_t>* pos_out,
                          std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const;

  // Commits (after a successful check).
  void map_pages(const std::vector<std::pair<int32_t, int32_t>>& new_pages);
  void mark_all_layers(int32_t seq, int32_t dst, int32_t len);
  // graft of len tokens at dst whose first token is library token lib_tok0:
  // with alias_v, the logical pages inside [dst, dst + len) map their values
  // onto the library
  void alias_pages(int32_t seq, int32_t dst, int32_t len, int64_t lib_tok0);
  void mark(int32_t seq, int32_t layer, int32_t pos);
  void reset(int32_t seq);
  // keep [0, pos) in every layer (the caller checked the range); a split
  // page mapped onto the library is appended to *unalias and unmapped
  void truncate(int32_t seq, int32_t pos, std::vector<Unalias>* unalias = nullptr);

  // Queries.
  bool written(int32_t seq, int32_t layer, int32_t pos) const;
  int32_t seq_len(int32_t seq, int32_t layer) const { return len_[idx(seq, layer)]; }
  int32_t count(int32_t seq, int32_t layer) const { return cnt_[idx(seq, layer)]; }
  const int32_t* page_row(int32_t seq) const { return page_table_.data() + (size_t)seq * NLP_; }
  int32_t page_of(int32_t seq, int32_t pos) const { return page_table_[(size_t)seq * NLP_ + pos / P_]; }
  // [NLP] library token of each logical page's first position, -1 = the page's own values
  const int32_t* alias_row(int32_t seq) const { return valias_.data() + (size_t)seq * NLP_; }

 private:
  size_t idx(int32_t seq, int32_t layer) const { return (size_t)seq * L_ + layer; }
  const uint64_t* bits(int32_t seq, int32_t layer) const { return bits_.data() + idx(seq, layer) * W_; }
  uint64_t* bits(int32_t seq, int32_t layer) { return bits_.data() + idx(seq, layer) * W_; }
  bool any_in_range(int32_t seq, int32_t layer, int32_t a, int32_t b) const;  // [a, b)
  int32_t count_below(int32_t seq, int32_t layer, int32_t b) const;           // written in [0, b)
  fcg_status collect_pages(const std::vector<std::pair<int32_t, int32_t>>& seq_lpage,
                           std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const;

  int32_t L_, S_, T_, P_, NP_, NLP_, W_;
  bool AV_;
  std::vector<uint64_t> bits_;       // [S][L][W] written bits
  std::vector<int32_t> len_, cnt_;   // [S][L]
  std::vector<int32_t> page_table_;  // [S][NLP], -1 = unmapped
  std::vector<int32_t> valias_;      // [S][NLP], library token or -1
  std::set<int32_t> free_;           // free physical pages, ascending
};

}  // namespace fcg
