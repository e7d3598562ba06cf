// Host-side layout planner (see planner.hpp).  Checks run in a fixed order:
// EINVAL, ERANGE, ESTATE, EOVERLAP, EHOLE, ENOMEM; the first failing class is
// reported and nothing is changed.
#include "planner.hpp"

#include <algorithm>
#include <cstdio>

namespace fcg {

static std::string fmt(const char* f, long long a = 0, long long b = 0, long long c = 0) {
  char buf[256];
  std::snprintf(buf, sizeof buf, f, a, b, c);
  return buf;
}

Planner::Planner(int32_t n_layers, int32_t n_seqs, int32_t max_tokens, int32_t page_size, int32_t n_pages,
                 bool alias_v)
    : L_(n_layers), S_(n_seqs), T_(max_tokens), P_(page_size), NP_(page_size ? n_pages : 0),
      NLP_(page_size ? (max_tokens + page_size - 1) / page_size : 0), W_((max_tokens + 63) / 64),
      AV_(alias_v && page_size != 0) {
  bits_.assign((size_t)S_ * L_ * W_, 0);
  len_.assign((size_t)S_ * L_, 0);
  cnt_.assign((size_t)S_ * L_, 0);
  page_table_.assign((size_t)S_ * NLP_, -1);
  valias_.assign((size_t)S_ * NLP_, -1);
  for (int32_t p = 0; p < NP_; ++p) free_.insert(free_.end(), p);
}

bool Planner::written(int32_t seq, int32_t layer, int32_t pos) const {
  return (bits(seq, layer)[pos >> 6] >> (pos & 63)) & 1u;
}

bool Planner::any_in_range(int32_t seq, int32_t layer, int32_t a, int32_t b) const {
  const uint64_t* w = bits(seq, layer);
  for (int32_t p = a; p < b;) {
    int32_t word = p >> 6, lo = p & 63;
    int32_t hi = std::min(64, lo + (b - p));
    uint64_t mask = (hi == 64 ? ~0ull : ((1ull << hi) - 1)) & ~((1ull << lo) - 1);
    if (w[word] & mask) return true;
    p += hi - lo;
  }
  return false;
}

int32_t Planner::count_below(int32_t seq, int32_t layer, int32_t b) const {
  const uint64_t* w = bits(seq, layer);
  int32_t c = 0, full = b >> 6;
  for (int32_t i = 0; i < full; ++i) c += __builtin_popcountll(w[i]);
  if (b & 63) c += __builtin_popcountll(w[full] & ((1ull << (b & 63)) - 1));
  return c;
}

fcg_status Planner::collect_pages(const std::vector<std::pair<int32_t, int32_t>>& seq_lpage,
                                  std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const {
  new_pages->clear();
  if (!P_) return FCG_OK;
  std::vector<std::pair<int32_t, int32_t>> v;
  for (auto& sl : seq_lpage)
    if (page_table_[(size_t)sl.first * NLP_ + sl.second] < 0) v.push_back(sl);
  std::sort(v.begin(), v.end());
  v.erase(std::unique(v.begin(), v.end()), v.end());
  if (v.size() > free_.size()) {
    *msg = fmt("%lld new pages needed, %lld free", (long long)v.size(), (long long)free_.size());
    return FCG_ENOMEM;
  }
  *new_pages = std::move(v);
  return FCG_OK;
}

fcg_status Planner::check_graft(const std::vector<Span>& spans,
                                std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const {
  for (const Span& s : spans) {
    if (s.seq < 0 || s.seq >= S_) { *msg = fmt("sequence %lld out of range", s.seq); return FCG_ERANGE; }
    if (s.dst < 0 || (int64_t)s.dst + s.len > T_) {
      *msg = fmt("span [%lld, %lld) outside the sequence", s.dst, (long long)s.dst + s.len);
      return FCG_ERANGE;
    }
  }
  // spans of one call must be disjoint per sequence
  std::vector<const Span*> order;
  for (const Span& s : spans) order.push_back(&s);
  std::sort(order.begin(), order.end(), [](const Span* a, const Span* b) {
    return a->seq != b->seq ? a->seq < b->seq : a->dst < b->dst;
  });
  for (size_t i = 1; i < order.size(); ++i)
    if (order[i]->seq == order[i - 1]->seq && order[i]->dst < order[i - 1]->dst + order[i - 1]->len) {
      *msg = fmt("spans of sequence %lld overlap at %lld", order[i]->seq, order[i]->dst);
      return FCG_EOVERLAP;
    }
  for (const Span& s : spans)
    for (int32_t l = 0; l < L_; ++l)
      if (s.len && any_in_range(s.seq, l, s.dst, s.dst + s.len)) {
        *msg = fmt("span at %lld of sequence %lld meets written positions (layer %lld)", s.dst, s.seq, l);
        return FCG_EOVERLAP;
      }
  std::vector<std::pair<int32_t, int32_t>> touched;
  if (P_)
    for (const Span& s : spans)
      for (int32_t lp = s.dst / P_; s.len && lp <= (s.dst + s.len - 1) / P_; ++lp) touched.push_back({s.seq, lp});
  return collect_pages(touched, new_pages, msg);
}

fcg_status Planner::check_append(int32_t layer, int32_t n, const int32_t* seq, const int32_t* pos,
                                 std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const {
  if (layer < 0 || layer >= L_) { *msg = fmt("layer %lld out of range", layer); return FCG_ERANGE; }
  for (int32_t t = 0; t < n; ++t) {
    if (seq[t] < 0 || seq[t] >= S_) { *msg = fmt("sequence %lld out of range", seq[t]); return FCG_ERANGE; }
    if (pos[t] < 0 || pos[t] >= T_) { *msg = fmt("position %lld out of range", pos[t]); return FCG_ERANGE; }
  }
  std::vector<std::pair<int32_t, int32_t>> sp(n);
  for (int32_t t = 0; t < n; ++t) sp[t] = {seq[t], pos[t]};
  std::sort(sp.begin(), sp.end());
  for (int32_t t = 0; t < n; ++t) {
    if ((t > 0 && sp[t] == sp[t - 1]) || written(sp[t].first, layer, sp[t].second)) {
      *msg = fmt("position %lld of sequence %lld given twice or already written", sp[t].second, sp[t].first);
      return FCG_EOVERLAP;
    }
  }
  // hole check per sequence: positions [0, top] all written once the call's tokens are in
  for (int32_t t = 0; t < n;) {
    int32_t s = sp[t].first, u = t;
    while (u < n && sp[u].first == s) ++u;
    int32_t top = sp[u - 1].second;
    if (count_below(s, layer, top + 1) + (u - t) != top + 1) {
      *msg = fmt("sequence %lld has unwritten positions below %lld (layer %lld)", s, top, layer);
      return FCG_EHOLE;
    }
    t = u;
  }
  std::vector<std::pair<int32_t, int32_t>> touched;
  if (P_)
    for (auto& x : sp) touched.push_back({x.first, x.second / P_});
  return collect_pages(touched, new_pages, msg);
}

fcg_status Planner::check_decode(int32_t layer, int32_t n, const int32_t* seq, std::vector<int32_t>* pos_out,
                                 std::vector<std::pair<int32_t, int32_t>>* new_pages, std::string* msg) const {
  std::vector<int32_t> s(seq, seq + n);
  std::sort(s.begin(), s.end());
  for (int32_t i = 1; i < n; ++i)
    if (s[i] == s[i - 1]) { *msg = fmt("sequence %lld given twice", s[i]); return FCG_EINVAL; }
  if (layer < 0 || layer >= L_) { *msg = fmt("layer %lld out of range", layer); return FCG_ERANGE; }
  for (int32_t i = 0; i < n; ++i)
    if (seq[i] < 0 || seq[i] >= S_) { *msg = fmt("sequence %lld out of range", seq[i]); return FCG_ERANGE; }
  for (int32_t i = 0; i < n; ++i)
    if (seq_len(seq[i], layer) >= T_) { *msg = fmt("sequence %lld is full", seq[i]); return FCG_ERANGE; }
  for (int32_t i = 0; i < n; ++i)
    if (seq_len(seq[i], layer) == 0) {
      *msg = fmt("sequence %lld has nothing written in layer %lld", seq[i], layer);
      return FCG_ESTATE;
    }
  for (int32_t i = 0; i < n; ++i)
    if (count(seq[i], layer) != seq_len(seq[i], layer)) {
      *msg = fmt("sequence %lld has a hole below %lld (layer %lld)", seq[i], seq_len(seq[i], layer), layer);
      return FCG_EHOLE;
    }
  pos_out->resize(n);
  std::vector<std::pair<int32_t, int32_t>> touched;
  for (int32_t i = 0; i < n; ++i) {
    (*pos_out)[i] = seq_len(seq[i], layer);
    if (P_) touched.push_back({seq[i], (*pos_out)[i] / P_});
  }
  return collect_pages(touched, new_pages, msg);
}

void Planner::map_pages(const std::vector<std::pair<int32_t, int32_t>>& new_pages) {
  for (auto& sl : new_pages) {
    int32_t p = *free_.begin();
    free_.erase(free_.begin());
    page_table_[(size_t)sl.first * NLP_ + sl.second] = p;
  }
}

void Planner::mark(int32_t seq, int32_t layer, int32_t pos) {
  uint64_t& w = bits(seq, layer)[pos >> 6];
  uint64_t b = 1ull << (pos & 63);
  if (!(w & b)) {
    w |= b;
    ++cnt_[idx(seq, layer)];
    len_[idx(seq, layer)] = std::max(len_[idx(seq, layer)], pos + 1);
  }
}

void Planner::mark_all_layers(int32_t seq, int32_t dst, int32_t len) {
  for (int32_t l = 0; l < L_; ++l)
    for (int32_t p = dst; p < dst + len; ++p) mark(seq, l, p);
}

void Planner::alias_pages(int32_t seq, int32_t dst, int32_t len, int64_t lib_tok0) {
  if (!AV_) return;
  for (int32_t lp = (dst + P_ - 1) / P_; (lp + 1) * P_ <= dst + len; ++lp)
    valias_[(size_t)seq * NLP_ + lp] = (int32_t)(lib_tok0 + (int64_t)lp * P_ - dst);
}

void Planner::reset(int32_t seq) {
  std::fill(valias_.begin() + (size_t)seq * NLP_, valias_.begin() + (size_t)(seq + 1) * NLP_, -1);
  for (int32_t l = 0; l < L_; ++l) {
    std::fill(bits(seq, l), bits(seq, l) + W_, 0ull);
    len_[idx(seq, l)] = 0;
    cnt_[idx(seq, l)] = 0;
  }
  for (int32_t lp = 0; lp < NLP_; ++lp) {
    int32_t& e = page_table_[(size_t)seq * NLP_ + lp];
    if (e >= 0) { free_.insert(e); e = -1; }
  }
}

void Planner::truncate(int32_t seq, int32_t pos, std::vector<Unalias>* unalias) {
  if (P_ && pos % P_ && pos < T_) {
    int32_t& a = valias_[(size_t)seq * NLP_ + pos / P_];
    if (a >= 0) {
      if (unalias) unalias->push_back(Unalias{seq, page_table_[(size_t)seq * NLP_ + pos / P_], pos % P_, a});
      a = -1;
    }
  }
  for (int32_t l = 0; l < L_; ++l) {
    uint64_t* b = bits(seq, l);
    for (int32_t wi = 0; wi < W_; ++wi) {
      const int32_t lo = wi * 64;
      if (lo >= pos) b[wi] = 0;
      else if (lo + 64 > pos) b[wi] &= (1ull << (pos - lo)) - 1;
    }
    int32_t cnt = 0, len = 0;
    for (int32_t wi = 0; wi < W_; ++wi)
      if (b[wi]) {
        cnt += __builtin_popcountll(b[wi]);
        len = wi * 64 + 64 - __builtin_clzll(b[wi]);
      }
    cnt_[idx(seq, l)] = cnt;
    len_[idx(seq, l)] = len;
  }
  if (P_)
    for (int32_t lp = (pos + P_ - 1) / P_; lp < NLP_; ++lp) {
      int32_t& e = page_table_[(size_t)seq * NLP_ + lp];
      if (e >= 0) { free_.insert(e); e = -1; }
      valias_[(size_t)seq * NLP_ + lp] = -1;
    }
}

}  // namespace fcg
