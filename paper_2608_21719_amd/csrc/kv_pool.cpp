#include "kv_pool.h"

#include <algorithm>

#include "../../include/ps.h"

namespace ps {

namespace {
// splitmix64 (Steele, Lea, Flood 2014): a tiny counter-based mixer used to
// shuffle the initial free list.
uint64_t splitmix64(uint64_t& state) {
  uint64_t z = (state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
}  // namespace

KvPool::KvPool(int32_t n_pages, int32_t max_seqs, int32_t max_pages_per_seq, uint64_t seed)
    : n_pages_(n_pages), max_seqs_(max_seqs), max_pages_per_seq_(max_pages_per_seq), seqs_(max_seqs) {
  // order[i] = i-th page handed out. Identity for seed 0, else Fisher-Yates.
  std::vector<int32_t> order(n_pages);
  for (int32_t i = 0; i < n_pages; ++i) order[i] = i;
  if (seed != 0) {
    uint64_t st = seed;
    for (int32_t i = n_pages - 1; i > 0; --i) {
      int32_t j = (int32_t)(splitmix64(st) % (uint64_t)(i + 1));
      std::swap(order[i], order[j]);
    }
  }
  free_.assign(order.rbegin(), order.rend());
}

int KvPool::check_open(int32_t s, std::string& err) const {
  if (s < 0 || s >= max_seqs_ || !seqs_[s].open) {
    err = "sequence " + std::to_string(s) + " is not open";
    return PS_E_INVALID;
  }
  return PS_OK;
}

int KvPool::open(int32_t* seq, std::string& err) {
  for (int32_t s = 0; s < max_seqs_; ++s) {
    if (!seqs_[s].open) {
      seqs_[s].open = true;
      seqs_[s].len = 0;
      seqs_[s].pages.clear();
      *seq = s;
      return PS_OK;
    }
  }
  err = "all " + std::to_string(max_seqs_) + " sequence slots are open";
  return PS_E_CAPACITY;
}

int KvPool::reserve(int32_t s, int32_t n_tokens, std::string& err) {
  if (int rc = check_open(s, err)) return rc;
  if (n_tokens < 0) {
    err = "negative reservation";
    return PS_E_INVALID;
  }
  KvSeq& q = seqs_[s];
  int64_t want_tokens = (int64_t)q.len + n_tokens;
  int64_t want_pages = (want_tokens + 15) / 16;
  int64_t have = (int64_t)q.pages.size();
  if (want_pages <= have) return PS_OK;
  if (want_pages > max_pages_per_seq_) {
    err = "sequence " + std::to_string(s) + " would need " + std::to_string(want_pages) +
          " pages, above max_pages_per_seq " + std::to_string(max_pages_per_seq_);
    return PS_E_CAPACITY;
  }
  int64_t need = want_pages - have;
  if (need > (int64_t)free_.size()) {
    err = "KV pool has " + std::to_string(free_.size()) + " free pages, " + std::to_string(need) +
          " needed";
    return PS_E_NO_PAGES;
  }
  for (int64_t i = 0; i < need; ++i) {
    q.pages.push_back(free_.back());
    free_.pop_back();
  }
  return PS_OK;
}

int KvPool::check_writable(int32_t s, int32_t n_tokens, std::string& err) const {
  if (int rc = check_open(s, err)) return rc;
  if (n_tokens < 0) {
    err = "negative token count";
    return PS_E_INVALID;
  }
  const KvSeq& q = seqs_[s];
  if ((int64_t)q.len + n_tokens > (int64_t)q.pages.size() * 16) {
    err = "sequence " + std::to_string(s) + ": writing " + std::to_string(n_tokens) +
          " tokens at length " + std::to_string(q.len) + " exceeds its reserved capacity " +
          std::to_string(q.pages.size() * 16);
    return PS_E_CAPACITY;
  }
  return PS_OK;
}

int KvPool::commit(int32_t n, const int32_t* seqs, const int32_t* n_tok, std::string& err) {
  if (n < 0 || (n > 0 && (!seqs || !n_tok))) {
    err = "bad commit arguments";
    return PS_E_INVALID;
  }
  for (int32_t i = 0; i < n; ++i) {
    if (int rc = check_writable(seqs[i], n_tok[i], err)) return rc;
    for (int32_t j = 0; j < i; ++j)
      if (seqs[j] == seqs[i]) {
        err = "sequence " + std::to_string(seqs[i]) + " listed twice";
        return PS_E_INVALID;
      }
  }
  for (int32_t i = 0; i < n; ++i) seqs_[seqs[i]].len += n_tok[i];
  if (n > 0) ++gen_;
  return PS_OK;
}

int KvPool::truncate(int32_t s, int32_t new_len, std::string& err) {
  if (int rc = check_open(s, err)) return rc;
  if (new_len < 0 || new_len > seqs_[s].len) {
    err = "truncate to " + std::to_string(new_len) + " outside [0, " + std::to_string(seqs_[s].len) + "]";
    return PS_E_INVALID;
  }
  seqs_[s].len = new_len;
  ++gen_;
  return PS_OK;
}

int KvPool::release(int32_t s, std::string& err) {
  if (int rc = check_open(s, err)) return rc;
  KvSeq& q = seqs_[s];
  for (auto it = q.pages.rbegin(); it != q.pages.rend(); ++it) free_.push_back(*it);
  q.pages.clear();
  q.len = 0;
  q.open = false;
  ++gen_;
  return PS_OK;
}

}  // namespace ps
