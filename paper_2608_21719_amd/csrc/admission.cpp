#include "admission.h"

#include <algorithm>

#include "../../include/ps.h"

namespace ps {

namespace {
constexpr int32_t kPage = 16;
int64_t pages_for(int64_t tokens) { return (tokens + kPage - 1) / kPage; }
}  // namespace

Admission::Admission(KvPool& pool, int32_t window, int32_t cs_initial, int32_t cs_min, int32_t cs_max)
    : pool_(pool), window_(window), cs_initial_(cs_initial), cs_min_(cs_min), cs_max_(cs_max),
      order_(pool.max_seqs(), 0) {}

int32_t Admission::chunk_size() const {
  int64_t cs = cs_initial_;
  if (!obs_.empty()) {
    const int64_t n = (int64_t)obs_.size();
    cs = kPage * ((obs_sum_ + kPage * n - 1) / (kPage * n));  // the mean, rounded up to a page
  }
  return (int32_t)std::min<int64_t>(std::max<int64_t>(cs, cs_min_), cs_max_);
}

int32_t Admission::running() const {
  return (int32_t)std::count_if(order_.begin(), order_.end(), [](uint64_t o) { return o != 0; });
}

int Admission::admit(int32_t ctx, int32_t* seq, std::string& err) {
  *seq = -1;
  if (ctx < 0) {
    err = "negative context";
    return PS_E_INVALID;
  }
  const int64_t want = pages_for((int64_t)ctx + chunk_size());
  if (want > pool_.max_pages_per_seq()) {
    err = "a request of " + std::to_string(ctx) + " context tokens plus one chunk exceeds max_pages_per_seq";
    return PS_E_CAPACITY;
  }
  if (want > pool_.free_pages()) return PS_OK;
  int32_t s;
  std::string e;
  if (pool_.open(&s, e) != PS_OK) return PS_OK;  // no free sequence slot
  if (int rc = pool_.reserve(s, (int32_t)(want * kPage), e)) {  // cannot fail: pages and limit checked
    std::string e2;
    pool_.release(s, e2);
    err = e;
    return rc;
  }
  order_[s] = ++counter_;
  *seq = s;
  return PS_OK;
}

void Admission::drop(int32_t s) {
  std::string e;
  pool_.release(s, e);
  order_[s] = 0;
}

int Admission::reserve_step(int32_t n, const int32_t* seqs, const int32_t* n_tok, int32_t cap, int32_t* preempted,
                            int32_t* n_preempted, std::string& err) {
  if (n < 0 || (n > 0 && (!seqs || !n_tok)) || !n_preempted || (!preempted && cap > 0)) {
    err = "bad arguments";
    return PS_E_INVALID;
  }
  if (cap < pool_.max_seqs()) {
    err = "the preempted buffer must hold max_seqs ids";
    return PS_E_INVALID;
  }
  const int64_t limit = (int64_t)pool_.max_pages_per_seq() * kPage;
  for (int32_t i = 0; i < n; ++i) {
    if (!mine(seqs[i])) {
      err = "sequence " + std::to_string(seqs[i]) + " was not admitted by this scheduler";
      return PS_E_INVALID;
    }
    if (n_tok[i] < 0) {
      err = "negative token count";
      return PS_E_INVALID;
    }
    for (int32_t j = 0; j < i; ++j)
      if (seqs[j] == seqs[i]) {
        err = "sequence listed twice";
        return PS_E_INVALID;
      }
    if ((int64_t)pool_.seq(seqs[i]).len + n_tok[i] > limit) {
      err = "sequence " + std::to_string(seqs[i]) + " outgrows max_pages_per_seq";
      return PS_E_CAPACITY;
    }
  }
  *n_preempted = 0;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = seqs[i];
    if (!mine(s)) continue;  // preempted earlier in this call
    const int64_t need = (int64_t)pool_.seq(s).len + n_tok[i];
    const int64_t have = (int64_t)pool_.seq(s).pages.size();
    if (need <= have * kPage) continue;
    const int64_t cs = chunk_size();
    const int64_t chunks = (need - have * kPage + cs - 1) / cs;
    const int64_t want = std::min<int64_t>(pages_for(have * kPage + chunks * cs), pool_.max_pages_per_seq());
    const int64_t extra = want - have;
    while (extra > pool_.free_pages()) {
      int32_t victim = -1;
      for (int32_t v = 0; v < (int32_t)order_.size(); ++v)
        if (order_[v] && (victim < 0 || order_[v] > order_[victim])) victim = v;
      drop(victim);
      preempted[(*n_preempted)++] = victim;
      if (victim == s) break;
    }
    if (!mine(s)) continue;
    std::string e;
    if (int rc = pool_.reserve(s, (int32_t)(want * kPage - pool_.seq(s).len), e)) {  // cannot fail
      err = e;
      return rc;
    }
  }
  return PS_OK;
}

int Admission::finish(int32_t seq, int32_t stage_tokens, std::string& err) {
  if (!mine(seq)) {
    err = "sequence " + std::to_string(seq) + " was not admitted by this scheduler";
    return PS_E_INVALID;
  }
  if (stage_tokens < 0) {
    err = "negative stage length";
    return PS_E_INVALID;
  }
  obs_.push_back(stage_tokens);
  obs_sum_ += stage_tokens;
  if ((int32_t)obs_.size() > window_) {
    obs_sum_ -= obs_.front();
    obs_.pop_front();
  }
  drop(seq);
  return PS_OK;
}

}  // namespace ps
