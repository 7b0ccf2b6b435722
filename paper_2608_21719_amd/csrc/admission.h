// Per-stage KV reservation and admission by observed lengths (host only).
//
// A stage pool reserves each request's KV in whole chunks of CS_i tokens,
// the stage's "KV chunk size" (§IV-A; the design-space table of §III-B lists
// 512 / 1024 / 2048). CS_i follows the lengths the stage actually produced:
// the mean of the last `window` completed requests' stage lengths, rounded up
// to a page and clamped (§IV-D, PSRoute admits by observation instead of
// predicting lengths). A request is admitted when a sequence slot is free and
// the free pages cover its context plus one chunk; a running sequence that
// outgrows its reservation takes further chunks, and when the pool cannot
// cover them the most recently admitted sequence is preempted (pages freed,
// request back to the caller's queue). Integer arithmetic throughout.
#pragma once
#include <stdint.h>

#include <deque>
#include <string>
#include <vector>

#include "kv_pool.h"

namespace ps {

class Admission {
 public:
  Admission(KvPool& pool, int32_t window, int32_t cs_initial, int32_t cs_min, int32_t cs_max);
  int32_t chunk_size() const;
  // *seq = admitted sequence id (ctx + CS_i tokens reserved), or -1 when no
  // slot or too few free pages; PS_E_CAPACITY if ctx + CS_i exceeds what a
  // sequence may ever hold. Nothing changes unless admitted.
  int admit(int32_t ctx, int32_t* seq, std::string& err);
  // Covers len + n_tok[i] for every listed sequence, preempting (freeing)
  // the most recently admitted sequences when pages run out; preempted ids
  // in preemption order. Validates everything before changing anything.
  int reserve_step(int32_t n, const int32_t* seqs, const int32_t* n_tok, int32_t cap, int32_t* preempted,
                   int32_t* n_preempted, std::string& err);
  // Records the request's stage length and frees its sequence.
  int finish(int32_t seq, int32_t stage_tokens, std::string& err);
  int32_t running() const;

 private:
  bool mine(int32_t s) const { return s >= 0 && s < (int32_t)order_.size() && order_[s] != 0; }
  void drop(int32_t s);
  KvPool& pool_;
  int32_t window_, cs_initial_, cs_min_, cs_max_;
  std::deque<int32_t> obs_;
  int64_t obs_sum_ = 0;
  std::vector<uint64_t> order_;  // admission counter per sequence id, 0 = not admitted here
  uint64_t counter_ = 0;
};

}  // namespace ps
