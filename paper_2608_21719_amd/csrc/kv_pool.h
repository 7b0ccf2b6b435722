// Host-side metadata of the paged KV cache: free list, per-sequence page
// lists, committed lengths and reservations. No device calls.
//
// The per-request KV reservation in tokens is the "KV chunk size" CS_i of
// the paper's design (§IV-A, and the PSRoute admission of §IV-D): a
// sequence reserves capacity up front and pages are taken from the pool as
// the reservation grows. Every mutating call validates fully before changing
// anything, so a failed call leaves the pool exactly as it was.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

namespace ps {

struct KvSeq {
  bool open = false;
  int32_t len = 0;               // committed tokens
  std::vector<int32_t> pages;    // logical page i -> physical page id
};

class KvPool {
 public:
  KvPool(int32_t n_pages, int32_t max_seqs, int32_t max_pages_per_seq, uint64_t seed);

  // All return 0 on success or a PS_E_* code with `err` filled in.
  int open(int32_t* seq, std::string& err);
  int reserve(int32_t seq, int32_t n_tokens, std::string& err);
  int check_writable(int32_t seq, int32_t n_tokens, std::string& err) const;
  int commit(int32_t n, const int32_t* seqs, const int32_t* n_tok, std::string& err);
  int truncate(int32_t seq, int32_t new_len, std::string& err);
  int release(int32_t seq, std::string& err);
  int check_open(int32_t seq, std::string& err) const;

  const KvSeq& seq(int32_t s) const { return seqs_[s]; }
  int32_t capacity(int32_t s) const { return (int32_t)seqs_[s].pages.size() * 16; }
  int32_t free_pages() const { return (int32_t)free_.size(); }
  int32_t n_pages() const { return n_pages_; }
  int32_t max_seqs() const { return max_seqs_; }
  int32_t max_pages_per_seq() const { return max_pages_per_seq_; }
  // bumped by every change to a committed length or a page list that a
  // planned launch may have captured (commit, truncate, release)
  uint64_t generation() const { return gen_; }

 private:
  uint64_t gen_ = 0;
  int32_t n_pages_, max_seqs_, max_pages_per_seq_;
  std::vector<int32_t> free_;  // stack: back() is handed out next
  std::vector<KvSeq> seqs_;
};

}  // namespace ps
