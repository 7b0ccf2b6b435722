// Host-only parts of libps under AddressSanitizer and UBSan: the KV page
// pool metadata, the admission scheduler, the DVFS daemon and the PSOpt
// solver, driven through seeded random sequences of calls (valid and
// invalid). Built and run by tests/test_host_sanitize.py with g++; exits
// non-zero on any failed check, and the sanitizers abort on any memory or
// undefined-behaviour error.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <string>
#include <vector>

#include "../paper_2608_21719_amd/csrc/admission.h"
#include "../paper_2608_21719_amd/csrc/control.h"
#include "../paper_2608_21719_amd/csrc/kv_pool.h"

#define CHECK(c)                                               \
  do {                                                         \
    if (!(c)) {                                                \
      std::fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      std::exit(1);                                            \
    }                                                          \
  } while (0)

static int lock_calls = 0;
static int32_t fake_lock(void*, int32_t) { return ++lock_calls, 0; }
static int32_t fake_limit(void*, int32_t) { return 0; }

int main() {
  std::mt19937_64 rng(12345);
  std::string e;
  // pool: random reserve / commit / truncate / release, invariants checked
  for (int round = 0; round < 20; ++round) {
    const int n_pages = 64 + (int)(rng() % 64), max_seqs = 8, max_pages = 32;
    ps::KvPool pool(n_pages, max_seqs, max_pages, rng());
    for (int op = 0; op < 3000; ++op) {
      int32_t s = (int32_t)(rng() % (max_seqs + 2)) - 1;  // includes invalid ids
      int32_t n = (int32_t)(rng() % 80) - 5;
      switch (rng() % 5) {
        case 0: { int32_t id; pool.open(&id, e); break; }
        case 1: pool.reserve(s, n, e); break;
        case 2: pool.commit(1, &s, &n, e); break;
        case 3: pool.truncate(s, n, e); break;
        case 4: pool.release(s, e); break;
      }
      int64_t used = 0;
      for (int q = 0; q < max_seqs; ++q) {
        used += (int64_t)pool.seq(q).pages.size();
        if (pool.seq(q).open) CHECK(pool.seq(q).len <= (int32_t)pool.seq(q).pages.size() * 16);
      }
      CHECK(used + pool.free_pages() == n_pages);
    }
  }
  // admission: random admissions, steps, completions
  for (int round = 0; round < 10; ++round) {
    ps::KvPool pool(200, 16, 64, rng());
    ps::Admission adm(pool, 4, 64, 16, 512);
    std::vector<int32_t> running;
    std::vector<int32_t> pre(16);
    for (int step = 0; step < 3000; ++step) {
      int32_t s;
      if (adm.admit((int32_t)(rng() % 200), &s, e) == 0 && s >= 0) running.push_back(s);
      std::vector<int32_t> ones(running.size(), 1);
      int32_t np = 0;
      int rc = adm.reserve_step((int32_t)running.size(), running.data(), ones.data(), 16, pre.data(), &np, e);
      if (rc == 0) {
        for (int i = 0; i < np; ++i)
          for (size_t j = 0; j < running.size(); ++j)
            if (running[j] == pre[i]) { running.erase(running.begin() + j); break; }
        std::vector<int32_t> one(running.size(), 1);
        if (!running.empty()) CHECK(pool.commit((int32_t)running.size(), running.data(), one.data(), e) == 0);
      } else {
        // a sequence outgrew the pool's limit: finish it
        for (int32_t q : running) adm.finish(q, pool.seq(q).len, e);
        running.clear();
      }
      if (!running.empty() && rng() % 7 == 0) {
        const size_t j = rng() % running.size();
        CHECK(adm.finish(running[j], pool.seq(running[j]).len, e) == 0);
        running.erase(running.begin() + j);
      }
      CHECK(adm.chunk_size() >= 16 && adm.chunk_size() <= 512);
    }
  }
  // daemon: votes, retracts, ticks; then the background thread
  {
    std::vector<int32_t> ladder = {800, 1200, 1600, 2000, 2400};
    ps::Dvfs d(ladder, 4.0, 1.0, 1400, 2400, fake_lock, fake_limit, nullptr);
    for (int i = 0; i < 5000; ++i) {
      if (rng() % 2) d.vote((int64_t)(rng() % 100), (int32_t)(400 + rng() % 2400), 1.0 + (double)(rng() % 100));
      else d.retract((int64_t)(rng() % 100));
      if (i % 10 == 0) { int32_t f, ch; CHECK(d.tick(&f, &ch) == 0); }
    }
    CHECK(d.start(1));
    for (int i = 0; i < 2000; ++i) d.vote((int64_t)(rng() % 100), (int32_t)(400 + rng() % 2400), 2.0);
    d.stop();
  }
  // solver: random groups, including unreachable caps
  for (int round = 0; round < 30; ++round) {
    std::vector<ps_psopt_group> g(9);
    for (auto& x : g) {
      x.w = 1 + (double)(rng() % 100); x.delta = 0.01 * (1 + rng() % 50); x.k = 1 + (double)(rng() % 8);
      x.nu = 0.9; x.c = 1 + (double)(rng() % 10); x.gamma = (double)(rng() % 101) / 100.0;
      x.lam = 0.8 * x.c * x.k; x.sigma = 0.1 * x.lam + 0.01; x.c2 = 6e-8; x.c1 = 0.1; x.c0 = 300;
    }
    std::vector<int32_t> ladder;
    for (int f = 800; f <= 2400; f += 100) ladder.push_back(f);
    std::vector<ps_psopt_result> out(9);
    double mu, pr, pp;
    const double cap = 500.0 * (1 + rng() % 60);
    int rc = ps::psopt_solve(g.data(), 9, cap, 800, 2400, 0.0, ladder.data(), (int)ladder.size(), out.data(), &mu,
                             &pr, &pp);
    CHECK(rc == 0 || rc == PS_E_CAPACITY);
    for (auto& r : out) CHECK(r.f >= 800 - 1e-9 && r.f <= 2400 + 1e-9 && r.f_step >= 800 && r.f_step <= 2400);
  }
  std::printf("host sanitize ok (%d clock locks)\n", lock_calls);
  return 0;
}
