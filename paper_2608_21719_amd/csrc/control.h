// Phase-aware frequency control (host only): the vote-commit DVFS daemon of
// §V (Alg. 1) and the per-epoch optimiser of §IV-C (eqs. dual, kkt-f,
// dcap-df, rank; App. B.1 eq. lagrangian).
#pragma once
#include <stdint.h>

#include <atomic>
#include <condition_variable>
#include <map>
#include <mutex>
#include <thread>
#include <vector>

#include "../../include/ps.h"

namespace ps {

class Dvfs {
 public:
  Dvfs(std::vector<int32_t> ladder, double under_w, double over_w, int32_t power_limit, int32_t f0,
       ps_dvfs_lock_fn lock, ps_dvfs_limit_fn limit, void* ctx);
  ~Dvfs();
  void vote(int64_t r, int32_t target, double weight);
  void retract(int64_t r);
  // One commit: the ladder frequency maximising the summed vote benefit;
  // lock only on change; power limit every tick. Returns the actuator's
  // first non-zero status (0 = all calls succeeded).
  int32_t tick(int32_t* f, int32_t* changed);
  bool start(int32_t period_ms);
  void stop();

 private:
  double score(int32_t f) const;  // callers hold mu_
  std::vector<int32_t> ladder_;
  double under_w_, over_w_;
  int32_t power_limit_, f_;
  ps_dvfs_lock_fn lock_;
  ps_dvfs_limit_fn limit_;
  void* ctx_;
  std::map<int64_t, std::pair<int32_t, double>> votes_;  // ordered by request id
  std::mutex mu_;
  std::thread th_;
  std::condition_variable cv_;
  bool stop_ = false, running_ = false;
};

// PSOpt on the relaxation; returns 0 when the cap is met (after projection),
// PS_E_CAPACITY when even the lowest admissible frequencies exceed it (out
// then holds that minimum-power point).
int psopt_solve(const ps_psopt_group* g, int n, double p_max, double f_min, double f_max, double dt,
                const int32_t* ladder, int n_ladder, ps_psopt_result* out, double* mu, double* p_relaxed,
                double* p_projected);

}  // namespace ps
