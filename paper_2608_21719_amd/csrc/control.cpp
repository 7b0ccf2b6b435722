#include "control.h"

#include <algorithm>
#include <chrono>
#include <cmath>

namespace ps {

// ------------------------------------------------------------- vote-commit
Dvfs::Dvfs(std::vector<int32_t> ladder, double under_w, double over_w, int32_t power_limit, int32_t f0,
           ps_dvfs_lock_fn lock, ps_dvfs_limit_fn limit, void* ctx)
    : ladder_(std::move(ladder)), under_w_(under_w), over_w_(over_w), power_limit_(power_limit), f_(f0),
      lock_(lock), limit_(limit), ctx_(ctx) {}

Dvfs::~Dvfs() { stop(); }

void Dvfs::vote(int64_t r, int32_t target, double weight) {
  std::lock_guard<std::mutex> g(mu_);
  votes_[r] = {target, weight};
}

void Dvfs::retract(int64_t r) {
  std::lock_guard<std::mutex> g(mu_);
  votes_.erase(r);
}

// b(f; f*) = -(under_w * max(0, f* - f) + over_w * max(0, f - f*)), weighted
// by the vote's class weight, summed in ascending request id
double Dvfs::score(int32_t f) const {
  double s = 0.0;
  for (const auto& kv : votes_) {
    const double t = kv.second.first, w = kv.second.second;
    s = s - w * (under_w_ * std::max(0.0, t - f) + over_w_ * std::max(0.0, f - t));
  }
  return s;
}

int32_t Dvfs::tick(int32_t* f_out, int32_t* changed) {
  std::lock_guard<std::mutex> g(mu_);
  int32_t best = ladder_[0];
  double best_s = score(best);
  for (size_t i = 1; i < ladder_.size(); ++i) {
    const double s = score(ladder_[i]);
    if (s > best_s) best = ladder_[i], best_s = s;  // ties keep the lower frequency
  }
  int32_t rc = 0;
  const bool ch = best != f_;
  if (ch) {
    rc = lock_ ? lock_(ctx_, best) : 0;
    f_ = best;
  }
  const int32_t rl = limit_ ? limit_(ctx_, power_limit_) : 0;
  if (!rc) rc = rl;
  if (f_out) *f_out = best;
  if (changed) *changed = ch;
  return rc;
}

bool Dvfs::start(int32_t period_ms) {
  {
    std::lock_guard<std::mutex> g(mu_);
    if (running_) return false;
    running_ = true;
    stop_ = false;
  }
  th_ = std::thread([this, period_ms] {
    std::unique_lock<std::mutex> lk(mu_);
    while (!stop_) {
      lk.unlock();
      tick(nullptr, nullptr);
      lk.lock();
      cv_.wait_for(lk, std::chrono::milliseconds(period_ms), [this] { return stop_; });
    }
  });
  return true;
}

void Dvfs::stop() {
  {
    std::lock_guard<std::mutex> g(mu_);
    if (!running_) return;
    stop_ = true;
  }
  cv_.notify_all();
  th_.join();
  std::lock_guard<std::mutex> g(mu_);
  running_ = false;
}

// ------------------------------------------------------------------ PSOpt
namespace {
constexpr double kInvSqrt2Pi = 0.39894228040143267794;
double pdf(double x) { return kInvSqrt2Pi * std::exp(-0.5 * x * x); }
double cdf(double x) { return 0.5 * std::erfc(-x / std::sqrt(2.0)); }

struct Group {
  const ps_psopt_group& g;
  double f_max;
  double cap(double f) const { return g.c * std::pow(g.k, g.nu) * (1.0 - g.gamma + g.gamma * f / f_max); }
  double dcap() const { return g.c * std::pow(g.k, g.nu) * g.gamma / f_max; }  // eq. dcap-df
  double pw(double f) const { return g.k * (g.c2 * f * f * f + g.c1 * f + g.c0); }
  double dpw(double f) const { return g.k * (3.0 * g.c2 * f * f + g.c1); }
  // I(C) = (1/lambda) int_C^C0 p(l)(l - C) dl for l ~ N(lambda, sigma), in closed form
  double impact(double C) const {
    const double C0 = cap(f_max);
    if (C >= C0) return 0.0;
    const double a = (C - g.lam) / g.sigma, b = (C0 - g.lam) / g.sigma;
    return (g.sigma * (pdf(a) - pdf(b)) + (g.lam - C) * (cdf(b) - cdf(a))) / g.lam;
  }
  double dimpact(double C) const {  // dI/dC (<= 0)
    const double C0 = cap(f_max);
    if (C >= C0) return 0.0;
    return -(cdf((C0 - g.lam) / g.sigma) - cdf((C - g.lam) / g.sigma)) / g.lam;
  }
};

template <typename F>
double bisect_increasing(F fn, double lo, double hi) {  // root of an increasing fn on [lo, hi]
  for (int it = 0; it < 200 && hi - lo > 1e-12 * std::max(1.0, std::fabs(hi)); ++it) {
    const double mid = 0.5 * (lo + hi);
    (fn(mid) < 0 ? lo : hi) = mid;
  }
  return 0.5 * (lo + hi);
}

// frequency of one group at power multiplier mu: frequency stationarity
// (eq. kkt-f) (dt + mu) dP/df = -(w + eta) dI/dC dC/df with eta = 0, then
// raised to the lowest frequency meeting the impact bound
void group_at(const Group& G, double mu, double dt, double f_min, double f_max, double* f, double* f_bound) {
  const auto& g = G.g;
  auto stat = [&](double x) { return (dt + mu) * G.dpw(x) + g.w * G.dimpact(G.cap(x)) * G.dcap(); };
  double fu;
  if (stat(f_min) >= 0) fu = f_min;
  else if (stat(f_max) <= 0) fu = f_max;
  else fu = bisect_increasing(stat, f_min, f_max);
  double fb;
  auto excess = [&](double x) { return g.delta - G.impact(G.cap(x)); };  // increasing in f
  if (excess(f_min) >= 0) fb = f_min;
  else fb = bisect_increasing(excess, f_min, f_max);
  *f_bound = fb;
  *f = std::max(fu, fb);
}
}  // namespace

int psopt_solve(const ps_psopt_group* gs, int n, double p_max, double f_min, double f_max, double dt,
                const int32_t* ladder, int n_ladder, ps_psopt_result* out, double* mu_out, double* p_relaxed,
                double* p_projected) {
  std::vector<Group> G;
  for (int i = 0; i < n; ++i) G.push_back(Group{gs[i], f_max});
  std::vector<double> f(n), fb(n);
  auto total = [&](double mu) {
    double p = 0;
    for (int i = 0; i < n; ++i) {
      group_at(G[i], mu, dt, f_min, f_max, &f[i], &fb[i]);
      p += G[i].pw(f[i]);
    }
    return p;
  };
  double mu = 0.0;
  bool feasible = true;
  if (total(0.0) > p_max) {
    double hi = 1e-12;
    while (total(hi) > p_max && hi < 1e30) hi *= 4.0;
    if (total(hi) > p_max) {
      feasible = false;
      mu = hi;
    } else {
      double lo = 0.0;
      for (int it = 0; it < 300 && hi - lo > 1e-15 * hi; ++it) {
        const double mid = 0.5 * (lo + hi);
        (total(mid) > p_max ? lo : hi) = mid;
      }
      mu = hi;  // the feasible side
    }
  }
  double pr = total(mu);
  // multipliers and ranking keys at the relaxed optimum
  for (int i = 0; i < n; ++i) {
    const auto& g = gs[i];
    const double dI = G[i].dimpact(G[i].cap(f[i]));
    double eta = 0.0;
    if (f[i] == fb[i] && f[i] > f_min && dI < 0 && G[i].dcap() > 0)
      eta = std::max(0.0, -(dt + mu) * G[i].dpw(f[i]) / (dI * G[i].dcap()) - g.w);
    out[i].f = f[i];
    out[i].eta = eta;
    out[i].impact = G[i].impact(G[i].cap(f[i]));
    out[i].rank = (g.w + eta) * std::fabs(dI) * G[i].dcap() / G[i].dpw(f[i]);  // eq. rank
  }
  // projection onto the DVFS ladder: round up (keeps every impact bound),
  // then lower frequencies one step at a time in ascending rank (the
  // degradation ordering) while the cap is exceeded and the bound allows
  std::vector<int> step(n);
  auto up = [&](double x) {
    int s = 0;
    while (s < n_ladder - 1 && ladder[s] < x - 1e-9) ++s;
    return s;
  };
  std::vector<int> floor_step(n);
  for (int i = 0; i < n; ++i) {
    step[i] = up(f[i]);
    floor_step[i] = up(fb[i]);
  }
  auto proj_power = [&]() {
    double p = 0;
    for (int i = 0; i < n; ++i) p += G[i].pw(ladder[step[i]]);
    return p;
  };
  std::vector<int> order(n);
  for (int i = 0; i < n; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return out[a].rank < out[b].rank; });
  bool moved = true;
  while (proj_power() > p_max && moved) {
    moved = false;
    for (int i : order)
      if (step[i] > floor_step[i]) {
        --step[i];
        moved = true;
        break;
      }
  }
  for (int i = 0; i < n; ++i) out[i].f_step = ladder[step[i]];
  if (mu_out) *mu_out = mu;
  if (p_relaxed) *p_relaxed = pr;
  const double pp = proj_power();
  if (p_projected) *p_projected = pp;
  return (feasible && pp <= p_max * (1 + 1e-12)) ? 0 : PS_E_CAPACITY;
}

}  // namespace ps
