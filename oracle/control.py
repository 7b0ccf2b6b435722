"""Phase-aware frequency control: plain models of the vote-commit daemon and
of the per-epoch optimisation it serves.

TEST INFRASTRUCTURE ONLY: never imported by the product path.

1. Vote-commit DVFS (§V "How is GPU frequency actually set", Alg. 1). Each
   request entering a stage on a GPU registers a vote (target frequency f*,
   SLO-class weight w); leaving removes it. Every tick the daemon picks, over
   the DVFS ladder F, the frequency maximising the weighted sum of b(f; f*),
   where b penalises running below a vote's target (SLO risk) and above it
   (wasted power); it locks the clock only when the choice changed, and
   reasserts the power limit every tick. Readings (the paper names b's two
   penalties but not its form):
     b(f; f*) = -(alpha * max(0, f* - f) + beta * max(0, f - f*)),
     alpha > beta (a missed SLO costs more than a wasted watt);
   ties go to the lowest frequency; with no votes every f scores 0, so the
   lowest ladder frequency is chosen. Sums run over votes in ascending
   request id, left to right, in float64.

2. PSOpt (§IV-C "Joint formulation", eq. dual; App. B.1 eq. lagrangian).
   For each stage-class group i with k_i GPUs at frequency f_i:
     capacity  C_i(f) = c_i k_i^nu_i (1 - gamma_i + gamma_i f / f_max)
               (its frequency slope is c_i k_i^nu_i gamma_i / f_max, eq.
               dcap-df: proportional to the compute-bound fraction);
     power     k_i P_i(f), P_i(f) = c2_i f^3 + c1_i f + c0_i (§IV-C);
     impact    I_i(C) = (1 / lambda_i) * integral_C^C0 p_i(l) (l - C) dl
               (§IV-B), with the arrival rate l ~ Normal(lambda_i, sigma_i)
               and C0 the capacity at f_max (readings);
   minimise sum_i w_i I_i(C_i(f_i)) + dt * sum_i k_i P_i(f_i)
   subject to sum_i k_i P_i(f_i) <= p_max, I_i <= delta_i,
   f_min <= f_i <= f_max, with the GPU counts k_i given (the paper also
   relaxes k; here k is an input). This model solves the relaxation with a
   general-purpose constrained optimiser (scipy SLSQP) on an impact computed
   by numerical quadrature, independently of the closed form and the
   KKT/bisection route of the library.
   The ranking key of eq. rank, R_i = (w_i + eta_i) |dI_i/dC_i| gamma_i
   k_i^(nu_i - 1) / (f_max (3 c2_i f_i^2 + c1_i)), impact per watt
   reclaimed, carries the capacity scale c_i (the printed form takes a unit
   per-GPU capacity).
"""
import math

import numpy as np


# --------------------------------------------------------------- vote-commit
class DvfsModel:
    def __init__(self, ladder, alpha: float, beta: float, power_limit: int, f0: int):
        self.ladder = sorted(ladder)
        self.alpha, self.beta = alpha, beta
        self.power_limit = power_limit
        self.f = f0
        self.votes = {}
        self.actions = []   # ("lock", f) and ("limit", watts), in order

    def vote(self, r: int, target: int, weight: float):
        self.votes[r] = (target, weight)

    def retract(self, r: int):
        self.votes.pop(r, None)

    def score(self, f: int) -> float:
        s = 0.0
        for r in sorted(self.votes):
            t, w = self.votes[r]
            s = s - w * (self.alpha * max(0, t - f) + self.beta * max(0, f - t))
        return s

    def tick(self):
        best, best_s = None, None
        for f in self.ladder:
            sc = self.score(f)
            if best is None or sc > best_s:
                best, best_s = f, sc
        changed = best != self.f
        if changed:
            self.actions.append(("lock", best))
            self.f = best
        self.actions.append(("limit", self.power_limit))
        return best, changed


# --------------------------------------------------------------- PSOpt
def capacity(g: dict, f: float) -> float:
    return g["c"] * g["k"] ** g["nu"] * (1.0 - g["gamma"] + g["gamma"] * f / g["f_max"])


def power(g: dict, f: float) -> float:
    return g["k"] * (g["c2"] * f ** 3 + g["c1"] * f + g["c0"])


def impact(g: dict, C: float) -> float:
    """(1/lambda) * integral_C^C0 p(l) (l - C) dl by adaptive quadrature."""
    from scipy import integrate
    C0 = capacity(g, g["f_max"])
    if C >= C0:
        return 0.0
    lam, sig = g["lam"], g["sigma"]

    def p(x):
        return math.exp(-0.5 * ((x - lam) / sig) ** 2) / (sig * math.sqrt(2 * math.pi))
    pts = [lam] if C < lam < C0 else None   # the density's peak, so a narrow one is not stepped over
    val, _ = integrate.quad(lambda x: p(x) * (x - C), C, C0, epsabs=1e-13, epsrel=1e-11, limit=200, points=pts)
    return val / lam


def solve(groups, p_max: float, f_min: float, f_max: float, dt: float = 0.0):
    """The relaxed problem by SLSQP on x = f / f_max from several starting
    points; the best feasible optimum (or None if none is feasible)."""
    from scipy.optimize import minimize
    n = len(groups)
    scale = max(power(g, f_max) for g in groups)
    wsum = sum(g["w"] for g in groups)

    def fs(x):
        return np.asarray(x) * f_max

    def obj(x):
        return (sum(g["w"] * impact(g, capacity(g, fi)) for g, fi in zip(groups, fs(x))) +
                dt * sum(power(g, fi) for g, fi in zip(groups, fs(x)))) / wsum

    def cap_slack(x):
        return (p_max - sum(power(g, fi) for g, fi in zip(groups, fs(x)))) / scale
    cons = [{"type": "ineq", "fun": cap_slack}]
    for i, g in enumerate(groups):
        cons.append({"type": "ineq", "fun": lambda x, i=i, g=g: g["delta"] - impact(g, capacity(g, x[i] * f_max))})
    lo = f_min / f_max
    best = None
    for start in (0.5 * (lo + 1.0), 0.9, 1.0, lo + 0.1 * (1.0 - lo)):
        res = minimize(obj, np.full(n, start), method="SLSQP", bounds=[(lo, 1.0)] * n, constraints=cons,
                       options={"ftol": 1e-15, "maxiter": 1000})
        feasible = all(c["fun"](res.x) >= -1e-9 for c in cons)
        if feasible and (best is None or res.fun < best.fun):
            best = res
    return None if best is None else fs(best.x)


def objective(groups, f, dt: float = 0.0) -> float:
    return sum(g["w"] * impact(g, capacity(g, fi)) for g, fi in zip(groups, f)) + \
        dt * sum(power(g, fi) for g, fi in zip(groups, f))


def rank_key(g: dict, f: float, eta: float, dI_dC: float) -> float:
    """Eq. rank: impact incurred per watt reclaimed, (w + eta) |dI/dC| dC/df
    over the group's dP/df. The printed form takes a unit per-GPU capacity;
    with capacity scale c it carries the factor c."""
    return (g["w"] + eta) * abs(dI_dC) * g["c"] * g["gamma"] * g["k"] ** (g["nu"] - 1.0) / \
        (g["f_max"] * (3.0 * g["c2"] * f ** 2 + g["c1"]))
