// planner.cpp -- the cache configurator (arXiv 2509.08342, Sec. 3.4,
// Eq. (5)-(11), Algorithm 1): per-layer VRAM budgets and split ratios that
// minimise the summed exposed expert-loading latency, from the statistics
// H_i, P_i, PH_i the runtime gathers (Sec. 3.4.2).
//
// Every product, quotient and sum is taken in double in a fixed order and
// without contraction, so a plan is reproducible bit for bit from the same
// statistics.  Readings: the sub-problem searches the cache sizes whose
// split ratio is at most 1 (all experts whole when the budget covers them),
// equal m keeps the smaller size, m is clipped to [0, K]; in the exposed
// latency and the next window alpha + beta theta is approximated by m and
// beta (1 - theta) + gamma by K - m (as the paper does); a layer without
// budget is infeasible; arg max / arg min ties take the lower layer.
#pragma clang fp contract(off)

#include "planner.h"

#include <cmath>
#include <limits>

namespace msp {

namespace {

// m for cache size C at split ratio theta (Eq. (8)-(10)), prefetching in
// predicted order while the window lasts.
double share(const Problem& p, int layer, int C, double theta, double T_wind) {
  const double* H = p.hit + static_cast<size_t>(layer) * (p.N + 1);
  const double* P = p.pred + static_cast<size_t>(layer) * p.N;
  const double* PH = p.pred_hit + static_cast<size_t>(layer) * p.N * (p.N + 1);
  double m = static_cast<double>(p.K) * H[C] * theta;  // A_cache
  double t = 0.0;
  for (int y = 0; y < p.N; ++y) {
    const double ph = PH[static_cast<size_t>(y) * (p.N + 1) + C];
    const double tp = (1.0 - ph * theta) * p.T_load;  // Eq. (9)
    if (t + tp > T_wind) break;
    t += tp;
    m += (1.0 - ph * theta) * P[y];  // Eq. (10)
  }
  return std::fmin(std::fmax(m, 0.0), static_cast<double>(p.K));
}

}  // namespace

void subproblem(const Problem& p, int layer, uint64_t V, double T_wind, double* theta, int* C, double* m) {
  bool found = false;
  for (int c = 1; c <= p.N; ++c) {
    const double th = static_cast<double>(V) / (static_cast<double>(c) * p.U_e);
    if (th > 1.0) continue;
    const double mm = share(p, layer, c, th, T_wind);
    if (!found || mm > *m) {
      *theta = th;
      *C = c;
      *m = mm;
      found = true;
    }
  }
  if (!found) {  // the budget holds every expert whole
    *theta = 1.0;
    *C = p.N;
    *m = share(p, layer, p.N, 1.0, T_wind);
  }
}

Split expert_split(const Problem& p, const std::vector<int64_t>& V) {
  Split s;
  s.exposed.resize(p.L);
  s.theta.resize(p.L);
  s.m.resize(p.L);
  s.C.resize(p.L);
  const double T_exp = p.T_moe / static_cast<double>(p.K);
  double T_wind = p.T_head + p.T_att;
  for (int i = 0; i < p.L; ++i) {
    if (V[i] <= 0) {
      s.exposed[i] = std::numeric_limits<double>::infinity();
      s.theta[i] = 0.0;
      s.C[i] = 0;
      s.m[i] = 0.0;
      T_wind = p.T_moe + p.T_att;
      continue;
    }
    subproblem(p, i, static_cast<uint64_t>(V[i]), T_wind, &s.theta[i], &s.C[i], &s.m[i]);
    const double T_hide = s.m[i] * T_exp;                                  // Eq. (5)
    const double T_miss = (static_cast<double>(p.K) - s.m[i]) * p.T_load;
    s.exposed[i] = std::fmax(0.0, T_miss - T_hide);                       // Eq. (6)
    T_wind = (p.T_moe - std::fmin(T_hide, T_miss)) + p.T_att;             // Eq. (7)
  }
  return s;
}

int vram_allocation(const Problem& p, uint64_t V_e, double zeta, std::vector<int64_t>& V, int max_iter, Split* out) {
  const int64_t step = static_cast<int64_t>(std::floor(zeta * static_cast<double>(V_e)));
  int it = 0;
  for (;;) {
    Split s1 = expert_split(p, V);
    if (step <= 0 || p.L < 2 || it >= max_iter) {
      *out = s1;
      return it;
    }
    std::vector<int64_t> Vp(V), Vm(V);
    for (int i = 0; i < p.L; ++i) {
      Vp[i] += step;
      Vm[i] -= step;
    }
    const Split s2 = expert_split(p, Vp), s3 = expert_split(p, Vm);
    int i1 = 0;
    for (int i = 1; i < p.L; ++i)
      if (s1.exposed[i] - s2.exposed[i] > s1.exposed[i1] - s2.exposed[i1]) i1 = i;
    int i2 = -1;
    for (int i = 0; i < p.L; ++i) {
      if (i == i1) continue;
      if (i2 < 0 || s3.exposed[i] - s1.exposed[i] < s3.exposed[i2] - s1.exposed[i2]) i2 = i;
    }
    std::vector<int64_t> V4(V);
    V4[i1] += step;
    V4[i2] -= step;
    const Split s4 = expert_split(p, V4);
    double delta = 0.0;
    for (int i = 0; i < p.L; ++i) delta += s4.exposed[i] - s1.exposed[i];
    if (!(delta < 0.0)) {
      *out = s1;
      return it;
    }
    V = V4;
    ++it;
  }
}

}  // namespace msp
