// planner.h -- the cache configurator's solver (Sec. 3.4, Algorithm 1),
// internal to libmoesplit; the public entry point is ms_plan_solve.
#pragma once

#include <stdint.h>

#include <vector>

namespace msp {

struct Problem {
  int L, N, K;
  double U_e;                         // bytes per expert
  double T_att, T_moe, T_head, T_load;
  // per layer: H[C] C = 0..N; P[y] y = 0..N-1 (P_i(y+1)); PH[y][C]
  const double* hit;                  // [L][N+1]
  const double* pred;                 // [L][N]
  const double* pred_hit;             // [L][N][N+1]
};

struct Split {
  std::vector<double> exposed, theta, m;
  std::vector<int> C;
};

// Sub-problem of Eq. (11) for one layer: cache size and split ratio that
// maximise the expected loaded share m of the activated experts.
void subproblem(const Problem& p, int layer, uint64_t V, double T_wind, double* theta, int* C, double* m);
// ExpertSplit: the layers in order, each window from the previous layer.
Split expert_split(const Problem& p, const std::vector<int64_t>& V);
// VramAllocation; returns iterations taken.  V is updated in place.
int vram_allocation(const Problem& p, uint64_t V_e, double zeta, std::vector<int64_t>& V, int max_iter, Split* out);

}  // namespace msp
