// Expert rearrangement (Section 3.3; Algorithm 2 of the appendix): a host
// utility that places the surviving experts into device groups so that the
// per-group token loads are balanced.  Greedy: experts in descending load
// order (equal loads by index), each into the group with the smallest
// running load that still has room (ties to the lower group index); a full
// group's running load is set to +inf so it is never chosen again.
// Capacity per group is ceil(n / n_groups): with the printed floor the
// groups hold fewer than n experts whenever n_groups does not divide n.
#include <algorithm>
#include <cmath>
#include <limits>
#include <numeric>
#include <vector>

#include "../../include/laep_moe.h"

extern "C" int laep_rearrange(const double* loads, int n, int n_groups, int32_t* group_of,
                              int32_t* order, double* group_sums) {
  if (n < 0 || n_groups < 1) return LAEP_ERR_INVALID_ARG;
  if (n > 0 && (!loads || !group_of || !order)) return LAEP_ERR_INVALID_ARG;
  if (!group_sums) return LAEP_ERR_INVALID_ARG;
  for (int i = 0; i < n; ++i)
    if (std::isnan(loads[i])) return LAEP_ERR_INVALID_ARG;

  const int cap = (n + n_groups - 1) / n_groups;
  std::vector<int> p(n);
  std::iota(p.begin(), p.end(), 0);
  std::stable_sort(p.begin(), p.end(), [&](int a, int b) { return loads[a] > loads[b]; });

  std::vector<std::vector<int>> groups(n_groups);
  std::vector<double> running(n_groups, 0.0);
  for (int idx : p) {
    for (;;) {
      int g = 0;
      for (int i = 1; i < n_groups; ++i)
        if (running[i] < running[g]) g = i;
      if ((int)groups[g].size() < cap) {
        groups[g].push_back(idx);
        running[g] += loads[idx];
        break;
      }
      running[g] = std::numeric_limits<double>::infinity();
    }
  }
  int pos = 0;
  for (int g = 0; g < n_groups; ++g) {
    double sum = 0.0;
    for (int e : groups[g]) {
      group_of[e] = g;
      order[pos++] = e;
      sum += loads[e];
    }
    group_sums[g] = sum;
  }
  return LAEP_OK;
}
