// LAEP prune mask for one layer and one counted batch (laep_prune_mask).
//
// Section 3.2, Eqs. (1)-(2), as carried out by the marking step of
// Algorithm 1: rank experts by (load, index) ascending, accumulate the
// loads inclusively in that order, prune an expert iff
//     running < total * beta   and   load < (total * alpha) / E
// with both sides evaluated in IEEE double.  One workgroup, one thread per
// expert (E <= 256).
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kPruneThreads = 256;

__global__ __launch_bounds__(kPruneThreads) void prune_kernel(const int32_t* __restrict__ counts,
                                                              int E, long long total, double alpha,
                                                              double beta,
                                                              uint8_t* __restrict__ alive,
                                                              int32_t* __restrict__ n_pruned) {
  __shared__ int s_c[kPruneThreads];
  __shared__ int s_sorted[kPruneThreads];
  __shared__ long long s_scan[2][kPruneThreads];
  __shared__ int s_flag[kPruneThreads];
  const int tid = threadIdx.x;
  if (tid < E) s_c[tid] = counts[tid];
  __syncthreads();
  // rank of expert tid in the (load, index) order
  if (tid < E) {
    const int c = s_c[tid];
    int rank = 0;
    for (int j = 0; j < E; ++j) {
      const int cj = s_c[j];
      rank += (cj < c) || (cj == c && j < tid);
    }
    s_sorted[rank] = tid;
  }
  __syncthreads();
  // inclusive scan of the sorted loads (Hillis-Steele, double-buffered)
  int cur = 0;
  s_scan[0][tid] = (tid < E) ? (long long)s_c[s_sorted[tid]] : 0ll;
  __syncthreads();
  for (int off = 1; off < kPruneThreads; off <<= 1) {
    const long long v = s_scan[cur][tid] + (tid >= off ? s_scan[cur][tid - off] : 0ll);
    s_scan[cur ^ 1][tid] = v;
    cur ^= 1;
    __syncthreads();
  }
  int pruned = 0;
  if (tid < E) {
    const int e = s_sorted[tid];
    const double running = (double)s_scan[cur][tid];
    const double load = (double)s_c[e];
    const double beta_thr = (double)total * beta;
    const double alpha_thr = ((double)total * alpha) / (double)E;
    pruned = (running < beta_thr) && (load < alpha_thr);
    alive[e] = pruned ? 0 : 1;
  }
  s_flag[tid] = pruned;
  __syncthreads();
  if (tid == 0) {
    int n = 0;
    for (int i = 0; i < E; ++i) n += s_flag[i];
    *n_pruned = n;
  }
}

}  // namespace

hipError_t launch_prune(const int32_t* counts, int E, int64_t total, double alpha, double beta,
                        uint8_t* alive, int32_t* n_pruned, hipStream_t s) {
  hipLaunchKernelGGL(prune_kernel, dim3(1), dim3(kPruneThreads), 0, s, counts, E,
                     (long long)total, alpha, beta, alive, n_pruned);
  return hipGetLastError();
}

}  // namespace laep
