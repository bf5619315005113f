// LAEP prune mask for one layer and one counted batch (laep_prune_mask), and
// Algorithm 1 over a recorded window (laep_expert_pruning).
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

// Algorithm 1 over a window of ITER recorded iterations (Appendix), one
// workgroup per layer, one thread per expert.
//   Step 2: per iteration, the marking rule above on ETN[iter, layer, :] with
//           the layer's alpha; Marker[e] counts the iterations that marked e
//           and Exp_dis the marks of all experts.
//   Step 3: N = floor(Exp_dis / ITER + 0.5) experts are pruned: the most
//           marked, ties to the lower mean load, then the lower index.  All
//           means share the divisor ITER, so they are compared as exact
//           int64 window sums (same order as the float64 means while the
//           sums stay below 2^52).
struct LayerAlphas {
  double a[kMaxLayers];
};

__global__ __launch_bounds__(kPruneThreads) void expert_pruning_kernel(
    const long long* __restrict__ etn, int ITER, int L, int E, long long total,
    const LayerAlphas alpha, double beta, uint8_t* __restrict__ alive,
    int32_t* __restrict__ n_pruned, int32_t* __restrict__ marker_out) {
  __shared__ long long s_c[kPruneThreads];
  __shared__ int s_sorted[kPruneThreads];
  __shared__ long long s_scan[2][kPruneThreads];
  __shared__ int s_mark[kPruneThreads];
  __shared__ long long s_sum[kPruneThreads];
  const int tid = threadIdx.x;
  const int layer = blockIdx.x;
  const double a = alpha.a[layer];
  const double beta_thr = (double)total * beta;
  const double alpha_thr = ((double)total * a) / (double)E;
  s_mark[tid] = 0;
  s_sum[tid] = 0;
  long long exp_dis = 0;
  for (int it = 0; it < ITER; ++it) {
    const long long* row = etn + ((size_t)it * L + layer) * E;
    if (tid < E) {
      s_c[tid] = row[tid];
      s_sum[tid] += row[tid];
    }
    __syncthreads();
    if (tid < E) {
      const long long c = s_c[tid];
      int rank = 0;
      for (int j = 0; j < E; ++j) {
        const long long cj = s_c[j];
        rank += (cj < c) || (cj == c && j < tid);
      }
      s_sorted[rank] = tid;
    }
    __syncthreads();
    int cur = 0;
    s_scan[0][tid] = (tid < E) ? s_c[s_sorted[tid]] : 0ll;
    __syncthreads();
    for (int off = 1; off < kPruneThreads; off <<= 1) {
      const long long v = s_scan[cur][tid] + (tid >= off ? s_scan[cur][tid - off] : 0ll);
      s_scan[cur ^ 1][tid] = v;
      cur ^= 1;
      __syncthreads();
    }
    int marked = 0;
    if (tid < E) {
      const int e = s_sorted[tid];
      const double running = (double)s_scan[cur][tid];
      const double load = (double)s_c[e];
      marked = (running < beta_thr) && (load < alpha_thr);
      s_mark[e] += marked;  // each expert has exactly one rank position
    }
    exp_dis += __syncthreads_count(marked);
  }
  __syncthreads();
  const long long n_dis = (long long)floor((double)exp_dis / (double)ITER + 0.5);
  if (tid < E) {
    const int m = s_mark[tid];
    const long long sm = s_sum[tid];
    int rank = 0;  // position in (marker desc, window load asc, index asc)
    for (int j = 0; j < E; ++j) {
      const int mj = s_mark[j];
      const long long sj = s_sum[j];
      rank += (mj > m) || (mj == m && (sj < sm || (sj == sm && j < tid)));
    }
    alive[(size_t)layer * E + tid] = rank < n_dis ? 0 : 1;
    if (marker_out) marker_out[(size_t)layer * E + tid] = m;
  }
  if (tid == 0) n_pruned[layer] = (int32_t)(n_dis < E ? n_dis : E);
}

}  // namespace

hipError_t launch_prune(const int32_t* counts, int E, int64_t total, double alpha, double beta,
                        uint8_t* alive, int32_t* n_pruned, hipStream_t s) {
  hipLaunchKernelGGL(prune_kernel, dim3(1), dim3(kPruneThreads), 0, s, counts, E,
                     (long long)total, alpha, beta, alive, n_pruned);
  return hipGetLastError();
}

hipError_t launch_expert_pruning(const int64_t* etn, int iters, int L, int E, int64_t total,
                                 const double* alpha, double beta, uint8_t* alive,
                                 int32_t* n_pruned, int32_t* marker, hipStream_t s) {
  LayerAlphas la;
  for (int l = 0; l < kMaxLayers; ++l) la.a[l] = l < L ? alpha[l] : 0.0;
  hipLaunchKernelGGL(expert_pruning_kernel, dim3(L), dim3(kPruneThreads), 0, s,
                     reinterpret_cast<const long long*>(etn), iters, L, E, (long long)total, la,
                     beta, alive, n_pruned, marker);
  return hipGetLastError();
}

}  // namespace laep
