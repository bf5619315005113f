// Physical expert compaction after pruning (Section 3.2: pruned experts are
// removed from the model, which is the parameter reduction LAEP reports).
//
//   expert_map_kernel: per layer, the surviving experts keep their order and
//     take consecutive slots: map[e] = #{alive j < e} if e is alive, else -1.
//   repack_kernel: copies each surviving expert's parameter block (a W_r row,
//     a [2f, d] gate/up matrix, a [d, f] down matrix, or an optimizer state of
//     the same shape) from its logical index to its slot; a pure HBM copy.
#include "common.hpp"
#include "internal.hpp"
#include "tiles.hpp"

namespace laep {
namespace {

// One workgroup per layer, one thread per expert (E <= 256).
__global__ __launch_bounds__(kTableThreads) void expert_map_kernel(
    const uint8_t* __restrict__ alive, int E, int32_t* __restrict__ expert_map,
    int32_t* __restrict__ n_alive) {
  __shared__ int s_tmp[4];
  const int layer = blockIdx.x;
  const int e = threadIdx.x;
  const int a = (e < E && alive[(size_t)layer * E + e] != 0) ? 1 : 0;
  const int slot = block_excl_scan_256(a, s_tmp);
  if (e < E) expert_map[(size_t)layer * E + e] = a ? slot : -1;
  if (e == kTableThreads - 1) n_alive[layer] = slot + a;
}

// Workgroup (chunk, expert).  Blocks of an expert that is pruned, or whose
// slot is not below n_out, copy nothing.  bytes_per_expert % 16 == 0.
constexpr int kRepackThreads = 256;
constexpr int kRepackUnroll = 4;
__global__ __launch_bounds__(kRepackThreads) void repack_kernel(
    const int32_t* __restrict__ expert_map, int n_out, const uint4* __restrict__ src,
    uint4* __restrict__ dst, long long vec_per_expert) {
  const int e = blockIdx.y;
  const int p = expert_map[e];
  if (p < 0 || p >= n_out) return;
  const uint4* in = src + (size_t)e * vec_per_expert;
  uint4* out = dst + (size_t)p * vec_per_expert;
  const long long stride = (long long)gridDim.x * kRepackThreads * kRepackUnroll;
  for (long long i0 = (long long)blockIdx.x * kRepackThreads * kRepackUnroll + threadIdx.x;
       i0 < vec_per_expert; i0 += stride) {
    uint4 v[kRepackUnroll];
#pragma unroll
    for (int u = 0; u < kRepackUnroll; ++u) {
      const long long i = i0 + (long long)u * kRepackThreads;
      if (i < vec_per_expert) v[u] = in[i];
    }
#pragma unroll
    for (int u = 0; u < kRepackUnroll; ++u) {
      const long long i = i0 + (long long)u * kRepackThreads;
      if (i < vec_per_expert) out[i] = v[u];
    }
  }
}

// Per-expert scalars (a bias entry): one thread per expert.
__global__ __launch_bounds__(256) void repack_scalar_kernel(const int32_t* __restrict__ expert_map,
                                                            int E, int n_out,
                                                            const float* __restrict__ src,
                                                            float* __restrict__ dst) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= E) return;
  const int p = expert_map[e];
  if (p >= 0 && p < n_out) dst[p] = src[e];
}

}  // namespace

hipError_t launch_expert_map(const uint8_t* alive, int L, int E, int32_t* expert_map,
                             int32_t* n_alive, hipStream_t s) {
  hipLaunchKernelGGL(expert_map_kernel, dim3(L), dim3(kTableThreads), 0, s, alive, E, expert_map,
                     n_alive);
  return hipGetLastError();
}

hipError_t launch_repack(const int32_t* expert_map, int E, int n_out, const void* src, void* dst,
                         size_t bytes_per_expert, hipStream_t s) {
  const long long vec = (long long)(bytes_per_expert / 16);
  // enough chunks per expert to fill the chip several times over
  long long chunks = (vec + kRepackThreads * kRepackUnroll - 1) / (kRepackThreads * kRepackUnroll);
  const long long want = (2048 + E - 1) / E;
  if (chunks > want) chunks = want;
  if (chunks < 1) chunks = 1;
  hipLaunchKernelGGL(repack_kernel, dim3((unsigned)chunks, (unsigned)E), dim3(kRepackThreads), 0,
                     s, expert_map, n_out, static_cast<const uint4*>(src), static_cast<uint4*>(dst),
                     vec);
  return hipGetLastError();
}

hipError_t launch_repack_scalar(const int32_t* expert_map, int E, int n_out, const float* src,
                                float* dst, hipStream_t s) {
  hipLaunchKernelGGL(repack_scalar_kernel, dim3((E + 255) / 256), dim3(256), 0, s, expert_map, E,
                     n_out, src, dst);
  return hipGetLastError();
}

}  // namespace laep
