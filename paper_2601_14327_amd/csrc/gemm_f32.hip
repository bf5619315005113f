// Grouped SwiGLU expert FFN, forward, in fp32 (moe_grouped_ffn_fwd with
// LAEP_F32).  This is the full-precision variant for small layers; it runs
// on the vector ALUs with plain fp32 fused multiply-adds:
// 64 x 64 output tiles, 256 threads, each thread a 4 x 4 register block, the
// operands staged through LDS 16 k at a time.
//
// The gate/up pass pairs gate and up columns inside each tile (tile columns
// 0..31 = gate f-columns, 32..63 = the same up f-columns), so the SwiGLU
// epilogue needs no second pass: act_save = A, H = silu(A_g) * A_u.
#include "common.hpp"
#include "internal.hpp"
#include "tiles.hpp"

namespace laep {
namespace {

constexpr int kT = 64;     // rows and columns per tile
constexpr int kKS = 16;    // k per LDS stage
constexpr int kF32Threads = 256;

template <bool GU>
__global__ __launch_bounds__(kF32Threads) void gemm_f32_kernel(
    const float* __restrict__ A, int lda, const float* __restrict__ B, int ldb,
    long long strideB, int N, int K, int f, const TileEntry* __restrict__ table,
    const int* __restrict__ n_entries, int n_tiles_n, float* __restrict__ out, int ldo,
    float* __restrict__ out2) {
  __shared__ float As[kKS][kT + 1];
  __shared__ float Bs[kKS][kT + 1];
  const int entry = blockIdx.x / n_tiles_n;
  const int nt = blockIdx.x % n_tiles_n;
  if (entry >= *n_entries) return;
  const TileEntry te = table[entry];
  const float* Bw = B + (long long)te.phys * strideB;
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;

  float acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0f;

  for (int k0 = 0; k0 < K; k0 += kKS) {
#pragma unroll
    for (int i = 0; i < (kT * kKS) / kF32Threads; ++i) {
      const int idx = tid + i * kF32Threads;
      const int r = idx / kKS, kk = idx % kKS;
      As[kk][r] = (r < te.rows) ? A[(long long)(te.row0 + r) * lda + k0 + kk] : 0.0f;
      int brow;
      bool ok;
      if (GU) {
        const int fcol = nt * 32 + (r & 31);
        ok = fcol < f;
        brow = (r < 32) ? fcol : f + fcol;
      } else {
        brow = nt * kT + r;
        ok = brow < N;
      }
      Bs[kk][r] = ok ? Bw[(long long)brow * ldb + k0 + kk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kKS; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = As[kk][ty * 4 + r];
#pragma unroll
      for (int c = 0; c < 4; ++c) b[c] = Bs[kk][tx + 16 * c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(a[r], b[c], acc[r][c]);
    }
    __syncthreads();
  }

#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = ty * 4 + r;
    if (row >= te.rows) continue;
    const long long grow = te.row0 + row;
    if (GU) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int fcol = nt * 32 + tx + 16 * c;
        if (fcol >= f) continue;
        const float g = acc[r][c], u = acc[r][c + 2];  // columns tx+16c and tx+16c+32
        out[grow * f + fcol] = (g / (1.0f + expf(-g))) * u;
        if (out2) {
          out2[grow * 2 * f + fcol] = g;
          out2[grow * 2 * f + f + fcol] = u;
        }
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = nt * kT + tx + 16 * c;
        if (col < N) out[grow * ldo + col] = acc[r][c];
      }
    }
  }
}

inline int ceil_div_i(long long a, long long b) { return (int)((a + b - 1) / b); }

}  // namespace

hipError_t launch_ffn_fwd_f32(const void* x_perm, const void* w_gu, const void* w_d,
                              const int32_t* offsets, const int32_t* expert_map, int E, int d,
                              int f, int64_t R, void* y_perm, void* act_save, void* ws,
                              hipStream_t s) {
  float* H = static_cast<float*>(ws);
  const int max_entries = ceil_div_i(R, kT) + E;
  TableWs tw = carve_table(static_cast<char*>(ws) + align_up((size_t)R * f * 4, 256), max_entries);
  hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, expert_map,
                     E, kT, 0, max_entries, tw.n_entries, tw.table);
  const int nt_gu = ceil_div_i(f, 32);
  hipLaunchKernelGGL((gemm_f32_kernel<true>), dim3(max_entries * nt_gu), dim3(kF32Threads), 0, s,
                     static_cast<const float*>(x_perm), d, static_cast<const float*>(w_gu), d,
                     (long long)2 * f * d, 2 * f, d, f, tw.table, tw.n_entries, nt_gu, H, f,
                     static_cast<float*>(act_save));
  const int nt_d = ceil_div_i(d, kT);
  hipLaunchKernelGGL((gemm_f32_kernel<false>), dim3(max_entries * nt_d), dim3(kF32Threads), 0, s,
                     H, f, static_cast<const float*>(w_d), f, (long long)d * f, d, f, f, tw.table,
                     tw.n_entries, nt_d, static_cast<float*>(y_perm), d, nullptr);
  return hipGetLastError();
}

}  // namespace laep
