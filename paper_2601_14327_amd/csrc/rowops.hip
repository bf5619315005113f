// Row movement kernels of the dispatch and return paths:
//   moe_permute      x_perm[dest_row[t*k + j]] = x[t]
//   moe_combine      out[t] = sum_j g[t, j] * y[dest_row[t*k + j]]
//   moe_permute_bwd  dx[t]  = sum_j dx_perm[dest_row[t*k + j]]
//   moe_combine_bwd  dgate[t, j] = <dout[t], y[row]>, dy[row] = g[t, j] * dout[t]
// All are HBM-bound.  Rows move as 16-byte vectors; consecutive threads own
// consecutive vectors of a row, so every wave access is one contiguous run.
// Rows read once go through streaming (non-temporal) loads, and x_perm
// through streaming stores; outputs the next call reads (out, dx, dy) keep
// ordinary stores, so they stay in the caches for it.
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kRowThreads = 256;

// Tokens per workgroup: enough vectors for every thread to have ~2.
__host__ __device__ inline int tokens_per_block(int vec_per_row) {
  int tpb = (2 * kRowThreads) / (vec_per_row > 0 ? vec_per_row : 1);
  return tpb < 1 ? 1 : (tpb > 16 ? 16 : tpb);
}

__global__ __launch_bounds__(kRowThreads) void permute_kernel(
    const u32x4_t* __restrict__ x, const int32_t* __restrict__ dest_row, int n_tok, int k,
    int vec_per_row, int tpb, u32x4_t* __restrict__ x_perm) {
  const int t_lo = blockIdx.x * tpb;
  const int n_vec = tpb * vec_per_row;
  for (int i = threadIdx.x; i < n_vec; i += kRowThreads) {
    const int t = t_lo + i / vec_per_row;
    const int v = i % vec_per_row;
    if (t >= n_tok) break;
    const u32x4_t val = ld_stream(x + (size_t)t * vec_per_row + v);
    for (int j = 0; j < k; ++j) {
      const int r = dest_row[(size_t)t * k + j];
      if (r >= 0) st_stream(x_perm + (size_t)r * vec_per_row + v, val);
    }
  }
}

// Dispatch in routed-row order: x_perm[r] = x[row_src[r] / k], one 16-byte
// vector per thread.  The token rows are read k times each (cached loads);
// x_perm is written once and read only by a later call (streaming stores).
__global__ __launch_bounds__(kRowThreads) void gather_rows_kernel(
    const u32x4_t* __restrict__ x, const int32_t* __restrict__ row_src, int k, int64_t R,
    int vec_per_row, u32x4_t* __restrict__ x_perm) {
  const long long i = (long long)blockIdx.x * kRowThreads + threadIdx.x;
  if (i >= R * vec_per_row) return;
  const long long r = i / vec_per_row;
  const int v = (int)(i % vec_per_row);
  const int t = row_src[r] / k;
  st_stream(x_perm + i, x[(size_t)t * vec_per_row + v]);
}

// One 8-element row vector in its storage format: load (zero when !ok) and
// acc[e] += g * value[e].
template <typename T> struct RawRow;
template <> struct RawRow<bf16_t> {
  typedef u32x4_t type;
  __device__ static __forceinline__ type load(const bf16_t* p, bool ok) {
    type v = {0u, 0u, 0u, 0u};
    if (ok) v = ld_stream(reinterpret_cast<const u32x4_t*>(p));
    return v;
  }
  __device__ static __forceinline__ void fma8(float acc[8], float g, const type& v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += g * lo_bf16(v[i]);
      acc[2 * i + 1] += g * hi_bf16(v[i]);
    }
  }
};
template <> struct RawRow<float> {
  struct type { f32x4_t a, b; };
  __device__ static __forceinline__ type load(const float* p, bool ok) {
    type v;
    v.a = f32x4_t{0.f, 0.f, 0.f, 0.f};
    v.b = v.a;
    if (ok) {
      v.a = ld_stream(reinterpret_cast<const f32x4_t*>(p));
      v.b = ld_stream(reinterpret_cast<const f32x4_t*>(p + 4));
    }
    return v;
  }
  __device__ static __forceinline__ void fma8(float acc[8], float g, const type& v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[i] += g * v.a[i];
      acc[4 + i] += g * v.b[i];
    }
  }
};

// Each thread owns UNR (token, vector) items per pass and issues every row
// load of the pass (up to 8 slots per item) before the first sum, so the two
// dependent rounds (dest_row / gate, then the rows) are paid once per pass.
template <typename T, bool GATED>
__global__ __launch_bounds__(kRowThreads) void combine_kernel(
    const T* __restrict__ y, const float* __restrict__ gate, const int32_t* __restrict__ dest_row,
    int n_tok, int k, int d, int tpb, T* __restrict__ out) {
  constexpr int UNR = sizeof(T) == 2 ? 2 : 1;
  const int vec_per_row = d / 8;
  const int t_lo = blockIdx.x * tpb;
  const int n_vec = tpb * vec_per_row;
  for (int i0 = threadIdx.x; i0 < n_vec; i0 += UNR * kRowThreads) {
    int t[UNR], v[UNR];
    bool ok[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u * kRowThreads;
      t[u] = t_lo + i / vec_per_row;
      v[u] = i % vec_per_row;
      ok[u] = i < n_vec && t[u] < n_tok;
    }
    float acc[UNR][8];
#pragma unroll
    for (int u = 0; u < UNR; ++u)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[u][q] = 0.0f;
    // slots in groups of 8; the sums run in slot order
    for (int j0 = 0; j0 < k; j0 += 8) {
      int r[UNR][8];
      float g[UNR][8];
#pragma unroll
      for (int u = 0; u < UNR; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int j = j0 + q;
          const size_t s = (size_t)t[u] * k + j;
          const bool in = ok[u] && j < k;
          r[u][q] = in ? dest_row[s] : -1;
          g[u][q] = (GATED && in) ? gate[s] : 1.0f;
        }
      // rows stay in their storage format until summed (bf16: 4 registers per row)
      typename RawRow<T>::type raw[UNR][8];
#pragma unroll
      for (int u = 0; u < UNR; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q)
          raw[u][q] = RawRow<T>::load(y + (size_t)(r[u][q] >= 0 ? r[u][q] : 0) * d +
                                      (size_t)v[u] * 8, r[u][q] >= 0);
#pragma unroll
      for (int u = 0; u < UNR; ++u)
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (r[u][q] >= 0) RawRow<T>::fma8(acc[u], g[u][q], raw[u][q]);
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (ok[u]) Elem<T>::store8(out + (size_t)t[u] * d + (size_t)v[u] * 8, acc[u]);
  }
}

// One workgroup per token.
template <typename T>
__global__ __launch_bounds__(kRowThreads) void combine_bwd_kernel(
    const T* __restrict__ dout, const T* __restrict__ y, const float* __restrict__ gate,
    const int32_t* __restrict__ dest_row, int n_tok, int k, int d, T* __restrict__ dy,
    float* __restrict__ dgate) {
  __shared__ float s_red[kRowThreads / 64];
  const int t = blockIdx.x;
  const int vec_per_row = d / 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const T* drow = dout + (size_t)t * d;
  for (int j = 0; j < k; ++j) {
    const size_t s = (size_t)t * k + j;
    const int r = dest_row[s];
    if (r < 0) {  // uniform across the workgroup
      if (threadIdx.x == 0) dgate[s] = 0.0f;
      continue;
    }
    const float g = gate[s];
    float part = 0.0f;
    for (int v = threadIdx.x; v < vec_per_row; v += kRowThreads) {
      float dv[8], yv[8], o[8];
      Elem<T>::load8(drow + (size_t)v * 8, dv);
      Elem<T>::load8_stream(y + (size_t)r * d + (size_t)v * 8, yv);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        part += dv[q] * yv[q];
        o[q] = g * dv[q];
      }
      if (dy != nullptr) Elem<T>::store8(dy + (size_t)r * d + (size_t)v * 8, o);
    }
    part = wave_sum(part);
    if (lane == 0) s_red[wave] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
      float tot = 0.0f;
      for (int w = 0; w < kRowThreads / 64; ++w) tot += s_red[w];
      dgate[s] = tot;
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_permute(const void* x, int elem_bytes, const int32_t* dest_row, int T, int k,
                          int d, void* x_perm, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int vec_per_row = d * elem_bytes / 16;
  const int tpb = tokens_per_block(vec_per_row);
  hipLaunchKernelGGL(permute_kernel, dim3((T + tpb - 1) / tpb), dim3(kRowThreads), 0, s,
                     static_cast<const u32x4_t*>(x), dest_row, T, k, vec_per_row, tpb,
                     static_cast<u32x4_t*>(x_perm));
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* x, const int32_t* row_src, int k, int64_t R, int d,
                              int elem_bytes, void* x_perm, hipStream_t s) {
  if (R == 0) return hipSuccess;
  const int vec_per_row = d * elem_bytes / 16;
  const long long n = R * (long long)vec_per_row;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)((n + kRowThreads - 1) / kRowThreads)),
                     dim3(kRowThreads), 0, s, static_cast<const u32x4_t*>(x), row_src, k, R,
                     vec_per_row, static_cast<u32x4_t*>(x_perm));
  return hipGetLastError();
}

hipError_t launch_combine(const void* y, const float* gate, const int32_t* dest_row, int T, int k,
                          int d, int dtype, void* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int tpb = tokens_per_block(d / 8);
  dim3 grid((T + tpb - 1) / tpb), block(kRowThreads);
  if (dtype == kDtypeBf16) {
    if (gate)
      hipLaunchKernelGGL((combine_kernel<bf16_t, true>), grid, block, 0, s,
                         static_cast<const bf16_t*>(y), gate, dest_row, T, k, d, tpb,
                         static_cast<bf16_t*>(out));
    else
      hipLaunchKernelGGL((combine_kernel<bf16_t, false>), grid, block, 0, s,
                         static_cast<const bf16_t*>(y), gate, dest_row, T, k, d, tpb,
                         static_cast<bf16_t*>(out));
  } else {
    if (gate)
      hipLaunchKernelGGL((combine_kernel<float, true>), grid, block, 0, s,
                         static_cast<const float*>(y), gate, dest_row, T, k, d, tpb,
                         static_cast<float*>(out));
    else
      hipLaunchKernelGGL((combine_kernel<float, false>), grid, block, 0, s,
                         static_cast<const float*>(y), gate, dest_row, T, k, d, tpb,
                         static_cast<float*>(out));
  }
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const void* dout, const void* y, const float* gate,
                              const int32_t* dest_row, int T, int k, int d, int dtype, void* dy,
                              float* dgate, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (dtype == kDtypeBf16)
    hipLaunchKernelGGL((combine_bwd_kernel<bf16_t>), dim3(T), dim3(kRowThreads), 0, s,
                       static_cast<const bf16_t*>(dout), static_cast<const bf16_t*>(y), gate,
                       dest_row, T, k, d, static_cast<bf16_t*>(dy), dgate);
  else
    hipLaunchKernelGGL((combine_bwd_kernel<float>), dim3(T), dim3(kRowThreads), 0, s,
                       static_cast<const float*>(dout), static_cast<const float*>(y), gate,
                       dest_row, T, k, d, static_cast<float*>(dy), dgate);
  return hipGetLastError();
}

}  // namespace laep
