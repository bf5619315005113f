// Backward of router scoring and gating (moe_route_bwd), with the top-k
// selection held fixed (it is piecewise constant in the logits):
//   dl[t, e] = dLoss/dlogits[t, e] from dgate (the softmax Jacobian),
//   dx[t]   (+)= sum_e dl[t, e] W_r[e]
//   dW_r[e]   = sum_t dl[t, e] x[t],   db[e] = sum_t dl[t, e]
// Renormalised gates make dl zero outside the k selected experts, so dx is a
// k-term weighted sum of W_r rows (like the combine) and dW_r[e] a weighted
// sum over the expert's routed rows, which moe_expert_counts already lists
// in expert order (row_src).  Full-softmax gates make dl dense over the alive
// experts; the same kernels then run over all E experts and all T tokens.
// Every sum runs in a fixed order: results are deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kDlThreads = 256;

// One thread per token.  renorm: dl_slot[t, j] = g_j (dg_j - sum_i g_i dg_i)
// (0 for unrouted slots).  Full softmax: dl_full[t, e] = p_e (q_e - sum_j g_j dg_j)
// over alive e, p = softmax of the alive logits, q_e = dg_j at e = idx[t, j].
// dlogits (optional) gets the dense [T, E] gradient in both cases.
__global__ __launch_bounds__(kDlThreads) void route_bwd_dl_kernel(
    const float* __restrict__ dgate, const int32_t* __restrict__ idx,
    const float* __restrict__ gate, const float* __restrict__ logits,
    const uint8_t* __restrict__ alive, int T, int E, int k, int renorm,
    float* __restrict__ dl_out, float* __restrict__ dlogits) {
  const int t = blockIdx.x * kDlThreads + threadIdx.x;
  if (t >= T) return;
  const size_t s0 = (size_t)t * k;
  float s = 0.0f;
  for (int j = 0; j < k; ++j)
    if (idx[s0 + j] >= 0) s += gate[s0 + j] * dgate[s0 + j];
  if (renorm) {
    if (dlogits)
      for (int e = 0; e < E; ++e) dlogits[(size_t)t * E + e] = 0.0f;
    for (int j = 0; j < k; ++j) {
      const int e = idx[s0 + j];
      const float v = e >= 0 ? gate[s0 + j] * (dgate[s0 + j] - s) : 0.0f;
      dl_out[s0 + j] = v;
      if (dlogits && e >= 0) dlogits[(size_t)t * E + e] = v;
    }
  } else {
    const float* l = logits + (size_t)t * E;
    float m = -INFINITY;
    for (int e = 0; e < E; ++e)
      if (alive == nullptr || alive[e]) m = fmaxf(m, l[e]);
    float z = 0.0f;
    for (int e = 0; e < E; ++e)
      if (alive == nullptr || alive[e]) z += __expf(l[e] - m);
    const float inv = z > 0.0f ? 1.0f / z : 0.0f;
    for (int e = 0; e < E; ++e) {
      float q = 0.0f;
      for (int j = 0; j < k; ++j)
        if (idx[s0 + j] == e) q = dgate[s0 + j];
      const bool a = alive == nullptr || alive[e];
      const float v = a ? __expf(l[e] - m) * inv * (q - s) : 0.0f;
      dl_out[(size_t)t * E + e] = v;
      if (dlogits) dlogits[(size_t)t * E + e] = v;
    }
  }
}

// dx[t] (+)= sum over slots of w * W_r[row]: `slots` per token, row ids from
// `ids` ([T, slots], -1 = none) or the slot number itself when ids == NULL,
// weights dl [T, slots].  Each thread owns one 8-column vector of one token.
template <typename T>
__global__ __launch_bounds__(256) void route_bwd_dx_kernel(
    const T* __restrict__ w_router, const int32_t* __restrict__ ids,
    const float* __restrict__ dl, int n_tok, int slots, int d, int accumulate,
    T* __restrict__ dx) {
  const int vec_per_row = d / 8;
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long long)n_tok * vec_per_row) return;
  const int t = (int)(i / vec_per_row), v = (int)(i % vec_per_row);
  float acc[8];
  if (accumulate) {
    Elem<T>::load8(dx + (size_t)t * d + (size_t)v * 8, acc);
  } else {
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = 0.0f;
  }
  // slot order; for full-softmax gates (ids == NULL) every expert is a slot
  float sum[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) sum[q] = 0.0f;
  for (int s = 0; s < slots; ++s) {
    const size_t o = (size_t)t * slots + s;
    const int r = ids ? ids[o] : s;
    const float w = dl[o];
    if (r < 0 || w == 0.0f) continue;
    float val[8];
    Elem<T>::load8(w_router + (size_t)r * d + (size_t)v * 8, val);
#pragma unroll
    for (int q = 0; q < 8; ++q) sum[q] += w * val[q];
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] += sum[q];
  Elem<T>::store8(dx + (size_t)t * d + (size_t)v * 8, acc);
}

// dW_r[e, c0 + 0..255] and db[e]: workgroup (e, column chunk); 8 row lanes x
// 32 vector lanes.  Row lane rl takes rows rl, rl + 8, ... of the expert; the
// 8 partial sums are then added in lane order through LDS.
//   renorm (row_src != NULL): rows = the expert's routed rows
//     [offsets[e], offsets[e+1]); slot s = row_src[r], token s / k, weight dl[s]
//   full softmax: rows = every token t, weight dl[t * E + e]
template <typename T>
__global__ __launch_bounds__(256) void route_bwd_dw_kernel(
    const T* __restrict__ x, const float* __restrict__ dl, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ row_src, int n_tok, int k, int E, int d,
    float* __restrict__ dw, float* __restrict__ db) {
  __shared__ float s_part[8][32 * 8 + 4];
  __shared__ float s_bias[8];
  const int e = blockIdx.x;
  const int chunk = blockIdx.y;
  const int rl = threadIdx.x >> 5, vl = threadIdx.x & 31;
  const int v = chunk * 32 + vl;              // 8-column vector index
  const bool col_ok = v * 8 < d;
  int r0, r1;
  if (row_src) {
    r0 = offsets[e];
    r1 = offsets[e + 1];
  } else {
    r0 = 0;
    r1 = n_tok;
  }
  float acc[8], bsum = 0.0f;
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] = 0.0f;
  // four rows in flight per thread
  for (int r = r0 + rl; r < r1; r += 32) {
    int tok[4];
    float w[4];
    float val[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int rr = r + 8 * u;
      tok[u] = -1;
      w[u] = 0.0f;
      if (rr < r1) {
        if (row_src) {
          const int s = row_src[rr];
          tok[u] = s / k;
          w[u] = dl[s];
        } else {
          tok[u] = rr;
          w[u] = dl[(size_t)rr * E + e];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (tok[u] >= 0 && col_ok) {
        Elem<T>::load8(x + (size_t)tok[u] * d + (size_t)v * 8, val[u]);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) val[u][q] = 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      bsum += w[u];
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] += w[u] * val[u][q];
    }
  }
#pragma unroll
  for (int q = 0; q < 8; ++q) s_part[rl][vl * 8 + q] = acc[q];
  if (vl == 0) s_bias[rl] = bsum;
  __syncthreads();
  if (rl == 0 && col_ok) {
    float out[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      float tsum = 0.0f;
      for (int j = 0; j < 8; ++j) tsum += s_part[j][vl * 8 + q];
      out[q] = tsum;
    }
    Elem<float>::store8(dw + (size_t)e * d + (size_t)v * 8, out);
  }
  if (db != nullptr && chunk == 0 && threadIdx.x == 0) {
    float tsum = 0.0f;
    for (int j = 0; j < 8; ++j) tsum += s_bias[j];
    db[e] = tsum;
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

}  // namespace

size_t route_bwd_ws_bytes(int T, int k, int E) {
  return align_up((size_t)T * (k > E ? k : E) * sizeof(float), 256);
}

hipError_t launch_route_bwd(const float* dgate, const int32_t* idx, const float* gate,
                            const float* logits, const uint8_t* alive, const void* x,
                            const void* w_router, const int32_t* offsets, const int32_t* row_src,
                            int dtype, int T_, int d, int E, int k, int renorm, float* dlogits,
                            float* dw_router, float* dbias, void* dx, int accumulate_dx, void* ws,
                            hipStream_t s) {
  if (T_ == 0) {
    // no tokens: zero weight gradients (dx has no rows)
    hipLaunchKernelGGL(fill_zero_kernel, dim3(64), dim3(256), 0, s, dw_router, (size_t)E * d);
    if (dbias) hipLaunchKernelGGL(fill_zero_kernel, dim3(1), dim3(256), 0, s, dbias, (size_t)E);
    return hipGetLastError();
  }
  float* dl = static_cast<float*>(ws);
  hipLaunchKernelGGL(route_bwd_dl_kernel, dim3((T_ + kDlThreads - 1) / kDlThreads),
                     dim3(kDlThreads), 0, s, dgate, idx, gate, logits, alive, T_, E, k, renorm,
                     dl, dlogits);
  const int slots = renorm ? k : E;
  const int32_t* ids = renorm ? idx : nullptr;
  const long long n_vec = (long long)T_ * (d / 8);
  const dim3 gdx((unsigned)((n_vec + 255) / 256)), gdw(E, (d / 8 + 31) / 32);
  const int32_t* rs = renorm ? row_src : nullptr;
  if (dtype == kDtypeBf16) {
    hipLaunchKernelGGL(route_bwd_dx_kernel<bf16_t>, gdx, dim3(256), 0, s,
                       static_cast<const bf16_t*>(w_router), ids, dl, T_, slots, d, accumulate_dx,
                       static_cast<bf16_t*>(dx));
    hipLaunchKernelGGL(route_bwd_dw_kernel<bf16_t>, gdw, dim3(256), 0, s,
                       static_cast<const bf16_t*>(x), dl, offsets, rs, T_, k, E, d, dw_router,
                       dbias);
  } else {
    hipLaunchKernelGGL(route_bwd_dx_kernel<float>, gdx, dim3(256), 0, s,
                       static_cast<const float*>(w_router), ids, dl, T_, slots, d, accumulate_dx,
                       static_cast<float*>(dx));
    hipLaunchKernelGGL(route_bwd_dw_kernel<float>, gdw, dim3(256), 0, s,
                       static_cast<const float*>(x), dl, offsets, rs, T_, k, E, d, dw_router,
                       dbias);
  }
  return hipGetLastError();
}

}  // namespace laep
