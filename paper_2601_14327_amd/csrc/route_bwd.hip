// Backward of router scoring and gating (moe_route_bwd), with the top-k
// selection held fixed (it is piecewise constant in the logits):
//   dl[t, e] = dLoss/dlogits[t, e] from dgate (the softmax Jacobian),
//   dx[t]   (+)= sum_e dl[t, e] W_r[e]
//   dW_r[e]   = sum_t dl[t, e] x[t],   db[e] = sum_t dl[t, e]
// Renormalised gates make dl zero outside the k selected experts, so dx is a
// k-term weighted sum of W_r rows (like the combine) and dW_r[e] a weighted
// sum over the expert's routed rows, which moe_expert_counts already lists
// in expert order (row_src).  Full-softmax gates make dl dense over the alive
// experts; dx then sums over all E experts and dW_r over all T tokens.
// Every sum runs in a fixed order: results are deterministic.
#include "common.hpp"
#include "internal.hpp"
#include "tiles.hpp"

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
// weights dl [T, slots].  One wave per token (its ids and weights are
// wave-uniform loads); each lane owns the 8-column vectors lane, lane + 64, ...
template <typename T>
__global__ __launch_bounds__(256) void route_bwd_dx_kernel(
    const T* __restrict__ w_router, const int32_t* __restrict__ ids,
    const float* __restrict__ dl, int n_tok, int slots, int d, int accumulate,
    T* __restrict__ dx) {
  const int t = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (int)(threadIdx.x >> 6));
  if (t >= n_tok) return;
  const int lane = threadIdx.x & 63;
  const int vec_per_row = d / 8;
  const size_t o = (size_t)t * slots;
  for (int v = lane; v < vec_per_row; v += 64) {
    float acc[8];
    if (accumulate) {
      Elem<T>::load8(dx + (size_t)t * d + (size_t)v * 8, acc);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[q] = 0.0f;
    }
    // slot order, in groups of 8 whose row loads are all issued before the
    // sums; for full-softmax gates (ids == NULL) every expert is a slot
    float sum[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) sum[q] = 0.0f;
    for (int s0 = 0; s0 < slots; s0 += 8) {
      int r[8];
      float w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int s = s0 + u;
        r[u] = -1;
        w[u] = 0.0f;
        if (s < slots) {
          r[u] = ids ? ids[o + s] : s;
          w[u] = dl[o + s];
        }
        if (w[u] == 0.0f) r[u] = -1;
      }
      float val[8][8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (r[u] >= 0) {
          Elem<T>::load8(w_router + (size_t)r[u] * d + (size_t)v * 8, val[u]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) val[u][q] = 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (r[u] >= 0) {
#pragma unroll
          for (int q = 0; q < 8; ++q) sum[q] += w[u] * val[u][q];
        }
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] += sum[q];
    Elem<T>::store8(dx + (size_t)t * d + (size_t)v * 8, acc);
  }
}

// Full-softmax gates: dW_r[e, c0 + 0..255] and db[e] over every token t with
// weight dl[t * E + e].  Workgroup (e, column chunk); 8 row lanes x 32 vector
// lanes.  Row lane rl takes tokens rl, rl + 8, ...; the 8 partial sums are
// then added in lane order through LDS.
template <typename T>
__global__ __launch_bounds__(256) void route_bwd_dw_kernel(
    const T* __restrict__ x, const float* __restrict__ dl, int n_tok, int E, int d,
    float* __restrict__ dw, float* __restrict__ db) {
  __shared__ float s_part[8][32 * 8 + 4];
  __shared__ float s_bias[8];
  const int e = blockIdx.x;
  const int chunk = blockIdx.y;
  const int rl = threadIdx.x >> 5, vl = threadIdx.x & 31;
  const int v = chunk * 32 + vl;              // 8-column vector index
  const bool col_ok = v * 8 < d;
  const int r0 = 0, r1 = n_tok;
  float acc[8], bsum = 0.0f;
#pragma unroll
  for (int q = 0; q < 8; ++q) acc[q] = 0.0f;
  // eight rows in flight per thread
  for (int r = r0 + rl; r < r1; r += 64) {
    int tok[8];
    float w[8];
    float val[8][8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int rr = r + 8 * u;
      tok[u] = -1;
      w[u] = 0.0f;
      if (rr < r1) {
        tok[u] = rr;
        w[u] = dl[(size_t)rr * E + e];
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (tok[u] >= 0 && col_ok) {
        Elem<T>::load8(x + (size_t)tok[u] * d + (size_t)v * 8, val[u]);
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) val[u][q] = 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
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

// Renormalised gates, weight gradient in two deterministic passes.
// Pass 1: one workgroup per 128-row segment of an expert's routed rows (the
// row-tile table); the segment's (token, weight) pairs go to LDS first, then
// every x row is read whole (each thread one 8-column vector, eight rows in
// flight) and the segment's partial dW_r row and bias sum are written.
constexpr int kSegRows = 128;
template <typename T, int VPT>
__global__ __launch_bounds__(256) void route_bwd_dw_seg_kernel(
    const T* __restrict__ x, const float* __restrict__ dl, const int32_t* __restrict__ row_src,
    const TileEntry* __restrict__ table, const int* __restrict__ n_entries, int k, int d,
    float* __restrict__ part, float* __restrict__ part_b) {
  __shared__ int s_tok[kSegRows];
  __shared__ float s_w[kSegRows];
  __shared__ float s_red[4];
  const int entry = blockIdx.x;
  if (entry >= *n_entries) return;
  const TileEntry te = table[entry];
  const int tid = threadIdx.x;
  if (tid < te.rows) {
    const int sl = row_src[te.row0 + tid];
    s_tok[tid] = sl / k;
    s_w[tid] = dl[sl];
  }
  __syncthreads();
  const int nvec = d / 8;
  float* out = part + (size_t)entry * d;
  for (int v0 = 0; v0 < nvec; v0 += 256 * VPT) {
    float acc[VPT][8];
#pragma unroll
    for (int u = 0; u < VPT; ++u)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[u][q] = 0.0f;
    for (int r0 = 0; r0 < te.rows; r0 += 8) {
      float val[8][VPT][8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
          const int v = v0 + u * 256 + tid;
          if (r0 + i < te.rows && v < nvec) {
            Elem<T>::load8(x + (size_t)s_tok[r0 + i] * d + (size_t)v * 8, val[i][u]);
          } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) val[i][u][q] = 0.0f;
          }
        }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float w = r0 + i < te.rows ? s_w[r0 + i] : 0.0f;
#pragma unroll
        for (int u = 0; u < VPT; ++u)
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[u][q] += w * val[i][u][q];
      }
    }
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int v = v0 + u * 256 + tid;
      if (v < nvec) Elem<float>::store8(out + (size_t)v * 8, acc[u]);
    }
  }
  // the segment's bias sum, in row order
  float b = 0.0f;
  if (tid < 64) {
    for (int r = tid; r < te.rows; r += 64) b += s_w[r];
    b = wave_sum(b);
  }
  if (tid == 0) part_b[entry] = b;
}

// Pass 2: dW_r[e] = sum of the expert's segment partials in table order.
__global__ __launch_bounds__(256) void route_bwd_dw_reduce_kernel(
    const float* __restrict__ part, const float* __restrict__ part_b,
    const TileEntry* __restrict__ table, const int* __restrict__ n_entries, int E, int d,
    float* __restrict__ dw, float* __restrict__ db) {
  // the expert's segments are consecutive in the table; find them in parallel
  __shared__ int s_first, s_count;
  const int e = blockIdx.x;
  if (threadIdx.x == 0) {
    s_first = INT_MAX;
    s_count = 0;
  }
  __syncthreads();
  const int n = *n_entries;
  for (int i = threadIdx.x; i < n; i += 256)
    if (table[i].expert == e) {
      atomicMin(&s_first, i);
      atomicAdd(&s_count, 1);
    }
  __syncthreads();
  const int first = s_first, count = s_count;
  for (int c = blockIdx.y * 256 + threadIdx.x; c < d; c += gridDim.y * 256) {
    float acc = 0.0f;
    for (int i = 0; i < count; ++i) acc += part[(size_t)(first + i) * d + c];
    dw[(size_t)e * d + c] = acc;
  }
  if (db != nullptr && blockIdx.y == 0 && threadIdx.x == 0) {
    float acc = 0.0f;
    for (int i = 0; i < count; ++i) acc += part_b[first + i];
    db[e] = acc;
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

}  // namespace

// ws: dl, then (renormalised gates) the segment table, partial rows and sums.
// The segment partials need d; the workspace query has none, so the partial
// area is sized for the largest d_model the caller passes (d_model is an
// argument of moe_workspace_bytes for the backward calls).
inline int seg_max(int T, int k, int E) { return (int)(((int64_t)T * k + kSegRows - 1) / kSegRows) + E; }

size_t route_bwd_ws_bytes(int T, int k, int E, int d) {
  const int m = seg_max(T, k, E);
  return align_up((size_t)T * (k > E ? k : E) * sizeof(float), 256) + table_bytes(m) +
         align_up((size_t)m * d * sizeof(float), 256) + align_up((size_t)m * sizeof(float), 256);
}

hipError_t launch_route_bwd(const float* dgate, const int32_t* idx, const float* gate,
                            const float* logits, const uint8_t* alive, const void* x,
                            const void* w_router, const int32_t* offsets, const int32_t* row_src,
                            int dtype, int T_, int d, int E, int k, int renorm, float* dlogits,
                            float* dw_router, float* dbias, void* dx, int accumulate_dx, void* ws,
                            hipStream_t s) {
  if (T_ == 0) {
    // no tokens: zero weight gradients (dx has no rows)
    if (dw_router)
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
  const dim3 gdx((unsigned)((T_ + 3) / 4)), gdw(E, (d / 8 + 31) / 32);
  // renormalised gates: segment table of the routed rows (pass 1 + 2)
  const int m = seg_max(T_, k, E);
  char* base = static_cast<char*>(ws) + align_up((size_t)T_ * (k > E ? k : E) * sizeof(float), 256);
  TableWs tw = carve_table(base, m);
  float* part = reinterpret_cast<float*>(base + table_bytes(m));
  float* part_b = reinterpret_cast<float*>(base + table_bytes(m) + align_up((size_t)m * d * 4, 256));
  // dx (optional) and the weight gradients (optional, with dbias)
  if (renorm && dw_router)
    hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, nullptr, E,
                       kSegRows, 0, m, tw.n_entries, tw.table);
  const dim3 gred(E, (d + 255) / 256 < 8 ? (d + 255) / 256 : 8);
  if (dtype == kDtypeBf16) {
    if (dx)
      hipLaunchKernelGGL(route_bwd_dx_kernel<bf16_t>, gdx, dim3(256), 0, s,
                         static_cast<const bf16_t*>(w_router), ids, dl, T_, slots, d, accumulate_dx,
                         static_cast<bf16_t*>(dx));
    if (dw_router && renorm) {
      hipLaunchKernelGGL((route_bwd_dw_seg_kernel<bf16_t, 1>), dim3(m), dim3(256), 0, s,
                         static_cast<const bf16_t*>(x), dl, row_src, tw.table, tw.n_entries, k, d,
                         part, part_b);
      hipLaunchKernelGGL(route_bwd_dw_reduce_kernel, gred, dim3(256), 0, s, part, part_b,
                         tw.table, tw.n_entries, E, d, dw_router, dbias);
    } else if (dw_router) {
      hipLaunchKernelGGL(route_bwd_dw_kernel<bf16_t>, gdw, dim3(256), 0, s,
                         static_cast<const bf16_t*>(x), dl, T_, E, d,
                         dw_router, dbias);
    }
  } else {
    if (dx)
      hipLaunchKernelGGL(route_bwd_dx_kernel<float>, gdx, dim3(256), 0, s,
                         static_cast<const float*>(w_router), ids, dl, T_, slots, d, accumulate_dx,
                         static_cast<float*>(dx));
    if (dw_router && renorm) {
      hipLaunchKernelGGL((route_bwd_dw_seg_kernel<float, 1>), dim3(m), dim3(256), 0, s,
                         static_cast<const float*>(x), dl, row_src, tw.table, tw.n_entries, k, d,
                         part, part_b);
      hipLaunchKernelGGL(route_bwd_dw_reduce_kernel, gred, dim3(256), 0, s, part, part_b,
                         tw.table, tw.n_entries, E, d, dw_router, dbias);
    } else if (dw_router) {
      hipLaunchKernelGGL(route_bwd_dw_kernel<float>, gdw, dim3(256), 0, s,
                         static_cast<const float*>(x), dl, T_, E, d,
                         dw_router, dbias);
    }
  }
  return hipGetLastError();
}

}  // namespace laep
