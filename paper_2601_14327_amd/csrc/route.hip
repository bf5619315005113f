// Router scoring and top-k gating (moe_route).
//
// One workgroup of 512 threads handles 32 tokens.
//  1. logits[32 x EP] = x_tile . W_r^T on the matrix cores.  The reduction
//     dimension is split over the 8 waves (chunks of consecutive 16-wide
//     k-steps dealt round robin); each wave holds a 32 x 32 fp32 block per 32
//     experts.  The eight partial blocks are summed through LDS in wave
//     order, so the result is deterministic.
//  2. top-k: 8 lanes per token, each lane owning experts e = 8q + lane.  k
//     passes of a (value desc, index asc) arg-max across the 8 lanes.  The
//     slot order is descending logit, ties to the lower expert index.
//  3. gates: exp(l_j - l_max) divided by the sum over the selected k
//     (renorm) or over all alive experts.
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kRouteTokens = 32;
constexpr int kRouteWaves = 8;
constexpr int kRouteThreads = 64 * kRouteWaves;
constexpr int kTopkThreads = 8 * kRouteTokens;  // 8 lanes per token

// One k-step of the router GEMM for element type T.
//   bf16: 16 k per step; lane loads 8 consecutive k (16 bytes) of its row.
//   f32 :  8 k per step; lane loads 4 consecutive k, fed to 4 MFMA 32x32x2.
template <typename T> struct RouterStep;

template <> struct RouterStep<bf16_t> {
  static constexpr int kK = 16;
  static constexpr int kLaneK = 8;
  __device__ static __forceinline__ void mma(f32x16_t& acc, u32x4_t a, u32x4_t b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
};

template <> struct RouterStep<float> {
  static constexpr int kK = 8;
  static constexpr int kLaneK = 4;
  __device__ static __forceinline__ void mma(f32x16_t& acc, u32x4_t a, u32x4_t b) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[i]), __uint_as_float(b[i]),
                                                 acc, 0, 0, 0);
  }
};

template <typename T>
__device__ __forceinline__ u32x4_t load16_or_zero(const T* p, bool ok) {
  u32x4_t v = {0u, 0u, 0u, 0u};
  if (ok) v = *reinterpret_cast<const u32x4_t*>(p);
  return v;
}

template <typename T, int NB>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(
    const T* __restrict__ x, const T* __restrict__ w, const float* __restrict__ bias,
    const uint8_t* __restrict__ alive, int n_tok, int d, int E, int k, int renorm,
    float* __restrict__ logits_out, int32_t* __restrict__ idx_out,
    float* __restrict__ gate_out) {
  constexpr int EP = 32 * NB;        // experts padded to 32
  constexpr int LD = EP + 1;         // LDS row stride (floats)
  constexpr int EPL = EP / 8;        // experts owned per top-k lane
  using Step = RouterStep<T>;

  __shared__ float s_log[kRouteTokens * LD];
  __shared__ float s_bias[EP];
  __shared__ uint8_t s_alive[EP];

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int t0 = blockIdx.x * kRouteTokens;

  for (int e = tid; e < EP; e += kRouteThreads) {
    s_bias[e] = (bias != nullptr && e < E) ? bias[e] : 0.0f;
    s_alive[e] = (e < E) ? (alive == nullptr ? 1 : (alive[e] != 0)) : 0;
  }

  // ---- 1. router GEMM -----------------------------------------------------
  f32x16_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.0f;

  const int row = lane & 31;
  const int kh = lane >> 5;
  const int tok = t0 + row;
  const bool tok_ok = tok < n_tok;
  const T* xrow = x + (size_t)(tok_ok ? tok : 0) * d;
  const int n_steps = (d + Step::kK - 1) / Step::kK;
  // The reduction is cut into chunks of U consecutive k-steps dealt round
  // robin to the waves.  A chunk's loads are all issued before its MFMAs,
  // so each wave keeps U row loads of x in flight (the router GEMM is
  // bound by reading x once from HBM).
  constexpr int U = NB >= 8 ? 2 : (NB >= 4 ? 4 : 8);
  for (int c = wave; c * U < n_steps; c += kRouteWaves) {
    u32x4_t a[U];
    u32x4_t b[U][NB];
#pragma unroll
    for (int i = 0; i < U; ++i) {
      const int kk = (c * U + i) * Step::kK + kh * Step::kLaneK;
      const bool k_ok = kk < d;  // d % 8 == 0: a lane's k-group is all in or all out
      a[i] = load16_or_zero(xrow + kk, tok_ok && k_ok);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int e = nb * 32 + row;
        b[i][nb] = load16_or_zero(w + (size_t)(e < E ? e : 0) * d + kk, k_ok && e < E);
      }
    }
#pragma unroll
    for (int i = 0; i < U; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) Step::mma(acc[nb], a[i], b[i][nb]);
  }

  // acc[nb][r]: token (r/4)*8 + kh*4 + r%4, expert nb*32 + row.
  for (int wv = 0; wv < kRouteWaves; ++wv) {
    __syncthreads();
    if (wave == wv) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int t = (r >> 2) * 8 + kh * 4 + (r & 3);
          const int e = nb * 32 + row;
          float* dst = &s_log[t * LD + e];
          *dst = (wv == 0) ? acc[nb][r] : (*dst + acc[nb][r]);
        }
    }
  }
  __syncthreads();

  // bias, optional logits output
  for (int i = tid; i < kRouteTokens * EP; i += kRouteThreads) {
    const int t = i / EP, e = i % EP;
    s_log[t * LD + e] += s_bias[e];
  }
  __syncthreads();
  if (logits_out != nullptr) {
    for (int i = tid; i < kRouteTokens * E; i += kRouteThreads) {
      const int t = i / E, e = i % E;
      if (t0 + t < n_tok)
        logits_out[(size_t)(t0 + t) * E + e] = s_alive[e] ? s_log[t * LD + e] : -INFINITY;
    }
  }

  // ---- 2. top-k (the first 256 threads; the others idle through it) -----------
  const bool tk = tid < kTopkThreads;
  const int ti = tk ? (tid >> 3) : 0;  // token within the tile
  const int g = tid & 7;               // lane within the token's group of 8
  float v[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * 8 + g;
    v[q] = (tk && s_alive[e]) ? s_log[ti * LD + e] : -INFINITY;
  }
  __syncthreads();  // s_log is reused below for the gate numerators

  // row maximum and (renorm == 0) the softmax denominator over alive experts
  float vmax = -INFINITY;
#pragma unroll
  for (int q = 0; q < EPL; ++q) vmax = fmaxf(vmax, v[q]);
#pragma unroll
  for (int off = 1; off < 8; off <<= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, off, 8));
  const bool none_alive = (vmax == -INFINITY);
  float s_all = 0.0f;
  if (!none_alive) {
#pragma unroll
    for (int q = 0; q < EPL; ++q)
      if (v[q] != -INFINITY) s_all += expf(v[q] - vmax);
  }
#pragma unroll
  for (int off = 1; off < 8; off <<= 1) s_all += __shfl_xor(s_all, off, 8);

  float* s_ex = s_log;  // [32][k] gate numerators (k <= E <= EP < LD)
  const int t_glob = t0 + ti;
  const bool write_ok = tk && t_glob < n_tok;
  float s_sel = 0.0f;
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int be = 0x7FFFFFFF;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const int e = q * 8 + g;
      if (v[q] > bv) { bv = v[q]; be = e; }  // ascending e: strict keeps the lower index
    }
#pragma unroll
    for (int off = 1; off < 8; off <<= 1) {
      const float ov = __shfl_xor(bv, off, 8);
      const int oe = __shfl_xor(be, off, 8);
      if (ov > bv || (ov == bv && oe < be)) { bv = ov; be = oe; }
    }
    const bool found = (bv != -INFINITY);
    if (found && (be & 7) == g) {
#pragma unroll
      for (int q = 0; q < EPL; ++q)
        if (q * 8 + g == be) v[q] = -INFINITY;
    }
    const float ex = found ? expf(bv - vmax) : 0.0f;
    s_sel += ex;
    if (tk && g == 0) {
      s_ex[ti * k + j] = ex;
      if (write_ok) idx_out[(size_t)t_glob * k + j] = found ? be : -1;
    }
  }
  __syncthreads();
  const float denom = renorm ? s_sel : s_all;
  const float inv_ok = (denom > 0.0f) ? 1.0f : 0.0f;
  if (write_ok) {
    for (int j = g; j < k; j += 8) {
      const float ex = s_ex[ti * k + j];
      gate_out[(size_t)t_glob * k + j] = inv_ok * (ex / (denom > 0.0f ? denom : 1.0f));
    }
  }
}

template <typename T>
hipError_t launch_route_t(const void* x, const void* w, const float* bias, const uint8_t* alive,
                          int T_, int d, int E, int k, int renorm, float* logits, int32_t* idx,
                          float* gate, hipStream_t s) {
  const int nb = (E + 31) / 32;
  dim3 grid((T_ + kRouteTokens - 1) / kRouteTokens), block(kRouteThreads);
  const T* xp = static_cast<const T*>(x);
  const T* wp = static_cast<const T*>(w);
#define LAEP_ROUTE_CASE(N)                                                                    \
  case N:                                                                                     \
    hipLaunchKernelGGL((route_kernel<T, N>), grid, block, 0, s, xp, wp, bias, alive, T_, d, E, \
                       k, renorm, logits, idx, gate);                                         \
    break;
  switch (nb) {
    LAEP_ROUTE_CASE(1)
    LAEP_ROUTE_CASE(2)
    LAEP_ROUTE_CASE(3)
    LAEP_ROUTE_CASE(4)
    LAEP_ROUTE_CASE(5)
    LAEP_ROUTE_CASE(6)
    LAEP_ROUTE_CASE(7)
    LAEP_ROUTE_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef LAEP_ROUTE_CASE
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const void* x, const void* w, const float* bias, const uint8_t* alive,
                        int dtype, int T_, int d, int E, int k, int renorm, float* logits,
                        int32_t* idx, float* gate, hipStream_t s) {
  if (T_ == 0) return hipSuccess;
  if (dtype == kDtypeBf16)
    return launch_route_t<bf16_t>(x, w, bias, alive, T_, d, E, k, renorm, logits, idx, gate, s);
  return launch_route_t<float>(x, w, bias, alive, T_, d, E, k, renorm, logits, idx, gate, s);
}

}  // namespace laep
