// Router scoring and top-k gating (moe_route).
//
// One workgroup of 512 threads handles 32 tokens.
//  1. logits[32 x EP] = x_tile . W_r^T on the matrix cores.  The reduction
//     dimension is split over the 8 waves; each wave holds a 32 x 32 fp32
//     block per 32 experts.  The eight partial blocks are summed through LDS
//     in a fixed order, so the result is deterministic: in one round (all
//     eight blocks staged, each thread summing its elements over the waves)
//     where the stage buffers hold them, else as a tree.
//     bf16 with up to 128 experts: x and W_r go through LDS in chunks of 256
//     (or 128) columns by LDS-DMA, in two rings (x 5-8 stages deep, W_r two),
//     so every global request is a whole 128-byte line (in the MFMA operand
//     layout a direct load touches 32 bytes of each of 32 rows, four requests
//     per line) and several chunks of x are in flight.  Other cases load the
//     operands directly, U k-steps per chunk in flight.
//  2. top-k: 16 lanes (one DPP row) per token, lane g owning experts
//     e = 16q + g.  k passes of a (value desc, index asc) arg-max across the
//     16 lanes, exchanged by DPP lane permutations.  The slot order is
//     descending logit, ties to the lower expert index.
//  3. gates: exp(l_j - l_max) divided by the sum over the selected k
//     (renorm) or over all alive experts.
//  4. optionally (moe_route_count), the expert masks of the counting pass:
//     for each expert, the 32-bit set of this workgroup's tokens that chose
//     it, written as its half of the 64-token wave tile's mask.
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kRouteTokens = 32;
constexpr int kRouteWaves = 8;
constexpr int kRouteThreads = 64 * kRouteWaves;

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

// x and W_r chunks of KC columns staged through LDS by LDS-DMA (whole 128-byte
// lines per request), for bf16 and d % KC == 0, in two rings: NSX stages of
// x (32 token rows) and two of W_r (EP expert rows).  16-byte chunk c of
// row r of a stage sits at c ^ (r & 15).
template <int NB, int KC>
struct RouterStage {
  static constexpr int EP = 32 * NB;
  static constexpr int RB = KC * 2;          // bytes per staged row
  static constexpr int CPR = RB / 16;        // chunks per row
  static constexpr int XS = 32 * RB;         // x stage bytes
  static constexpr int WS = EP * RB;         // W_r stage bytes
  static constexpr int NCHX = 32 * CPR / kRouteThreads;  // DMA chunks per thread and stage
  static constexpr int NCHW = EP * CPR / kRouteThreads;
  static_assert(NCHX * kRouteThreads == 32 * CPR && NCHW * kRouteThreads == EP * CPR,
                "stage chunks must divide over the threads");
  static constexpr int NSW = 2;
  // x stages: as many as fit beside the two W_r stages and the logits tile,
  // at most 8
  static constexpr int LOGITS = 32 * (EP + 1) * 4;
  static constexpr int FITX = (156 * 1024 - LOGITS - NSW * WS) / XS;
  static constexpr int NSX = FITX > 8 ? 8 : FITX;
  static_assert(NSX >= 2, "at least two x stages");
  static constexpr int BYTES = NSX * XS + NSW * WS;
};

template <int NB, int KC>
struct StageBytes {
  static constexpr int value = RouterStage<NB, KC>::BYTES;
};
template <int NB>
struct StageBytes<NB, 0> {
  static constexpr int value = 16;
};

// Lane exchange inside a 16-lane DPP row (no LDS round trip): quad_perm
// [1,0,3,2] and [2,3,0,1] swap neighbours at distance 1 and 2, row_half_mirror
// and row_mirror pair lane i with 7-i and 15-i.  Applied in that order, a
// symmetric pairwise combine leaves every lane of the row with the row's result.
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
// (value desc, index asc) arg-max step
template <int CTRL>
__device__ __forceinline__ void argmax_step(float& bv, int& be) {
  const float ov = dpp_f<CTRL>(bv);
  const int oe = dpp_i<CTRL>(be);
  // bitwise, so the compiler keeps it a select rather than branches
  const bool take = (ov > bv) | ((ov == bv) & (oe < be));
  bv = take ? ov : bv;
  be = take ? oe : be;
}

// fourth word of a raw buffer resource: 32-bit data format, no swizzle
constexpr int kRouteBufferFlags = 0x00020000;

// One stage of LDS-DMA loads through buffer loads with the LDS flag: chunk i
// of this thread at byte voff[i] + soff of its operand's buffer (x or W_r,
// chosen per chunk and wave: each wave's 64 chunks lie in the same operand).
// The buffer form matters: with the global-segment form of the same copy the
// compiler cannot tell the DMA's LDS writes from the stage reads and waits
// for every load in flight (vmcnt(0)) before the reads, so no chunk's load
// overlapped another's compute.
template <int NCH, int XCH>
__device__ __forceinline__ void route_dma(char* dst, __amdgpu_buffer_rsrc_t rx,
                                          __amdgpu_buffer_rsrc_t rw, const uint32_t* voff,
                                          int soff, int wave) {
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    // chunks [0, XCH) of the stage are x rows (wave-uniform test)
    const bool is_x = i * kRouteThreads + wave * 64 < XCH;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        is_x ? rx : rw,
        (__attribute__((address_space(3))) void*)(dst + (i * kRouteThreads + wave * 64) * 16), 16,
        voff[i], soff, 0, 0);
  }
}

// A workgroup barrier ordering LDS accesses only: unlike __syncthreads it does
// not wait for this wave's global stores to be acknowledged (which costs a
// memory round trip right after the top-k writes its slots).
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int N>
__device__ __forceinline__ void route_wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <typename T, int NB, int KC>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(
    const T* __restrict__ x, const T* __restrict__ w, const float* __restrict__ bias,
    const uint8_t* __restrict__ alive, int n_tok, int d, int E, int k, int renorm,
    float* __restrict__ logits_out, int32_t* __restrict__ idx_out,
    float* __restrict__ gate_out, uint32_t* __restrict__ masks32) {
  constexpr int EP = 32 * NB;        // experts padded to 32
  constexpr int LD = EP + 1;         // LDS row stride (floats)
  constexpr int EPL = EP / 16;       // experts owned per top-k lane
  // One LDS array, carved by hand.  Separate __shared__ arrays get alias
  // scopes of their own, and the stage reads then share the LDS-DMA copies'
  // scope: the compiler would wait for every copy in flight (vmcnt(0)) before
  // each chunk's reads and serialise the stages.  The stage loop's explicit
  // waits and barriers order the copies and the reads.
  constexpr int STAGE_B = (StageBytes<NB, KC>::value + 15) / 16 * 16;
  constexpr int LOG_OFF = STAGE_B;
  constexpr int BIAS_OFF = LOG_OFF + kRouteTokens * LD * 4;
  constexpr int MASK_OFF = BIAS_OFF + EP * 4;
  constexpr int ALIVE_OFF = MASK_OFF + EP * 4;
  __shared__ __attribute__((aligned(1024))) char s_mem[ALIVE_OFF + EP];
  // LDS-staged path: the operand stages, reused for the cross-wave partial sums
  char* const s_stage = s_mem;
  float* const s_log = reinterpret_cast<float*>(s_mem + LOG_OFF);
  float* const s_bias = reinterpret_cast<float*>(s_mem + BIAS_OFF);
  uint32_t* const s_mask = reinterpret_cast<uint32_t*>(s_mem + MASK_OFF);
  uint8_t* const s_alive = reinterpret_cast<uint8_t*>(s_mem + ALIVE_OFF);

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int t0 = blockIdx.x * kRouteTokens;

  // expert e = tid (EP <= 256 < the thread count): its bias and alive flag are
  // loaded now and stored to LDS after the GEMM, so the operand loads are
  // not queued behind a round trip for them
  static_assert(EP <= kRouteThreads, "one expert per thread");
  // (the raw byte is kept: testing it here would wait for the load)
  float bias_e = 0.0f;
  uint32_t alive_raw = 1;
  if (tid < E) {
    if (bias != nullptr) bias_e = bias[tid];
    if (alive != nullptr) alive_raw = alive[tid];
  }

  // ---- 1. router GEMM -----------------------------------------------------
  f32x16_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.0f;

  const int row = lane & 31;
  const int kh = lane >> 5;
  if constexpr (KC > 0) {
    // LDS-staged: every thread fills NCHX chunks of each x stage and NCHW of
    // each W_r stage; the waves share the KC/16 k-steps of a chunk round robin.
    using St = RouterStage<NB, KC>;
    // x from the workgroup's first token (32 rows: 32-bit offsets), W_r whole
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(x + (size_t)t0 * d), 0, -1, kRouteBufferFlags);
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(w), 0, -1, kRouteBufferFlags);
    const int wave_s = __builtin_amdgcn_readfirstlane(wave);
    uint32_t voffx[St::NCHX], voffw[St::NCHW];
#pragma unroll
    for (int i = 0; i < St::NCHX; ++i) {
      const int q = i * kRouteThreads + tid;
      const int r = q / St::CPR;
      const int lc = (q % St::CPR) ^ (r & 15);
      const int t = t0 + r < n_tok ? r : n_tok - 1 - t0;
      voffx[i] = (uint32_t)(((size_t)t * d + lc * 8) * 2);
    }
#pragma unroll
    for (int i = 0; i < St::NCHW; ++i) {
      const int q = i * kRouteThreads + tid;
      const int r = q / St::CPR;
      const int lc = (q % St::CPR) ^ (r & 15);
      const int e = r < E ? r : E - 1;
      voffw[i] = (uint32_t)(((size_t)e * d + lc * 8) * 2);
    }
    const int n_chunks = d / KC;
    // Two rings.  x streams from HBM, NSX-1 chunks ahead; W_r (L2-resident)
    // one chunk ahead.  The load counter completes in issue order, so a
    // W_r chunk issued behind x's lands only after them; with x and W_r in
    // one stage (as before) that held x to the stage depth (2 chunks of x in
    // flight, 8 MB over the chip, well short of what HBM latency needs).
    // Iteration c issues x(c+NSX-1), then W(c+1), and waits for W(c): 
    // everything issued before it, x(c) .. x(c+NSX-2) included, has landed.
    // Past the end the last chunk is loaded again into the free stage (never
    // read), so one constant vmcnt serves every wait.
    constexpr int NSX = St::NSX;
    char* const s_x = s_stage;
    char* const s_w = s_stage + NSX * St::XS;
    // Workgroups on one XCD (block i runs on XCD i % 8) start at different
    // chunks, so they do not all request the same W_r lines at once.
    const int rot = (int)((blockIdx.x >> 3) % n_chunks);
    auto rotated = [&](int c) {
      const int cl = c < n_chunks ? c : n_chunks - 1;
      return cl + rot < n_chunks ? cl + rot : cl + rot - n_chunks;
    };
    auto issue_x = [&](int c) {
      route_dma<St::NCHX, St::NCHX * kRouteThreads>(s_x + (c % NSX) * St::XS, rx, rw, voffx,
                                                     rotated(c) * KC * 2, wave_s);
    };
    auto issue_w = [&](int c) {
      route_dma<St::NCHW, 0>(s_w + (c & 1) * St::WS, rx, rw, voffw, rotated(c) * KC * 2, wave_s);
    };
    static_assert(KC / 16 % kRouteWaves == 0, "every wave takes the same number of k-steps");
    constexpr int U = KC / 16 / kRouteWaves;  // k-steps per wave and chunk
#pragma unroll
    for (int c = 0; c < NSX - 1; ++c) issue_x(c);
    issue_w(0);
    for (int c = 0; c < n_chunks; ++c) {
      issue_x(c + NSX - 1);                   // into the x stage chunk c-1 used
      issue_w(c + 1);                         // into the W_r stage chunk c-1 used
      // chunk c has landed: this thread's loads (the counter), then every
      // thread's (a bare barrier: __syncthreads' fence would make the compiler
      // wait for every load in flight, the later chunks' too)
      route_wait_vmcnt<St::NCHX + St::NCHW>();
      __builtin_amdgcn_s_barrier();
      const char* sx = s_x + (c % NSX) * St::XS;
      const char* sw = s_w + (c & 1) * St::WS;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int s = wave + u * kRouteWaves;
        const int lc = 2 * s + kh;
        const u32x4_t a =
            *reinterpret_cast<const u32x4_t*>(sx + row * St::RB + ((lc ^ (row & 15)) << 4));
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int r = nb * 32 + row;
          const u32x4_t bv =
              *reinterpret_cast<const u32x4_t*>(sw + r * St::RB + ((lc ^ (r & 15)) << 4));
          RouterStep<bf16_t>::mma(acc[nb], a, bv);
        }
      }
      // every thread's reads of chunk c's stages are done: they are refilled
      // at the next iteration
      __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));  // lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
    }
    // no LDS-DMA may still be writing when the stage area is reused for the
    // partial sums: this thread's copies (the counter), then every thread's
    route_wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
  } else {
    using Step = RouterStep<T>;
    const int tok = t0 + row;
    const bool tok_ok = tok < n_tok;
    const T* xrow = x + (size_t)(tok_ok ? tok : 0) * d;
    const int n_steps = (d + Step::kK - 1) / Step::kK;
    // The reduction is cut into chunks of U consecutive k-steps dealt round
    // robin to the waves.  A chunk's loads are all issued before its MFMAs.
    constexpr int U = NB >= 5 ? 2 : (NB >= 3 ? 4 : 8);
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
  }

  // opaque to the compiler until here, so the test of the byte is not hoisted
  // next to its load (with a wait for it in front of the operand loads)
  asm volatile("" : "+v"(alive_raw));
  if (tid < EP) {  // published by the first barrier of the cross-wave sum
    s_bias[tid] = bias_e;
    s_alive[tid] = tid < E && alive_raw != 0;
    s_mask[tid] = 0u;
  }

  // ---- cross-wave sum, deterministic ----------------------------------------------
  // acc[nb][r]: token (r/4)*8 + kh*4 + r%4, expert nb*32 + row.
  auto tile_at = [&](int nb, int r, int& t, int& e) {
    t = (r >> 2) * 8 + kh * 4 + (r & 3);
    e = nb * 32 + row;
  };
  // one-round partial blocks: [wave][expert][token], rows padded to 36 floats
  // so the 16-byte writes of 8 lanes (8 experts) fall in distinct banks
  constexpr int kPartTP = 36;
  constexpr bool kOneRound =
      KC > 0 && kRouteWaves * EP * kPartTP * 4 <= StageBytes<NB, KC>::value;
  if constexpr (kOneRound) {
    // every wave's partial block to the idle stage buffers (acc[nb][4g..4g+3]
    // are tokens 8g + 4kh .. +3 of one expert: one 16-byte write), then each
    // thread sums 4 tokens of one expert over the waves in wave order and adds
    // the bias
    float* part = reinterpret_cast<float*>(s_stage);
    constexpr int SL = EP * kPartTP;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4_t v4 = {acc[nb][4 * g4], acc[nb][4 * g4 + 1], acc[nb][4 * g4 + 2],
                            acc[nb][4 * g4 + 3]};
        *reinterpret_cast<f32x4_t*>(part + wave * SL + (nb * 32 + row) * kPartTP + g4 * 8 +
                                    kh * 4) = v4;
      }
    lds_sync();
    for (int i = tid; i < EP * 8; i += kRouteThreads) {
      const int e = i >> 3, t = (i & 7) * 4;
      f32x4_t sum = *reinterpret_cast<const f32x4_t*>(part + e * kPartTP + t);
#pragma unroll
      for (int wv = 1; wv < kRouteWaves; ++wv)
        sum += *reinterpret_cast<const f32x4_t*>(part + wv * SL + e * kPartTP + t);
#pragma unroll
      for (int q = 0; q < 4; ++q) s_log[(t + q) * LD + e] = sum[q] + s_bias[e];
    }
  } else if constexpr (KC > 0) {
    // a tree over the waves (8 -> 4 -> 2 -> 1) through the idle stage buffers
    static_assert(4 * 32 * EP * 4 <= StageBytes<NB, KC>::value, "partials must fit the stages");
    float* part = reinterpret_cast<float*>(s_stage);
    constexpr int SL = 32 * EP;
    for (int half = kRouteWaves / 2; half >= 1; half >>= 1) {
      if (wave >= half && wave < 2 * half) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int t, e;
            tile_at(nb, r, t, e);
            part[(wave - half) * SL + t * EP + e] = acc[nb][r];
          }
      }
      __syncthreads();
      if (wave < half) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int t, e;
            tile_at(nb, r, t, e);
            acc[nb][r] += part[wave * SL + t * EP + e];
          }
      }
      __syncthreads();
    }
    if (wave == 0) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int t, e;
          tile_at(nb, r, t, e);
          s_log[t * LD + e] = acc[nb][r];
        }
    }
    __syncthreads();
    for (int i = tid; i < kRouteTokens * EP; i += kRouteThreads) {
      const int t = i / EP, e = i % EP;
      s_log[t * LD + e] += s_bias[e];
    }
  } else {
    for (int wv = 0; wv < kRouteWaves; ++wv) {
      __syncthreads();
      if (wave == wv) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int t, e;
            tile_at(nb, r, t, e);
            float* dst = &s_log[t * LD + e];
            *dst = (wv == 0) ? acc[nb][r] : (*dst + acc[nb][r]);
          }
      }
    }
    __syncthreads();
    for (int i = tid; i < kRouteTokens * EP; i += kRouteThreads) {
      const int t = i / EP, e = i % EP;
      s_log[t * LD + e] += s_bias[e];
    }
  }
  lds_sync();

  if (logits_out != nullptr) {
    for (int i = tid; i < kRouteTokens * E; i += kRouteThreads) {
      const int t = i / E, e = i % E;
      if (t0 + t < n_tok)
        logits_out[(size_t)(t0 + t) * E + e] = s_alive[e] ? s_log[t * LD + e] : -INFINITY;
    }
  }

  // ---- 2. top-k: 16 lanes (one DPP row) per token --------------------------------
  const int ti = tid >> 4;  // token within the tile
  const int g = tid & 15;   // lane within the token's row; owns experts e = 16 q + g
  float v[EPL];
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = q * 16 + g;
    v[q] = s_alive[e] ? s_log[ti * LD + e] : -INFINITY;
  }
  lds_sync();  // s_log is reused below for the gate numerators

  // row maximum and (renorm == 0) the softmax denominator over alive experts
  float vmax = -INFINITY;
#pragma unroll
  for (int q = 0; q < EPL; ++q) vmax = fmaxf(vmax, v[q]);
  vmax = fmaxf(vmax, dpp_f<kDppXor1>(vmax));
  vmax = fmaxf(vmax, dpp_f<kDppXor2>(vmax));
  vmax = fmaxf(vmax, dpp_f<kDppHalfMirror>(vmax));
  vmax = fmaxf(vmax, dpp_f<kDppMirror>(vmax));
  const bool none_alive = (vmax == -INFINITY);
  float s_all = 0.0f;
  if (!none_alive) {
#pragma unroll
    for (int q = 0; q < EPL; ++q)
      if (v[q] != -INFINITY) s_all += __expf(v[q] - vmax);
  }
  s_all += dpp_f<kDppXor1>(s_all);
  s_all += dpp_f<kDppXor2>(s_all);
  s_all += dpp_f<kDppHalfMirror>(s_all);
  s_all += dpp_f<kDppMirror>(s_all);

  float* s_ex = s_log;  // [32][k] gate numerators (k <= E <= EP < LD)
  const int t_glob = t0 + ti;
  const bool write_ok = t_glob < n_tok;
  float s_sel = 0.0f;
  // Up to 16 slots: pass j's result stays in lane j of the token's row.  Each
  // pass takes the largest value across the row, then the lowest expert index
  // holding it (the order of a (value desc, index asc) arg-max), on integer
  // keys that order like the floats: -0 is first made +0 and NaN -inf, so
  // equal keys are exactly equal values, and each step is one DPP max or min.
  // Taken slots get INT_MIN, below the key of -inf (a dead expert, never
  // taken: the pass then finds nothing).
  const bool by_lane = k <= 16;
  int my_e = -1;
  float my_ex = 0.0f;
  if (by_lane) {
    constexpr int kKeyNegInf = (int)(0xFF800000u ^ 0x7FFFFFFFu);
    int key[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const float f = v[q] != v[q] ? -INFINITY : v[q] + 0.0f;
      const int b = __float_as_int(f);
      key[q] = b >= 0 ? b : b ^ 0x7FFFFFFF;
    }
    for (int j = 0; j < k; ++j) {
      int m = key[0];
#pragma unroll
      for (int q = 1; q < EPL; ++q) m = max(m, key[q]);
      m = max(m, dpp_i<kDppXor1>(m));
      m = max(m, dpp_i<kDppXor2>(m));
      m = max(m, dpp_i<kDppHalfMirror>(m));
      m = max(m, dpp_i<kDppMirror>(m));
      int ce = 0x7FFFFFFF;
#pragma unroll
      for (int q = EPL - 1; q >= 0; --q) ce = key[q] == m ? q * 16 + g : ce;
      ce = min(ce, dpp_i<kDppXor1>(ce));
      ce = min(ce, dpp_i<kDppXor2>(ce));
      ce = min(ce, dpp_i<kDppHalfMirror>(ce));
      ce = min(ce, dpp_i<kDppMirror>(ce));
      const bool found = m > kKeyNegInf;
#pragma unroll
      for (int q = 0; q < EPL; ++q) key[q] = q * 16 + g == ce ? (int)0x80000000 : key[q];
      const float mv = __int_as_float(m >= 0 ? m : m ^ 0x7FFFFFFF);
      const float ex = found ? __expf(mv - vmax) : 0.0f;
      s_sel += ex;
      my_e = g == j ? (found ? ce : -1) : my_e;
      my_ex = g == j ? ex : my_ex;
    }
    if (write_ok && g < k) {
      idx_out[(size_t)t_glob * k + g] = my_e;
      if (masks32 != nullptr && my_e >= 0) atomicOr(&s_mask[my_e], 1u << ti);
    }
  } else {
    for (int j = 0; j < k; ++j) {
      float bv = -INFINITY;
      int be = 0x7FFFFFFF;
#pragma unroll
      for (int q = 0; q < EPL; ++q) {
        const int e = q * 16 + g;
        if (v[q] > bv) { bv = v[q]; be = e; }  // ascending e: strict keeps the lower index
      }
      argmax_step<kDppXor1>(bv, be);
      argmax_step<kDppXor2>(bv, be);
      argmax_step<kDppHalfMirror>(bv, be);
      argmax_step<kDppMirror>(bv, be);
      const bool found = (bv != -INFINITY);
      if (found && (be & 15) == g) {
#pragma unroll
        for (int q = 0; q < EPL; ++q)
          if (q * 16 + g == be) v[q] = -INFINITY;
      }
      const float ex = found ? __expf(bv - vmax) : 0.0f;
      s_sel += ex;
      if (g == 0) {
        s_ex[ti * k + j] = ex;
        if (write_ok) idx_out[(size_t)t_glob * k + j] = found ? be : -1;
        if (masks32 != nullptr && write_ok && found) atomicOr(&s_mask[be], 1u << ti);
      }
    }
  }
  lds_sync();  // the expert masks are complete (the slots' global stores need not be)
  if (masks32 != nullptr) {
    // mask word of (wave tile blockIdx/2, expert e): tokens 0-31 of the tile
    // in the low word, 32-63 in the high word; a last even workgroup also
    // clears the high word (no tokens there)
    const size_t wt = blockIdx.x >> 1;
    const int half = blockIdx.x & 1;
    const bool clear_hi = half == 0 && blockIdx.x == gridDim.x - 1;
    for (int e = tid; e < E; e += kRouteThreads) {
      masks32[2 * (wt * E + e) + half] = s_mask[e];
      if (clear_hi) masks32[2 * (wt * E + e) + 1] = 0u;
    }
  }
  const float denom = renorm ? s_sel : s_all;
  const float inv_ok = (denom > 0.0f) ? 1.0f : 0.0f;
  const float den = denom > 0.0f ? denom : 1.0f;
  if (write_ok) {
    if (by_lane) {
      if (g < k) gate_out[(size_t)t_glob * k + g] = inv_ok * (my_ex / den);
    } else {
      for (int j = g; j < k; j += 16)
        gate_out[(size_t)t_glob * k + j] = inv_ok * (s_ex[ti * k + j] / den);
    }
  }
}

template <typename T, int NB, int KC>
void launch_route_nb(dim3 grid, hipStream_t s, const void* x, const void* w, const float* bias,
                     const uint8_t* alive, int T_, int d, int E, int k, int renorm, float* logits,
                     int32_t* idx, float* gate, uint32_t* masks32) {
  hipLaunchKernelGGL((route_kernel<T, NB, KC>), grid, dim3(kRouteThreads), 0, s,
                     static_cast<const T*>(x), static_cast<const T*>(w), bias, alive, T_, d, E, k,
                     renorm, logits, idx, gate, masks32);
}

template <typename T>
hipError_t launch_route_t(const void* x, const void* w, const float* bias, const uint8_t* alive,
                          int T_, int d, int E, int k, int renorm, float* logits, int32_t* idx,
                          float* gate, uint32_t* masks32, hipStream_t s) {
  const int nb = (E + 31) / 32;
  const dim3 grid((T_ + kRouteTokens - 1) / kRouteTokens);
  // bf16 with up to 128 experts: LDS-staged chunks of 256 (NB <= 2) or 128 columns
  int kc = 0;
  if (sizeof(T) == 2 && nb <= 4) {
    if (nb <= 2 && d % 256 == 0) kc = 256;
    else if (d % 128 == 0) kc = 128;
  }
#define LAEP_ROUTE_ARGS grid, s, x, w, bias, alive, T_, d, E, k, renorm, logits, idx, gate, masks32
  if constexpr (sizeof(T) == 2) {
    if (kc == 256) {
      if (nb == 1) launch_route_nb<T, 1, 256>(LAEP_ROUTE_ARGS);
      else launch_route_nb<T, 2, 256>(LAEP_ROUTE_ARGS);
      return hipGetLastError();
    }
    if (kc == 128) {
      switch (nb) {
        case 1: launch_route_nb<T, 1, 128>(LAEP_ROUTE_ARGS); break;
        case 2: launch_route_nb<T, 2, 128>(LAEP_ROUTE_ARGS); break;
        case 3: launch_route_nb<T, 3, 128>(LAEP_ROUTE_ARGS); break;
        default: launch_route_nb<T, 4, 128>(LAEP_ROUTE_ARGS); break;
      }
      return hipGetLastError();
    }
  }
  switch (nb) {
    case 1: launch_route_nb<T, 1, 0>(LAEP_ROUTE_ARGS); break;
    case 2: launch_route_nb<T, 2, 0>(LAEP_ROUTE_ARGS); break;
    case 3: launch_route_nb<T, 3, 0>(LAEP_ROUTE_ARGS); break;
    case 4: launch_route_nb<T, 4, 0>(LAEP_ROUTE_ARGS); break;
    case 5: launch_route_nb<T, 5, 0>(LAEP_ROUTE_ARGS); break;
    case 6: launch_route_nb<T, 6, 0>(LAEP_ROUTE_ARGS); break;
    case 7: launch_route_nb<T, 7, 0>(LAEP_ROUTE_ARGS); break;
    case 8: launch_route_nb<T, 8, 0>(LAEP_ROUTE_ARGS); break;
    default: return hipErrorInvalidValue;
  }
#undef LAEP_ROUTE_ARGS
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const void* x, const void* w, const float* bias, const uint8_t* alive,
                        int dtype, int T_, int d, int E, int k, int renorm, float* logits,
                        int32_t* idx, float* gate, uint32_t* masks32, hipStream_t s) {
  if (T_ == 0) return hipSuccess;
  if (dtype == kDtypeBf16)
    return launch_route_t<bf16_t>(x, w, bias, alive, T_, d, E, k, renorm, logits, idx, gate,
                                  masks32, s);
  return launch_route_t<float>(x, w, bias, alive, T_, d, E, k, renorm, logits, idx, gate, masks32,
                               s);
}

}  // namespace laep
