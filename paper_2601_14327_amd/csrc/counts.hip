// Per-expert token loads, offsets and the stable dispatch permutation
// (moe_expert_counts).  No atomics: three passes over 64-token wave tiles.
//
//  1. masks:  for every wave tile w and expert e, the 64-bit ballot of the
//     tokens of w routed to e (a token never repeats an expert, so one bit
//     per token suffices).
//  2. scan:   counts[e] = sum_w popc(masks[w][e]); offsets = exclusive scan;
//     base[w][e] = offsets[e] + sum_{w' < w} popc(masks[w'][e]).
//  3. scatter: dest_row[t*k + j] = base[w][e] + popc(masks[w][e] & lanes < t),
//     i.e. rows grouped by expert, ordered by token inside a group.
// The router can write the masks itself (moe_route_count); the counting pass
// then starts at the scan.  Beyond 512 wave tiles the scan runs in two
// levels: partial sums per block of 64 tiles, one workgroup over the blocks,
// then each block's tile bases.
#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

constexpr int kCountThreads = 256;  // 4 wave tiles per workgroup
constexpr int kScanThreads = 1024;

__device__ __forceinline__ int valid_expert(int e, int E) { return (e >= 0 && e < E) ? e : -1; }

__global__ __launch_bounds__(kCountThreads) void count_masks_kernel(
    const int32_t* __restrict__ idx, int n_tok, int k, int E, int n_wt,
    uint64_t* __restrict__ masks) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * (kCountThreads / 64) + (threadIdx.x >> 6);
  if (w >= n_wt) return;  // whole wave exits together
  const int t = w * 64 + lane;
  uint64_t bits0 = 0, bits1 = 0, bits2 = 0, bits3 = 0;
  if (t < n_tok) {
    for (int j = 0; j < k; ++j) {
      const int e = valid_expert(idx[(size_t)t * k + j], E);
      if (e < 0) continue;
      const uint64_t b = 1ull << (e & 63);
      const int q = e >> 6;
      if (q == 0) bits0 |= b; else if (q == 1) bits1 |= b; else if (q == 2) bits2 |= b; else bits3 |= b;
    }
  }
  uint64_t* out = masks + (size_t)w * E;
  for (int e = 0; e < E; ++e) {
    const int q = e >> 6;
    const uint64_t mine = q == 0 ? bits0 : q == 1 ? bits1 : q == 2 ? bits2 : bits3;
    const uint64_t b = __ballot((mine >> (e & 63)) & 1ull);
    if (lane == (e & 63)) out[e] = b;
  }
}

// Single workgroup: thread (c, e) owns column e of wave-tile chunk c.
__global__ __launch_bounds__(kScanThreads) void count_scan_kernel(
    const uint64_t* __restrict__ masks, int n_wt, int E, int E_pad, int32_t* __restrict__ base,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int64_t* __restrict__ etn) {
  __shared__ int s_part[kScanThreads];
  __shared__ int s_off[257];  // at most 256 experts + the total
  const int tid = threadIdx.x;
  const int n_chunks = kScanThreads / E_pad;
  const int c = tid / E_pad;
  const int e = tid % E_pad;
  const int per = (n_wt + n_chunks - 1) / n_chunks;
  const int w_lo = c * per;
  const int w_hi = min(n_wt, w_lo + per);
  int part = 0;
  if (e < E)
    for (int w = w_lo; w < w_hi; ++w) part += __popcll(masks[(size_t)w * E + e]);
  s_part[tid] = part;
  __syncthreads();
  if (tid < E_pad) {
    int tot = 0;
    for (int cc = 0; cc < n_chunks; ++cc) tot += s_part[cc * E_pad + tid];
    s_off[tid] = (tid < E) ? tot : 0;
  }
  __syncthreads();
  if (tid == 0) {  // exclusive scan over at most 256 experts
    int run = 0;
    for (int i = 0; i < E; ++i) {
      const int cnt = s_off[i];
      s_off[i] = run;
      run += cnt;
    }
    s_off[E] = run;
  }
  __syncthreads();
  if (tid < E) {
    const int cnt = s_off[tid + 1] - s_off[tid];
    counts[tid] = cnt;
    offsets[tid] = s_off[tid];
    if (etn != nullptr) etn[tid] += cnt;
  }
  if (tid == 0) offsets[E] = s_off[E];
  if (e < E) {
    int run = s_off[e];
    for (int cc = 0; cc < c; ++cc) run += s_part[cc * E_pad + e];
    for (int w = w_lo; w < w_hi; ++w) {
      base[(size_t)w * E + e] = run;
      run += __popcll(masks[(size_t)w * E + e]);
    }
  }
}

// ---- large T: the scan in two levels -------------------------------------------
// Blocks of kTilesPerBlk wave tiles.  Thread (c, e) of a 256-thread block owns
// expert e in the c-th chunk of the block's tiles.
constexpr int kTilesPerBlk = 64;
constexpr int kLargeTiles = 512;  // more wave tiles than this: two-level scan

__device__ __forceinline__ void blk_chunk(int n_wt, int E_pad, int& c, int& e, int& w_lo,
                                          int& w_hi) {
  const int nc = kCountThreads / E_pad;               // chunks per block (E_pad <= 256)
  const int per = (kTilesPerBlk + nc - 1) / nc;
  c = threadIdx.x / E_pad;
  e = threadIdx.x % E_pad;
  const int b0 = blockIdx.x * kTilesPerBlk;
  w_lo = min(b0 + c * per, b0 + kTilesPerBlk);
  w_hi = min(min(w_lo + per, b0 + kTilesPerBlk), n_wt);
}

// partial[blk][e] = routed slots of expert e in the block's tiles
__global__ __launch_bounds__(kCountThreads) void count_partial_kernel(
    const uint64_t* __restrict__ masks, int n_wt, int E, int E_pad, int32_t* __restrict__ partial) {
  __shared__ int s_part[kCountThreads];
  int c, e, w_lo, w_hi;
  blk_chunk(n_wt, E_pad, c, e, w_lo, w_hi);
  int part = 0;
  if (e < E)
    for (int w = w_lo; w < w_hi; ++w) part += __popcll(masks[(size_t)w * E + e]);
  s_part[threadIdx.x] = part;
  __syncthreads();
  if (c == 0 && e < E) {
    int tot = 0;
    for (int cc = 0; cc < kCountThreads / E_pad; ++cc) tot += s_part[cc * E_pad + e];
    partial[(size_t)blockIdx.x * E + e] = tot;
  }
}

// Single workgroup over the block partials: counts, offsets, etn and
// blk_base[blk][e] = offsets[e] + slots of e in the blocks before blk.
__global__ __launch_bounds__(kScanThreads) void count_scan_blocks_kernel(
    const int32_t* __restrict__ partial, int n_blk, int E, int E_pad, int32_t* __restrict__ blk_base,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int64_t* __restrict__ etn) {
  __shared__ int s_part[kScanThreads];
  __shared__ int s_off[257];
  const int tid = threadIdx.x;
  const int n_chunks = kScanThreads / E_pad;
  const int c = tid / E_pad;
  const int e = tid % E_pad;
  const int per = (n_blk + n_chunks - 1) / n_chunks;
  const int b_lo = c * per;
  const int b_hi = min(n_blk, b_lo + per);
  int part = 0;
  if (e < E)
    for (int b = b_lo; b < b_hi; ++b) part += partial[(size_t)b * E + e];
  s_part[tid] = part;
  __syncthreads();
  if (tid < E_pad) {
    int tot = 0;
    for (int cc = 0; cc < n_chunks; ++cc) tot += s_part[cc * E_pad + tid];
    s_off[tid] = (tid < E) ? tot : 0;
  }
  __syncthreads();
  if (tid == 0) {  // exclusive scan over at most 256 experts
    int run = 0;
    for (int i = 0; i < E; ++i) {
      const int cnt = s_off[i];
      s_off[i] = run;
      run += cnt;
    }
    s_off[E] = run;
  }
  __syncthreads();
  if (tid < E) {
    const int cnt = s_off[tid + 1] - s_off[tid];
    counts[tid] = cnt;
    offsets[tid] = s_off[tid];
    if (etn != nullptr) etn[tid] += cnt;
  }
  if (tid == 0) offsets[E] = s_off[E];
  if (e < E) {
    int run = s_off[e];
    for (int cc = 0; cc < c; ++cc) run += s_part[cc * E_pad + e];
    for (int b = b_lo; b < b_hi; ++b) {
      blk_base[(size_t)b * E + e] = run;
      run += partial[(size_t)b * E + e];
    }
  }
}

// base[w][e] inside each block: the block's base plus the tiles before w
__global__ __launch_bounds__(kCountThreads) void count_base_kernel(
    const uint64_t* __restrict__ masks, int n_wt, int E, int E_pad,
    const int32_t* __restrict__ blk_base, int32_t* __restrict__ base) {
  __shared__ int s_part[kCountThreads];
  int c, e, w_lo, w_hi;
  blk_chunk(n_wt, E_pad, c, e, w_lo, w_hi);
  int part = 0;
  if (e < E)
    for (int w = w_lo; w < w_hi; ++w) part += __popcll(masks[(size_t)w * E + e]);
  s_part[threadIdx.x] = part;
  __syncthreads();
  if (e < E) {
    int run = blk_base[(size_t)blockIdx.x * E + e];
    for (int cc = 0; cc < c; ++cc) run += s_part[cc * E_pad + e];
    for (int w = w_lo; w < w_hi; ++w) {
      base[(size_t)w * E + e] = run;
      run += __popcll(masks[(size_t)w * E + e]);
    }
  }
}

__global__ __launch_bounds__(kCountThreads) void count_scatter_kernel(
    const int32_t* __restrict__ idx, int n_tok, int k, int E, int n_wt,
    const uint64_t* __restrict__ masks, const int32_t* __restrict__ base,
    int32_t* __restrict__ dest_row, int32_t* __restrict__ row_src) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * (kCountThreads / 64) + (threadIdx.x >> 6);
  if (w >= n_wt) return;
  const int t = w * 64 + lane;
  if (t >= n_tok) return;
  const uint64_t lt = lanemask_lt();
  for (int j = 0; j < k; ++j) {
    const size_t s = (size_t)t * k + j;
    const int e = valid_expert(idx[s], E);
    int dst = -1;
    if (e >= 0) {
      const size_t m = (size_t)w * E + e;
      dst = base[m] + __popcll(masks[m] & lt);
      if (row_src != nullptr) row_src[dst] = (int32_t)s;
    }
    dest_row[s] = dst;
  }
}

}  // namespace

size_t counts_ws_bytes(int T, int k, int E) {
  (void)k;
  const size_t n_wt = (size_t)(T + 63) / 64;
  const size_t n_blk = (n_wt + kTilesPerBlk - 1) / kTilesPerBlk;
  return align_up(n_wt * E * sizeof(uint64_t), 256) + align_up(n_wt * E * sizeof(int32_t), 256) +
         2 * align_up(n_blk * E * sizeof(int32_t), 256);  // block partials and bases
}

uint32_t* counts_masks(void* ws) { return static_cast<uint32_t*>(ws); }

hipError_t launch_counts(const int32_t* idx, int T, int k, int E, int32_t* counts,
                         int32_t* offsets, int32_t* dest_row, int32_t* row_src, int64_t* etn,
                         void* ws, hipStream_t s, bool masks_ready) {
  const int n_wt = (T + 63) / 64;
  uint64_t* masks = static_cast<uint64_t*>(ws);
  int32_t* base = reinterpret_cast<int32_t*>(static_cast<char*>(ws) +
                                             align_up((size_t)n_wt * E * sizeof(uint64_t), 256));
  int E_pad = 1;
  while (E_pad < E) E_pad <<= 1;
  const int wt_per_block = kCountThreads / 64;
  const int blocks = (n_wt + wt_per_block - 1) / wt_per_block;
  if (n_wt > 0 && !masks_ready)
    hipLaunchKernelGGL(count_masks_kernel, dim3(blocks), dim3(kCountThreads), 0, s, idx, T, k, E,
                       n_wt, masks);
  if (n_wt > kLargeTiles) {
    const int n_blk = (n_wt + kTilesPerBlk - 1) / kTilesPerBlk;
    int32_t* partial = reinterpret_cast<int32_t*>(
        reinterpret_cast<char*>(base) + align_up((size_t)n_wt * E * sizeof(int32_t), 256));
    int32_t* blk_base = reinterpret_cast<int32_t*>(
        reinterpret_cast<char*>(partial) + align_up((size_t)n_blk * E * sizeof(int32_t), 256));
    hipLaunchKernelGGL(count_partial_kernel, dim3(n_blk), dim3(kCountThreads), 0, s, masks, n_wt,
                       E, E_pad, partial);
    hipLaunchKernelGGL(count_scan_blocks_kernel, dim3(1), dim3(kScanThreads), 0, s, partial, n_blk,
                       E, E_pad, blk_base, counts, offsets, etn);
    hipLaunchKernelGGL(count_base_kernel, dim3(n_blk), dim3(kCountThreads), 0, s, masks, n_wt, E,
                       E_pad, blk_base, base);
  } else {
    hipLaunchKernelGGL(count_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, masks, n_wt, E,
                       E_pad, base, counts, offsets, etn);
  }
  if (n_wt > 0)
    hipLaunchKernelGGL(count_scatter_kernel, dim3(blocks), dim3(kCountThreads), 0, s, idx, T, k, E,
                       n_wt, masks, base, dest_row, row_src);
  return hipGetLastError();
}

}  // namespace laep
