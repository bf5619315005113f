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
// then starts at the scan.  Up to 32768 masks (e.g. 8192 tokens over 64
// experts) the scan and the scatter are one kernel: every workgroup sums the
// masks itself (L2-resident, at most 256 KB) into the expert totals, their
// exclusive scan and its own first base, so no single-workgroup scan and no
// launch sits between them.  Beyond that, and beyond 512 wave tiles, the scan
// runs in two levels: partial sums per block of 64 tiles, one workgroup over
// the blocks, then each block's tile bases.
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

// ---- small T·E: scan and scatter in one kernel ----------------------------------
constexpr int kFusedMasks = 32768;
constexpr int kCountWT = kCountThreads / 64;  // wave tiles per workgroup
constexpr int kPreSlots = 8;                  // routing slots per token loaded up front

// Workgroup b takes wave tiles 4b .. 4b+3 (wave i, tile 4b+i, lane = token).
//  1. thread (c, e) sums popc(masks[w][e]) over chunk c of all tiles, and over
//     the tiles before 4b; it keeps the masks of the workgroup's own tiles;
//  2. expert totals, their exclusive scan (wave prefix sums + wave totals),
//     and base[4b][e] = offset[e] + the slots of e in earlier tiles;
//  3. the bases of the four tiles, then the scatter as in count_scatter_kernel.
// Workgroup 0 also writes counts, offsets and the expert-token accumulator.
__global__ __launch_bounds__(kCountThreads) void count_scan_scatter_kernel(
    const int32_t* __restrict__ idx, int n_tok, int k, int E, int E_pad, int n_wt,
    const uint64_t* __restrict__ masks, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int64_t* __restrict__ etn, int32_t* __restrict__ dest_row,
    int32_t* __restrict__ row_src) {
  __shared__ int s_tot[kCountThreads];
  __shared__ int s_pre[kCountThreads];
  __shared__ int s_wsum[kCountWT];
  __shared__ int s_base[kCountWT][256];
  __shared__ uint64_t s_mask[kCountWT][256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int w0 = blockIdx.x * kCountWT;

  // the scatter's expert ids, loaded first so they arrive during the counting
  const int wt = w0 + wave;
  const int t = wt * 64 + lane;
  const bool tok_ok = wt < n_wt && t < n_tok;
  int e_pre[kPreSlots];
#pragma unroll
  for (int j = 0; j < kPreSlots; ++j)
    e_pre[j] = (tok_ok && j < k) ? idx[(size_t)t * k + j] : -1;

  // 1.
  const int nc = kCountThreads / E_pad;
  const int c = tid / E_pad, e = tid % E_pad;
  const int per = (n_wt + nc - 1) / nc;
  const int lo = min(c * per, n_wt), hi = min(lo + per, n_wt);
  int tot = 0, pre = 0;
  if (e < E) {
    // batches of 32 loads in flight (one batch at 8192 tokens over 64 experts)
    for (int w = lo; w < hi; w += 32) {
      uint64_t m[32];
#pragma unroll
      for (int u = 0; u < 32; ++u) m[u] = w + u < hi ? masks[(size_t)(w + u) * E + e] : 0ull;
#pragma unroll
      for (int u = 0; u < 32; ++u) {
        const int n = __popcll(m[u]);
        const int wu = w + u;
        tot += n;
        pre += wu < w0 ? n : 0;
        if (wu < hi && wu >= w0 && wu < w0 + kCountWT) s_mask[wu - w0][e] = m[u];
      }
    }
  }
  s_tot[tid] = tot;
  s_pre[tid] = pre;
  __syncthreads();

  // 2.
  int te = 0, pe = 0;
  if (tid < E) {
    for (int cc = 0; cc < nc; ++cc) {
      te += s_tot[cc * E_pad + tid];
      pe += s_pre[cc * E_pad + tid];
    }
  }
  int inc = te;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(inc, o);
    inc += lane >= o ? v : 0;
  }
  if (lane == 63) s_wsum[wave] = inc;
  __syncthreads();
  int before = 0;
  for (int wv = 0; wv < wave; ++wv) before += s_wsum[wv];
  const int off = before + inc - te;  // exclusive scan of the expert totals
  if (tid < E) {
    if (blockIdx.x == 0) {
      counts[tid] = te;
      offsets[tid] = off;
      if (etn != nullptr) etn[tid] += te;
      if (tid == E - 1) offsets[E] = off + te;
    }
    // 3.
    int run = off + pe;
#pragma unroll
    for (int i = 0; i < kCountWT; ++i) {
      s_base[i][tid] = run;
      run += w0 + i < n_wt ? __popcll(s_mask[i][tid]) : 0;
    }
  }
  __syncthreads();

  if (!tok_ok) return;
  const uint64_t lt = lanemask_lt();
  auto place = [&](int j, int raw) {
    const size_t s = (size_t)t * k + j;
    const int ev = valid_expert(raw, E);
    int dst = -1;
    if (ev >= 0) {
      dst = s_base[wave][ev] + __popcll(s_mask[wave][ev] & lt);
      if (row_src != nullptr) row_src[dst] = (int32_t)s;
    }
    dest_row[s] = dst;
  };
#pragma unroll
  for (int j = 0; j < kPreSlots; ++j)
    if (j < k) place(j, e_pre[j]);
  for (int j = kPreSlots; j < k; ++j) place(j, idx[(size_t)t * k + j]);
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
  if (n_wt <= kLargeTiles && (int64_t)n_wt * E <= kFusedMasks) {
    const int gb = n_wt > 0 ? blocks : 1;  // one workgroup still writes counts and offsets
    hipLaunchKernelGGL(count_scan_scatter_kernel, dim3(gb), dim3(kCountThreads), 0, s, idx, T, k,
                       E, E_pad, n_wt, masks, counts, offsets, etn, dest_row, row_src);
    return hipGetLastError();
  }
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
