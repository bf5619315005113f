// Device-side tile tables of the grouped GEMMs.  Built from the expert
// offsets on the GPU, so the host never learns the per-expert row counts.
#pragma once

#include "common.hpp"
#include "internal.hpp"

namespace laep {
namespace {

struct TileEntry {
  int row0;    // first routed row of the expert (ragged) / K base (wgrad)
  int rows;    // rows in this tile (ragged) / rows of the expert (wgrad)
  int expert;  // logical expert
  int phys;    // weight slot
  int nt;      // output column block (per-tile lists only)
};

// ---------------------------------------------------------------------------
// Tile tables
// ---------------------------------------------------------------------------
constexpr int kTableThreads = 256;
// ints into a table's 256-byte header (n_entries at 0): eight per-XCD tile
// counters of the persistent forward products
constexpr int kTileCtrOffset = 16;


__device__ __forceinline__ int block_excl_scan_256(int v, int* s_tmp) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int n = __shfl_up(inc, off, 64);
    if (lane >= off) inc += n;
  }
  if (lane == 63) s_tmp[wave] = inc;
  __syncthreads();
  int pre = 0;
  for (int w = 0; w < wave; ++w) pre += s_tmp[w];
  __syncthreads();
  return pre + inc - v;
}

// mode 0: one entry per BM-row tile of every expert with rows (ragged M)
// mode 1: one entry per expert that has a weight slot, longest first (wgrad)
__global__ __launch_bounds__(kTableThreads) void build_table_kernel(
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ expert_map, int E, int BM,
    int mode, int max_entries, int* __restrict__ n_entries, TileEntry* __restrict__ table) {
  __shared__ int s_rows[kTableThreads];
  __shared__ int s_ok[kTableThreads];
  __shared__ int s_tmp[4];
  const int e = threadIdx.x;
  int rows = 0, phys = -1;
  if (e < E) {
    rows = offsets[e + 1] - offsets[e];
    phys = expert_map ? expert_map[e] : e;
  }
  int cnt;
  if (mode == 0)
    cnt = (e < E && phys >= 0 && rows > 0) ? (rows + BM - 1) / BM : 0;
  else
    cnt = (e < E && phys >= 0) ? 1 : 0;
  s_rows[e] = rows;
  s_ok[e] = cnt;
  __syncthreads();
  int start;
  if (mode == 0) {
    start = block_excl_scan_256(cnt, s_tmp);
  } else {  // rank by rows descending, then index
    start = 0;
    if (cnt)
      for (int j = 0; j < E; ++j)
        start += s_ok[j] && (s_rows[j] > rows || (s_rows[j] == rows && j < e));
  }
  if (mode == 0) {
    for (int i = 0; i < cnt; ++i) {
      const int pos = start + i;
      if (pos < max_entries) {
        TileEntry te;
        te.row0 = offsets[e] + i * BM;
        te.rows = min(BM, rows - i * BM);
        te.expert = e;
        te.phys = phys;
        te.nt = 0;
        table[pos] = te;
      }
    }
    const int total = block_excl_scan_256(cnt, s_tmp) + cnt;  // last thread holds the total
    if (e == kTableThreads - 1) *n_entries = min(total, max_entries);
  } else {
    if (cnt && start < max_entries) {
      TileEntry te;
      te.row0 = offsets[e];
      te.rows = rows;
      te.expert = e;
      te.phys = phys;
      te.nt = 0;
      table[start] = te;
    }
    int tot = block_excl_scan_256(cnt, s_tmp) + cnt;
    if (e == kTableThreads - 1) *n_entries = min(tot, max_entries);
  }
}

// Per-tile lists of two row-tile products (one launch): every (row tile,
// column block) of every expert with rows, experts in order.  Within an expert
// the tiles are rasterised in groups of `group` row tiles: column blocks in
// the middle loop, the group's row tiles innermost.  The workgroups that run
// together (a contiguous run of the list on one XCD) then touch about
// group + 32/group operand panels instead of 2 + 16 or 16 + 2, which is what
// each k-step has to bring into that XCD's L2.
struct TileList {
  int n_tiles;     // column blocks of the product
  int group;       // row tiles per rasterisation group
  int max_entries;
  int* n_entries;
  TileEntry* table;
};

__device__ __forceinline__ void grouped_tile(int i, int mt, int n_tiles, int group, int& m, int& n) {
  const int per_group = group * n_tiles;
  const int g = i / per_group, r = i % per_group;
  const int gsize = min(group, mt - g * group);  // the last group may be short
  n = r / gsize;
  m = g * group + r % gsize;
}

// One thread per tile: every workgroup recomputes the per-expert tile starts
// (E <= 256, one LDS scan) and writes the tiles of its own range of the list,
// finding each tile's expert by binary search over the starts.  Launch with
// enough workgroups to cover the larger list's max_entries.
__global__ __launch_bounds__(kTableThreads) void build_tile_lists_kernel(
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ expert_map, int E, int BM,
    TileList la, TileList lb) {
  __shared__ int s_tmp[4];
  __shared__ int s_start[kTableThreads + 1];
  __shared__ int s_mt[kTableThreads];
  __shared__ int s_phys[kTableThreads];
  __shared__ int s_row0[kTableThreads];
  __shared__ int s_rows[kTableThreads];
  const int e = threadIdx.x;
  int rows = 0, phys = -1;
  if (e < E) {
    rows = offsets[e + 1] - offsets[e];
    phys = expert_map ? expert_map[e] : e;
  }
  const int mt = (e < E && phys >= 0 && rows > 0) ? (rows + BM - 1) / BM : 0;
  s_mt[e] = mt;
  s_phys[e] = phys;
  s_row0[e] = e < E ? offsets[e] : 0;
  s_rows[e] = rows;
  for (int which = 0; which < 2; ++which) {
    const TileList& L = which == 0 ? la : lb;
    const int cnt = mt * L.n_tiles;
    const int start = block_excl_scan_256(cnt, s_tmp);  // (synchronises the block)
    s_start[e] = start;
    if (e == kTableThreads - 1) s_start[kTableThreads] = start + cnt;
    __syncthreads();
    const int total = s_start[kTableThreads];
    if (blockIdx.x == 0 && e == 0) *L.n_entries = min(total, L.max_entries);
    // the persistent products' per-XCD tile counters (kTileCtrOffset ints into
    // the table header), zeroed for the launch that follows on the stream
    if (blockIdx.x == 0 && e < 8) L.n_entries[kTileCtrOffset + e] = 0;
    const int i = blockIdx.x * kTableThreads + e;
    if (i < total && i < L.max_entries) {
      int lo = 0, hi = kTableThreads - 1;  // last expert with start <= i
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_start[mid] <= i) lo = mid;
        else hi = mid - 1;
      }
      const int x = lo;  // experts with no tiles share a start; the last of them has tiles
      int m, n;
      grouped_tile(i - s_start[x], s_mt[x], L.n_tiles, L.group, m, n);
      TileEntry te;
      te.row0 = s_row0[x] + m * BM;
      te.rows = min(BM, s_rows[x] - m * BM);
      te.expert = x;
      te.phys = s_phys[x];
      te.nt = n;
      L.table[i] = te;
    }
    __syncthreads();  // s_start is rewritten for the second list
  }
}

struct TableWs {
  int* n_entries;
  TileEntry* table;
  int max_entries;
};

inline size_t table_bytes(int max_entries) {
  return align_up(256 + (size_t)max_entries * sizeof(TileEntry), 256);
}

inline TableWs carve_table(void* base, int max_entries) {
  TableWs t;
  t.n_entries = static_cast<int*>(base);
  t.table = reinterpret_cast<TileEntry*>(static_cast<char*>(base) + 256);
  t.max_entries = max_entries;
  return t;
}

}  // namespace
}  // namespace laep
