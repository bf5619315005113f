// Shared pieces of the grouped bf16 GEMM kernels (forward and backward).
#pragma once

#include "common.hpp"
#include "internal.hpp"
#include "tiles.hpp"

namespace laep {
namespace {

enum { EPI_GU = 0, EPI_STORE = 1, EPI_WGRAD = 3 };

struct GemmParams {
  const bf16_t* A;
  long long lda;
  const bf16_t* B;
  long long ldb;
  long long strideB;  // elements between weight slots
  int N;              // output columns
  int K;              // reduction length (ragged-M products)
  int Mw;             // output rows (wgrad)
  int f;              // d_ff
  const TileEntry* table;
  const int* n_entries;
  int tiles_per_entry;
  int n_tiles_n;
  bf16_t* out;
  long long ldo;
  bf16_t* out2;
  const bf16_t* aux;
  float* wout;
  long long strideW;
  int accumulate;
  const int32_t* row_src;  // gathered A rows: row r of the product is A row row_src[r] / slots_k
  int slots_k;
  // gate-scaled scatter of the down product (one slot per token): routed row r
  // also goes to out_tok row row_src[r] / slots_k, times gate[row_src[r]]
  const float* gate;
  bf16_t* out_tok;
  int group;               // row tiles per rasterisation group (backward products)
  // weight gradient with the B operand gathered (dW_gu = dA^T X with X's
  // routed row r read from token row row_src[r] / slots_k of B): bytes of B
  uint32_t b_extent;
  uint32_t a_extent;       // bytes of dout when data-gradient 1 / dW_d form dY on load
  // weight gradient: each XCD takes one block of an expert's output tiles, the
  // tile grid cut into xcd_gm x xcd_gn blocks (xcd_gm * xcd_gn = 8; 0 = tiles
  // dealt round robin)
  int xcd_gm;
  // persistent forward products: eight per-XCD tile counters, zero at launch
  int* tile_ctr;
};

// Row tiles per rasterisation group of the tile orders (within a group the
// column blocks run in the middle loop, the group's row tiles innermost).
// Forward: groups of 4 (persistent products; against one group per expert:
// -2.3 % on 16 experts of up to 42 row tiles, -0.5 % on 64 experts of about
// 4, and 6, 8 or 16 no better).  Backward: groups of 8 row tiles (a sweep
// of 2-32 measured 2-8 alike, 16 and more slower: too many weight panels of
// column blocks in flight).
constexpr int kFwdTileGroup = 4;
constexpr int kBwdTileGroup = 8;

__device__ __forceinline__ void store_bf16x4(bf16_t* p, float a, float b, float c, float d) {
  u32x2_t w = {pack_bf16x2(a, b), pack_bf16x2(c, d)};
  *reinterpret_cast<u32x2_t*>(p) = w;
}

__device__ __forceinline__ void load_bf16x4(const bf16_t* p, float v[4]) {
  const u32x2_t w = *reinterpret_cast<const u32x2_t*>(p);
  v[0] = lo_bf16(w[0]);
  v[1] = hi_bf16(w[0]);
  v[2] = lo_bf16(w[1]);
  v[3] = hi_bf16(w[1]);
}

// 128-byte LDS rows (64 k of bf16, 8 chunks of 16 bytes): chunk c of row r
// at c ^ ((r ^ r >> 3) & 7), measured free of bank conflicts for the
// ds_read_b128 fragment reads.
__device__ __forceinline__ int swz8(int row) { return (row ^ (row >> 3)) & 7; }

typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt lgkmcnt(0) only (vmcnt field at its maximum, 63)
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// s_waitcnt vmcnt(N) lgkmcnt(0)
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

inline int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }
inline int round8(int v) { return (v + 7) & ~7; }

}  // namespace
}  // namespace laep
