// Grouped bf16 GEMMs of the SwiGLU expert FFN on the gfx950 matrix cores
// (moe_grouped_ffn_fwd / moe_grouped_ffn_bwd).
//
// One kernel template serves every product of the layer:
//   gate/up   A = X_e [M_e, d]      x W_gu[p]^T [2f, d]  -> SwiGLU epilogue (H, act_save)
//   down      A = H_e [M_e, f]      x W_d[p]^T  [d, f]   -> Y
//   dgrad 1   A = dY_e [M_e, d]     x W_d[p]    [d, f]   -> SwiGLU backward epilogue (dA, H_b)
//   dgrad 2   A = dA_e [M_e, 2f]    x W_gu[p]   [2f, d]  -> dX
//   wgrad     A = dY_e^T / dA_e^T   x H_b / X            -> fp32 dW_d[p] / dW_gu[p]
//
// Tiling: BM x BN x 64 tiles, one LDS double buffer, one barrier per k-tile.
// LDS holds both operands K-contiguous ([rows][64] bf16); 16-byte chunk c of
// row r lives at chunk c ^ ((r ^ r >> 3) & 7), which keeps both the fragment
// reads and the transposed stores free of bank conflicts.  Operands whose K
// is the strided dimension (dgrad weights, both wgrad operands) are loaded
// as 4 (k) x 8 (m) blocks and transposed in registers on the way to LDS.
//
// MFMA v_mfma_f32_32x32x16_bf16 is issued with the operands swapped
// (weights as the "A" input, tokens as the "B" input), so each lane ends up
// owning one output row and 4 consecutive output columns per register quad:
// acc[tm][tn][4q + i] = C[m = tm*32 + lane%32][n = tn*32 + 8q + 4(lane/32) + i].
//
// Ragged expert rows come from a device-side tile table built from the
// expert offsets, so the host never learns the per-expert row counts.
// Workgroup ids are remapped so that each of the 8 XCDs walks a contiguous
// range of tiles (same expert, same activation rows -> its own L2).
#include "common.hpp"
#include "internal.hpp"
#include "tiles.hpp"

#include <cstdlib>
#include <cstring>

namespace laep {
namespace {

constexpr int BK = 64;

__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }
// element offset of 16-byte chunk `chunk` of LDS row `row`
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * BK + ((chunk ^ swz(row)) << 3);
}

// ---------------------------------------------------------------------------
// Global -> LDS tile loaders
// ---------------------------------------------------------------------------
// K-contiguous operand: element (r, k) at ptr(r)[k].
template <int ROWS, int NT>
struct LoaderK {
  static constexpr int N = ROWS * 8 / NT;  // 16-byte chunks per thread
  u32x4_t r[N];
  template <class RowPtr>
  __device__ __forceinline__ void load(const RowPtr& row_ptr, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int c = tid + i * NT;
      const bf16_t* p = row_ptr(c >> 3);
      u32x4_t v = {0u, 0u, 0u, 0u};
      if (p) v = *reinterpret_cast<const u32x4_t*>(p + k0 + ((c & 7) << 3));
      r[i] = v;
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int c = tid + i * NT;
      *reinterpret_cast<u32x4_t*>(lds + lds_off(c >> 3, c & 7)) = r[i];
    }
  }
};

// Row-contiguous operand (K strided): element (r, k) at base[k * ld + r].
// Each thread moves 4 (k) x 8 (r) blocks.
template <int ROWS, int NT>
struct LoaderT {
  static constexpr int NB = 2 * ROWS / NT;
  static constexpr int RB = ROWS / 8;  // 8-row groups per tile
  u32x4_t r[NB][4];
  __device__ __forceinline__ void load(const bf16_t* base, long long ld, int k0, int k_valid,
                                       int r_valid, int tid) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int q = tid + b * NT;
      const int rb = q % RB, kb = q / RB;
      const bool r_ok = rb * 8 < r_valid;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = k0 + kb * 4 + i;
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (r_ok && k < k_valid)
          v = *reinterpret_cast<const u32x4_t*>(base + (size_t)k * ld + rb * 8);
        r[b][i] = v;
      }
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds, int tid) const {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int q = tid + b * NT;
      const int rb = q % RB, kb = q / RB;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int sh = (j & 1) * 16;
        const int dw = j >> 1;
        const uint32_t e0 = (r[b][0][dw] >> sh) & 0xFFFFu;
        const uint32_t e1 = (r[b][1][dw] >> sh) & 0xFFFFu;
        const uint32_t e2 = (r[b][2][dw] >> sh) & 0xFFFFu;
        const uint32_t e3 = (r[b][3][dw] >> sh) & 0xFFFFu;
        u32x2_t w = {e0 | (e1 << 16), e2 | (e3 << 16)};
        const int row = rb * 8 + j;
        *reinterpret_cast<u32x2_t*>(lds + lds_off(row, kb >> 1) + ((kb & 1) << 2)) = w;
      }
    }
  }
};

// ---------------------------------------------------------------------------
// Kernel
// ---------------------------------------------------------------------------
enum { EPI_GU = 0, EPI_STORE = 1, EPI_GU_BWD = 2, EPI_WGRAD = 3 };

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
};

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

template <int BM, int BN, int NWM, int NWN, int EPI, bool A_T, bool B_T, bool GU_ROWS>
__global__ __launch_bounds__(64 * NWM * NWN) void grouped_gemm_kernel(GemmParams p) {
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(EPI != EPI_GU || (TN % 2 == 0), "SwiGLU epilogue pairs gate/up blocks");
  constexpr int STAGE = (BM + BN) * BK;
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * STAGE];

  // ---- tile schedule (XCD-contiguous) --------------------------------------
  const int n_valid = (*p.n_entries) * p.tiles_per_entry;
  const int per = (n_valid + 7) >> 3;
  const int slot = blockIdx.x >> 3;
  if (slot >= per) return;
  const int L = (blockIdx.x & 7) * per + slot;
  if (L >= n_valid) return;
  const TileEntry te = p.table[L / p.tiles_per_entry];
  const int rem = L % p.tiles_per_entry;
  const int mt = (EPI == EPI_WGRAD) ? rem / p.n_tiles_n : 0;
  const int nt = (EPI == EPI_WGRAD) ? rem % p.n_tiles_n : rem;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;

  const bf16_t* Bw = p.B + (long long)te.phys * p.strideB;

  // ---- operand addressing ---------------------------------------------------
  int n_k;                // reduction length of this tile
  if (EPI == EPI_WGRAD) n_k = te.rows;
  else n_k = p.K;
  const int nk = (n_k + BK - 1) / BK;

  // A: ragged rows (K-contiguous) or wgrad (row-contiguous over routed rows)
  const bf16_t* a_rows_base = p.A + (long long)te.row0 * p.lda;
  auto a_row_ptr = [&](int r) -> const bf16_t* {
    return r < te.rows ? a_rows_base + (long long)r * p.lda : nullptr;
  };
  const bf16_t* a_t_base = p.A + (long long)te.row0 * p.lda + (long long)mt * BM;
  const int a_t_valid = p.Mw - mt * BM;

  // B: weight rows (K-contiguous, optionally gate/up interleaved) or
  //    row-contiguous (dgrad weights, wgrad activations)
  auto b_row_ptr = [&](int r) -> const bf16_t* {
    int row;
    bool ok;
    if (GU_ROWS) {
      const int grp = r >> 6, w = r & 63;
      const int fcol = nt * (BN / 2) + grp * 32 + (w & 31);
      ok = fcol < p.f;
      row = (w < 32) ? fcol : p.f + fcol;
    } else {
      row = nt * BN + r;
      ok = row < p.N;
    }
    return ok ? Bw + (long long)row * p.ldb : nullptr;
  };
  const bf16_t* b_t_base =
      (EPI == EPI_WGRAD ? p.B + (long long)te.row0 * p.ldb : Bw) + (long long)nt * BN;
  const int b_t_valid = p.N - nt * BN;
  const int b_k_valid = (EPI == EPI_WGRAD) ? te.rows : p.K;

  LoaderK<BM, NT> la_k;
  LoaderT<BM, NT> la_t;
  LoaderK<BN, NT> lb_k;
  LoaderT<BN, NT> lb_t;
  auto load_tiles = [&](int k0) {
    if (A_T) la_t.load(a_t_base, p.lda, k0, n_k, a_t_valid, tid);
    else la_k.load(a_row_ptr, k0, tid);
    if (B_T) lb_t.load(b_t_base, p.ldb, k0, b_k_valid, b_t_valid, tid);
    else lb_k.load(b_row_ptr, k0, tid);
  };
  auto store_tiles = [&](int stage) {
    bf16_t* As = smem + stage * STAGE;
    bf16_t* Bs = As + BM * BK;
    if (A_T) la_t.store(As, tid);
    else la_k.store(As, tid);
    if (B_T) lb_t.store(Bs, tid);
    else lb_k.store(Bs, tid);
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // ---- main loop -----------------------------------------------------------
  if (nk > 0) {
    load_tiles(0);
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      const bool more = kt + 1 < nk;
      if (more) load_tiles((kt + 1) * BK);
      const bf16_t* As = smem + cur * STAGE;
      const bf16_t* Bs = As + BM * BK;
#pragma unroll
      for (int s = 0; s < BK / 16; ++s) {
        const int chunk = s * 2 + (lane >> 5);
        u32x4_t af[TM], bfr[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[i] = *reinterpret_cast<const u32x4_t*>(As + lds_off(wm * WTM + i * 32 + (lane & 31), chunk));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[j] = *reinterpret_cast<const u32x4_t*>(Bs + lds_off(wn * WTN + j * 32 + (lane & 31), chunk));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, bfr[j]), __builtin_bit_cast(bf16x8_t, af[i]),
                acc[i][j], 0, 0, 0);
      }
      if (more) store_tiles(cur ^ 1);
      __syncthreads();
    }
  }

  // ---- epilogues ---------------------------------------------------------------
  const int lrow = lane & 31;
  const int lcol = (lane >> 5) * 4;
  if (EPI == EPI_GU) {
    const int f = p.f;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WTM + i * 32 + lrow;
      if (r >= te.rows) continue;
      const long long grow = te.row0 + r;
#pragma unroll
      for (int pp = 0; pp < TN / 2; ++pp) {
        const int grp = (wn * WTN) / 64 + pp;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int fcol = nt * (BN / 2) + grp * 32 + q * 8 + lcol;
          if (fcol >= f) continue;
          float h[4], g[4], u[4];
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            g[c] = acc[i][2 * pp][q * 4 + c];
            u[c] = acc[i][2 * pp + 1][q * 4 + c];
            h[c] = fast_silu(g[c]) * u[c];
          }
          store_bf16x4(p.out + grow * f + fcol, h[0], h[1], h[2], h[3]);
          if (p.out2) {
            store_bf16x4(p.out2 + grow * 2 * f + fcol, g[0], g[1], g[2], g[3]);
            store_bf16x4(p.out2 + grow * 2 * f + f + fcol, u[0], u[1], u[2], u[3]);
          }
        }
      }
    }
  } else if (EPI == EPI_STORE) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WTM + i * 32 + lrow;
      if (r >= te.rows) continue;
      const long long grow = te.row0 + r;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = nt * BN + wn * WTN + j * 32 + q * 8 + lcol;
          if (col >= p.N) continue;
          store_bf16x4(p.out + grow * p.ldo + col, acc[i][j][q * 4], acc[i][j][q * 4 + 1],
                       acc[i][j][q * 4 + 2], acc[i][j][q * 4 + 3]);
        }
    }
  } else if (EPI == EPI_GU_BWD) {
    const int f = p.f;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WTM + i * 32 + lrow;
      if (r >= te.rows) continue;
      const long long grow = te.row0 + r;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = nt * BN + wn * WTN + j * 32 + q * 8 + lcol;
          if (col >= f) continue;
          float ag[4], au[4], dag[4], dau[4], hb[4];
          load_bf16x4(p.aux + grow * 2 * f + col, ag);
          load_bf16x4(p.aux + grow * 2 * f + f + col, au);
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const float dh = acc[i][j][q * 4 + c];
            const float s = fast_sigmoid(ag[c]);
            const float sl = ag[c] * s;
            dag[c] = dh * au[c] * s * (1.0f + ag[c] * (1.0f - s));
            dau[c] = dh * sl;
            hb[c] = sl * au[c];
          }
          store_bf16x4(p.out + grow * 2 * f + col, dag[0], dag[1], dag[2], dag[3]);
          store_bf16x4(p.out + grow * 2 * f + f + col, dau[0], dau[1], dau[2], dau[3]);
          store_bf16x4(p.out2 + grow * f + col, hb[0], hb[1], hb[2], hb[3]);
        }
    }
  } else {  // EPI_WGRAD
    float* W = p.wout + (long long)te.phys * p.strideW;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = mt * BM + wm * WTM + i * 32 + lrow;
      if (r >= p.Mw) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = nt * BN + wn * WTN + j * 32 + q * 8 + lcol;
          if (col >= p.N) continue;
          f32x4_t* dst = reinterpret_cast<f32x4_t*>(W + (long long)r * p.N + col);
          f32x4_t v = {acc[i][j][q * 4], acc[i][j][q * 4 + 1], acc[i][j][q * 4 + 2],
                       acc[i][j][q * 4 + 3]};
          if (p.accumulate) v += *dst;
          *dst = v;
        }
    }
  }
}

// ---------------------------------------------------------------------------
// Forward products (both operands K-contiguous): deep LDS-DMA pipeline.
//
// Global -> LDS moves use global_load_lds_dwordx4 (no register staging):
// every wave instruction fills 1 KB of LDS contiguously, lane i at +16*i, so
// the swizzle is applied on the global side (each lane fetches the chunk
// that belongs in its LDS slot).  BK = 32: an LDS row is 64 bytes (4 chunks)
// and chunk c of row r is stored at c ^ ((r >> 2) & 3).  With that layout the
// fragment reads (lane -> row lane % 32, chunk lane / 32) measured zero LDS
// bank-conflict cycles on gfx950 (SQ_LDS_BANK_CONFLICT), where the unswizzled
// layout costs 3 extra cycles per ds_read_b128.
// NS stages are in flight; one s_barrier per k-tile.  The wait before it is
// an explicit vmcnt on this thread's outstanding LDS-DMA loads, then the
// barrier makes every thread's loads visible.
// ---------------------------------------------------------------------------
constexpr int PBK = 32;          // k per pipeline stage
constexpr int PROW = PBK * 2;    // bytes per LDS row

__device__ __forceinline__ int pswz(int row) { return (row >> 2) & 3; }

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

// One k-tile of LDS-DMA loads for this thread: A chunks then B chunks.  (A
// device function, not a lambda: the host pass of a kernel must not see the
// LDS-DMA builtin inside a lambda, or the kernel's launch stub is dropped.)
template <int NA, int NB, int NT, int A_BYTES>
__device__ __forceinline__ void dma_tile(char* st, const bf16_t* const* a_src,
                                         const bf16_t* const* b_src, int k0, int wave) {
#pragma unroll
  for (int i = 0; i < NA; ++i)
    __builtin_amdgcn_global_load_lds(a_src[i] + k0, (lds_void_t*)(st + (i * NT + wave * 64) * 16),
                                     16, 0, 0);
#pragma unroll
  for (int i = 0; i < NB; ++i)
    __builtin_amdgcn_global_load_lds(b_src[i] + k0,
                                     (lds_void_t*)(st + A_BYTES + (i * NT + wave * 64) * 16), 16,
                                     0, 0);
}

template <int BM, int BN, int NWM, int NWN, int NS, int EPI, bool GU_ROWS>
__global__ __launch_bounds__(64 * NWM * NWN) void gemm_nt_pipe_kernel(GemmParams p) {
  constexpr int NT = 64 * NWM * NWN;
  static_assert((BM * 4) % NT == 0 && (BN * 4) % NT == 0, "chunks must divide over the threads");
  static_assert(NS >= 3, "at least three stages");
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * PROW, B_BYTES = BN * PROW;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int NA = BM * 4 / NT, NB = BN * 4 / NT;  // 16-byte chunks per thread
  constexpr int NLD = NA + NB;                        // loads per thread per k-tile
  constexpr int NFR = TM + TN;                        // fragment reads per k16 step
  static_assert(EPI != EPI_GU || (TN % 2 == 0), "SwiGLU epilogue pairs gate/up blocks");
  __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

  // ---- tile schedule (XCD-contiguous) --------------------------------------
  const int n_valid = (*p.n_entries) * p.tiles_per_entry;
  const int per = (n_valid + 7) >> 3;
  const int slot = blockIdx.x >> 3;
  if (slot >= per) return;
  const int L = (blockIdx.x & 7) * per + slot;
  if (L >= n_valid) return;
  const TileEntry te = p.table[L / p.tiles_per_entry];
  const int nt = L % p.tiles_per_entry;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;

  // ---- per-thread global source of each LDS chunk it fills ------------------
  const bf16_t* a_src[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int q = i * NT + tid;
    const int r = q >> 2;
    const int lc = (q & 3) ^ pswz(r);
    const int rr = r < te.rows ? r : te.rows - 1;   // rows past the expert: any valid row
    a_src[i] = p.A + (long long)(te.row0 + rr) * p.lda + lc * 8;
  }
  const bf16_t* Bw = p.B + (long long)te.phys * p.strideB;
  const bf16_t* b_src[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int q = i * NT + tid;
    const int r = q >> 2;
    const int lc = (q & 3) ^ pswz(r);
    int row;
    if (GU_ROWS) {
      const int grp = r >> 6, w = r & 63;
      int fcol = nt * (BN / 2) + grp * 32 + (w & 31);
      fcol = fcol < p.f ? fcol : p.f - 1;
      row = (w < 32) ? fcol : p.f + fcol;
    } else {
      row = nt * BN + r;
      row = row < p.N ? row : p.N - 1;
    }
    b_src[i] = Bw + (long long)row * p.ldb + lc * 8;
  }
  auto issue = [&](int kt) {
    dma_tile<NA, NB, NT, A_BYTES>(smem + (kt % NS) * STAGE, a_src, b_src, kt * PBK, wave);
  };
  // fragment LDS byte offsets within a stage for k16 step 0; step 1 is ^32
  int a_off[TM], b_off[TN];
  const int lc0 = lane >> 5;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * WTM + i * 32 + (lane & 31);
    a_off[i] = r * PROW + ((lc0 ^ pswz(r)) << 4);
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int r = wn * WTN + j * 32 + (lane & 31);
    b_off[j] = A_BYTES + r * PROW + ((lc0 ^ pswz(r)) << 4);
  }
  u32x4_t fa0[TM], fb0[TN], fa1[TM], fb1[TN];
  auto read_frags = [&](const char* st, int flip, u32x4_t* fa, u32x4_t* fb) {
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[i] = *reinterpret_cast<const u32x4_t*>(st + (a_off[i] ^ flip));
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[j] = *reinterpret_cast<const u32x4_t*>(st + (b_off[j] ^ flip));
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  auto mma_step = [&](const u32x4_t* fa, const u32x4_t* fb) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, fb[j]), __builtin_bit_cast(bf16x8_t, fa[i]), acc[i][j],
            0, 0, 0);
  };
  // interleave the fragment reads of the next step with this step's MFMAs
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < NFR; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - NFR, 0);
  };

  const int nk = p.K / PBK;
  // Every iteration issues exactly one k-tile of LDS-DMA loads (past the end
  // the last k-tile is loaded again into the free stage), so the number of
  // loads in flight is the same at every wait and one constant vmcnt
  // suffices: the loop body is straight-line code, which lets the compiler
  // keep exact LDS wait counts across the barrier.
  // prologue: tiles 0 .. NS-2 in flight (stage NS-1 stays free for the first
  // refill), tile 0 landed, its step-0 fragments read
#pragma unroll
  for (int t = 0; t < NS - 1; ++t) issue(t < nk ? t : nk - 1);
  wait_vmcnt<(NS - 2) * NLD>();
  __builtin_amdgcn_s_barrier();
  read_frags(smem, 0, fa0, fb0);

  for (int kt = 0; kt < nk; ++kt) {
    const char* st = smem + (kt % NS) * STAGE;
    // first half: MFMAs of step 0, fragment reads of step 1 of the same tile
    read_frags(st, 32, fa1, fb1);
    mma_step(fa0, fb0);
    interleave();
    // tile boundary: tile kt+1 has landed for every thread, and every wave is
    // done with stage (kt-1) % NS, which receives tile kt+NS-1
    wait_vmcnt<(NS - 3) * NLD>();
    __builtin_amdgcn_s_barrier();
    {
      const int t = kt + NS - 1;
      dma_tile<NA, NB, NT, A_BYTES>(smem + (t % NS) * STAGE, a_src, b_src,
                                    (t < nk ? t : nk - 1) * PBK, wave);
    }
    read_frags(smem + ((kt + 1) % NS) * STAGE, 0, fa0, fb0);
    // second half: MFMAs of step 1, step-0 fragment reads of the next tile
    mma_step(fa1, fb1);
    interleave();
  }
  // no LDS-DMA may still be writing when the workgroup retires
  wait_vmcnt<0>();

  // ---- epilogues: stage the tile in LDS, then write whole rows -----------------
  // Each lane holds one row and 4 consecutive columns per register quad, so a
  // direct store scatters 16 bytes into each of 32 rows.  Staging through the
  // (now idle) LDS lets every store instruction write 4 rows of 256 contiguous
  // bytes instead.
  wait_lgkm0();  // all LDS reads done
  __builtin_amdgcn_s_barrier();
  const int lrow = lane & 31;
  const int lcol = (lane >> 5) * 4;
  constexpr int SCOLS = (EPI == EPI_GU) ? BN : BN;  // staged columns per pass
  constexpr int PITCH = SCOLS * 2 + 16;               // bytes per staged row
  static_assert(BM * PITCH <= NS * STAGE, "staging tile must fit in LDS");
  // write the staged [BM][SCOLS] tile to global rows: columns [0, ncols) of
  // the staged tile go to dst + row * ld + col (bf16), rows < te.rows only
  auto flush = [&](bf16_t* dst, long long ld, int ncols, int scol0) {
    const int chunks_per_row = ncols / 8;
    const int total = BM * chunks_per_row;
    for (int c = tid; c < total; c += NT) {
      const int r = c / chunks_per_row, cc = c % chunks_per_row;
      if (r < te.rows) {
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(smem + r * PITCH + (scol0 + cc * 8) * 2);
        *reinterpret_cast<u32x4_t*>(dst + (te.row0 + r) * ld + cc * 8) = v;
      }
    }
  };
  auto stage = [&](int row, int col, float a, float b, float c, float d) {
    u32x2_t w = {pack_bf16x2(a, b), pack_bf16x2(c, d)};
    *reinterpret_cast<u32x2_t*>(smem + row * PITCH + col * 2) = w;
  };
  if (EPI == EPI_GU) {
    // staged columns: [0, BN/2) = gate f-columns, [BN/2, BN) = up f-columns
    const int f = p.f;
    const int fbase = nt * (BN / 2);
    const int fcols = min(BN / 2, f - fbase);
    if (p.out2) {  // pass 1: act_save (gate and up pre-activations)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WTM + i * 32 + lrow;
#pragma unroll
        for (int pp = 0; pp < TN / 2; ++pp) {
          const int grp = (wn * WTN) / 64 + pp;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int c = grp * 32 + q * 8 + lcol;
            stage(r, c, acc[i][2 * pp][q * 4], acc[i][2 * pp][q * 4 + 1],
                  acc[i][2 * pp][q * 4 + 2], acc[i][2 * pp][q * 4 + 3]);
            stage(r, BN / 2 + c, acc[i][2 * pp + 1][q * 4], acc[i][2 * pp + 1][q * 4 + 1],
                  acc[i][2 * pp + 1][q * 4 + 2], acc[i][2 * pp + 1][q * 4 + 3]);
          }
        }
      }
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      flush(p.out2 + fbase, 2LL * f, fcols, 0);
      flush(p.out2 + f + fbase, 2LL * f, fcols, BN / 2);
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
    }
    // pass 2: H = silu(gate) * up
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int pp = 0; pp < TN / 2; ++pp) {
        const int grp = (wn * WTN) / 64 + pp;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float h[4];
#pragma unroll
          for (int c = 0; c < 4; ++c)
            h[c] = fast_silu(acc[i][2 * pp][q * 4 + c]) * acc[i][2 * pp + 1][q * 4 + c];
          stage(r, grp * 32 + q * 8 + lcol, h[0], h[1], h[2], h[3]);
        }
      }
    }
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
    flush(p.out + fbase, f, fcols, 0);
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          stage(r, wn * WTN + j * 32 + q * 8 + lcol, acc[i][j][q * 4], acc[i][j][q * 4 + 1],
                acc[i][j][q * 4 + 2], acc[i][j][q * 4 + 3]);
    }
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
    flush(p.out + nt * BN, p.ldo, min(BN, p.N - nt * BN), 0);
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
constexpr int kBM = 128, kBN = 128, kNWM = 2, kNWN = 2;
constexpr int kThreads = 64 * kNWM * kNWN;

inline int ceil_div(long long a, long long b) { return (int)((a + b - 1) / b); }
inline int round8(int v) { return (v + 7) & ~7; }

inline int ragged_max_entries(int64_t R, int E) { return ceil_div(R, kBM) + E; }

template <int EPI, bool A_T, bool B_T, bool GU>
hipError_t launch_gemm(const GemmParams& p, int grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((grouped_gemm_kernel<kBM, kBN, kNWM, kNWN, EPI, A_T, B_T, GU>),
                     dim3(round8(grid)), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

// Forward tile shapes.  The default is 256 x 256 with 8 waves (2 x 4, each
// 128 x 64, two waves per SIMD so one wave's MFMAs cover the other's waits).
// 256 x 256 with 4 waves and 128 x 512 with 4 waves remain selectable through
// LAEP_GEMM_TILE=256x256 / 128x512 for tuning comparisons.
enum FwdTile { TILE_128x512 = 0, TILE_256x256 = 1, TILE_256x256_W8 = 2 };

FwdTile pick_fwd_tile(int64_t R, int E) {
  static const char* env = getenv("LAEP_GEMM_TILE");
  if (env && strcmp(env, "128x512") == 0) return TILE_128x512;
  if (env && strcmp(env, "256x256") == 0) return TILE_256x256;
  if (env && strcmp(env, "256x256w8") == 0) return TILE_256x256_W8;
  (void)R;
  (void)E;
  return TILE_256x256_W8;
}

template <int BM, int BN, int NWM, int NWN, int NS, int EPI, bool GU>
hipError_t launch_pipe(const GemmParams& p, int grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_nt_pipe_kernel<BM, BN, NWM, NWN, NS, EPI, GU>), dim3(round8(grid)),
                     dim3(64 * NWM * NWN), 0, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int NWM, int NWN, int NS>
hipError_t ffn_fwd_pipe(const void* x_perm, const void* w_gu, const void* w_d,
                        const int32_t* offsets, const int32_t* expert_map, int E, int d, int f,
                        int64_t R, void* y_perm, void* act_save, void* ws, hipStream_t s) {
  bf16_t* H = static_cast<bf16_t*>(ws);
  const int max_entries = ceil_div(R, BM) + E;
  TableWs tw = carve_table(static_cast<char*>(ws) + align_up((size_t)R * f * 2, 256), max_entries);
  hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, expert_map,
                     E, BM, 0, max_entries, tw.n_entries, tw.table);
  GemmParams g = {};
  g.table = tw.table;
  g.n_entries = tw.n_entries;
  g.f = f;
  // gate/up + SwiGLU: B rows interleaved gate/up per 32, BN/2 f-columns per tile
  g.A = static_cast<const bf16_t*>(x_perm);
  g.lda = d;
  g.B = static_cast<const bf16_t*>(w_gu);
  g.ldb = d;
  g.strideB = (long long)2 * f * d;
  g.N = 2 * f;
  g.K = d;
  g.n_tiles_n = ceil_div(f, BN / 2);
  g.tiles_per_entry = g.n_tiles_n;
  g.out = H;
  g.ldo = f;
  g.out2 = static_cast<bf16_t*>(act_save);
  hipError_t err = launch_pipe<BM, BN, NWM, NWN, NS, EPI_GU, true>(g, max_entries * g.n_tiles_n, s);
  if (err != hipSuccess) return err;
  // down projection
  g.A = H;
  g.lda = f;
  g.B = static_cast<const bf16_t*>(w_d);
  g.ldb = f;
  g.strideB = (long long)d * f;
  g.N = d;
  g.K = f;
  g.n_tiles_n = ceil_div(d, BN);
  g.tiles_per_entry = g.n_tiles_n;
  g.out = static_cast<bf16_t*>(y_perm);
  g.ldo = d;
  g.out2 = nullptr;
  return launch_pipe<BM, BN, NWM, NWN, NS, EPI_STORE, false>(g, max_entries * g.n_tiles_n, s);
}

}  // namespace

size_t ffn_fwd_ws_bytes(int64_t R, int E, int d, int f, int dtype) {
  (void)d;
  const size_t elem = dtype == kDtypeBf16 ? 2 : 4;
  // the table is sized for the smallest row tile of either dtype (64 rows)
  return align_up((size_t)R * f * elem, 256) + table_bytes(ceil_div(R, 64) + E);
}

hipError_t launch_ffn_fwd_bf16(const void* x_perm, const void* w_gu, const void* w_d,
                               const int32_t* offsets, const int32_t* expert_map, int E, int d,
                               int f, int64_t R, void* y_perm, void* act_save, void* ws,
                               hipStream_t s) {
  const FwdTile tile = pick_fwd_tile(R, E);
  if (tile == TILE_256x256_W8)
    return ffn_fwd_pipe<256, 256, 2, 4, 5>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                           y_perm, act_save, ws, s);
  if (tile == TILE_256x256)
    return ffn_fwd_pipe<256, 256, 2, 2, 5>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                        y_perm, act_save, ws, s);
  return ffn_fwd_pipe<128, 512, 1, 4, 4>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R, y_perm,
                                      act_save, ws, s);
}

size_t ffn_bwd_hb_offset(int64_t R, int f, int dtype) {
  const size_t elem = dtype == kDtypeBf16 ? 2 : 4;
  return align_up((size_t)R * 2 * f * elem, 256);
}

size_t ffn_bwd_ws_bytes(int64_t R, int E, int d, int f, int dtype) {
  (void)d;
  const size_t elem = dtype == kDtypeBf16 ? 2 : 4;
  return ffn_bwd_hb_offset(R, f, dtype) + align_up((size_t)R * f * elem, 256) +
         table_bytes(ragged_max_entries(R, E)) + table_bytes(E);
}

hipError_t launch_ffn_bwd_bf16(const void* dy, const void* x_perm, const void* act_save,
                               const void* w_gu, const void* w_d, const int32_t* offsets,
                               const int32_t* expert_map, int E, int d, int f, int64_t R,
                               void* dx_perm, float* dw_gu, float* dw_d, int accumulate,
                               void* ws, hipStream_t s) {
  char* base = static_cast<char*>(ws);
  bf16_t* dA = reinterpret_cast<bf16_t*>(base);
  bf16_t* Hb = reinterpret_cast<bf16_t*>(base + ffn_bwd_hb_offset(R, f, kDtypeBf16));
  char* tables = base + ffn_bwd_hb_offset(R, f, kDtypeBf16) + align_up((size_t)R * f * 2, 256);
  const int max_ragged = ragged_max_entries(R, E);
  TableWs tr = carve_table(tables, max_ragged);
  TableWs te = carve_table(tables + table_bytes(max_ragged), E);
  hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, expert_map,
                     E, kBM, 0, max_ragged, tr.n_entries, tr.table);
  hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, expert_map,
                     E, kBM, 1, E, te.n_entries, te.table);

  // dgrad 1: dH = dY W_d (B = W_d [d][f] row-contiguous), SwiGLU backward epilogue
  GemmParams g = {};
  g.table = tr.table;
  g.n_entries = tr.n_entries;
  g.f = f;
  g.A = static_cast<const bf16_t*>(dy);
  g.lda = d;
  g.B = static_cast<const bf16_t*>(w_d);
  g.ldb = f;
  g.strideB = (long long)d * f;
  g.N = f;
  g.K = d;
  g.n_tiles_n = ceil_div(f, kBN);
  g.tiles_per_entry = g.n_tiles_n;
  g.out = dA;
  g.out2 = Hb;
  g.aux = static_cast<const bf16_t*>(act_save);
  hipError_t err = launch_gemm<EPI_GU_BWD, false, true, false>(g, max_ragged * g.n_tiles_n, s);
  if (err != hipSuccess) return err;

  // dgrad 2: dX = dA W_gu (B = W_gu [2f][d] row-contiguous)
  g.A = dA;
  g.lda = 2 * f;
  g.B = static_cast<const bf16_t*>(w_gu);
  g.ldb = d;
  g.strideB = (long long)2 * f * d;
  g.N = d;
  g.K = 2 * f;
  g.n_tiles_n = ceil_div(d, kBN);
  g.tiles_per_entry = g.n_tiles_n;
  g.out = static_cast<bf16_t*>(dx_perm);
  g.ldo = d;
  g.out2 = nullptr;
  g.aux = nullptr;
  err = launch_gemm<EPI_STORE, false, true, false>(g, max_ragged * g.n_tiles_n, s);
  if (err != hipSuccess) return err;

  // wgrad W_d: dW_d[p] [d, f] = dY^T H_b over the expert's rows
  GemmParams w = {};
  w.table = te.table;
  w.n_entries = te.n_entries;
  w.f = f;
  w.A = static_cast<const bf16_t*>(dy);
  w.lda = d;
  w.B = Hb;
  w.ldb = f;
  w.Mw = d;
  w.N = f;
  w.n_tiles_n = ceil_div(f, kBN);
  w.tiles_per_entry = ceil_div(d, kBM) * w.n_tiles_n;
  w.wout = dw_d;
  w.strideW = (long long)d * f;
  w.accumulate = accumulate;
  err = launch_gemm<EPI_WGRAD, true, true, false>(w, E * w.tiles_per_entry, s);
  if (err != hipSuccess) return err;

  // wgrad W_gu: dW_gu[p] [2f, d] = dA^T X
  w.A = dA;
  w.lda = 2 * f;
  w.B = static_cast<const bf16_t*>(x_perm);
  w.ldb = d;
  w.Mw = 2 * f;
  w.N = d;
  w.n_tiles_n = ceil_div(d, kBN);
  w.tiles_per_entry = ceil_div(2 * f, kBM) * w.n_tiles_n;
  w.wout = dw_gu;
  w.strideW = (long long)2 * f * d;
  return launch_gemm<EPI_WGRAD, true, true, false>(w, E * w.tiles_per_entry, s);
}

}  // namespace laep
