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
#include "gemm_common.hpp"

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

template <int BM, int BN, int NWM, int NWN, int NS, int EPI, bool GU_ROWS, int SCHED>
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
  constexpr int SMEM = (NS * STAGE > BM * (BN * 2 + 16)) ? NS * STAGE : BM * (BN * 2 + 16);
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

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
  // order of the next step's fragment reads against this step's MFMAs:
  // SCHED 0 alternates one MFMA and one DS read; SCHED 1 issues every DS read
  // first (they then have the whole MFMA run to land)
  auto interleave = [&]() {
    if (SCHED == 0) {
#pragma unroll
      for (int i = 0; i < NFR; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, TM * TN - NFR, 0);
    } else {
      __builtin_amdgcn_sched_group_barrier(0x100, NFR, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);
    }
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
  static_assert(BM * PITCH <= SMEM, "staging tile must fit in LDS");
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
// Forward products, BK = 64 variant: every row segment a k-tile loads is one
// whole 128-byte line (the BK = 32 pipeline fetches half lines, which halves
// the bytes per L2 request).  Two 64 KB stages: the LDS-DMA of tile k+1 is
// issued when tile k starts and has that tile's four k16 steps to land.
// LDS rows are 128 bytes (8 chunks); chunk c of row r sits at
// c ^ ((r ^ r >> 3) & 7), measured free of bank conflicts for the fragment
// reads.  One barrier per tile, before the last k16 step, after every wave's
// reads of the current stage and every thread's loads of the next tile are
// complete.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int swz8(int row) { return (row ^ (row >> 3)) & 7; }

template <int NA, int NB, int NT, int A_BYTES>
__device__ __forceinline__ void dma_tile64(char* st, const bf16_t* const* a_src,
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

template <int BM, int BN, int NWM, int NWN, int EPI, bool GU_ROWS>
__global__ __launch_bounds__(64 * NWM * NWN) void gemm_nt_k64_kernel(GemmParams p) {
  constexpr int NT = 64 * NWM * NWN;
  constexpr int BKL = 64;                             // k per stage
  constexpr int ROWB = BKL * 2;                       // 128 bytes per LDS row
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * ROWB, B_BYTES = BN * ROWB;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int NA = BM * 8 / NT, NB = BN * 8 / NT;   // 16-byte chunks per thread
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0, "chunks must divide over the threads");
  static_assert(EPI != EPI_GU || (TN % 2 == 0), "SwiGLU epilogue pairs gate/up blocks");
  constexpr int SMEM = (2 * STAGE > BM * (BN * 2 + 16)) ? 2 * STAGE : BM * (BN * 2 + 16);
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

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

  const bf16_t* a_src[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int q = i * NT + tid;
    const int r = q >> 3;
    const int lc = (q & 7) ^ swz8(r);
    const int rr = r < te.rows ? r : te.rows - 1;
    a_src[i] = p.A + (long long)(te.row0 + rr) * p.lda + lc * 8;
  }
  const bf16_t* Bw = p.B + (long long)te.phys * p.strideB;
  const bf16_t* b_src[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int q = i * NT + tid;
    const int r = q >> 3;
    const int lc = (q & 7) ^ swz8(r);
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

  int a_off[TM], b_off[TN];
  const int lc0 = lane >> 5;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * WTM + i * 32 + (lane & 31);
    a_off[i] = r * ROWB + ((lc0 ^ swz8(r)) << 4);
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int r = wn * WTN + j * 32 + (lane & 31);
    b_off[j] = A_BYTES + r * ROWB + ((lc0 ^ swz8(r)) << 4);
  }
  // k16 step s of a stage: logical chunk 2s + lane/32, i.e. byte offset ^ (32 s)
  u32x4_t fa[2][TM], fb[2][TN];
  auto read_frags = [&](const char* st, int s, int buf) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
      fa[buf][i] = *reinterpret_cast<const u32x4_t*>(st + (a_off[i] ^ (s << 5)));
#pragma unroll
    for (int j = 0; j < TN; ++j)
      fb[buf][j] = *reinterpret_cast<const u32x4_t*>(st + (b_off[j] ^ (s << 5)));
  };

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  auto mma = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, fb[buf][j]), __builtin_bit_cast(bf16x8_t, fa[buf][i]),
            acc[i][j], 0, 0, 0);
  };

  const int nk = p.K / BKL;
  dma_tile64<NA, NB, NT, A_BYTES>(smem, a_src, b_src, 0, wave);
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  read_frags(smem, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const char* st = smem + (kt & 1) * STAGE;
    // the other stage was released by the barrier that ended tile kt-1
    if (kt + 1 < nk)
      dma_tile64<NA, NB, NT, A_BYTES>(smem + ((kt + 1) & 1) * STAGE, a_src, b_src,
                                      (kt + 1) * BKL, wave);
    read_frags(st, 1, 1);
    mma(0);
    read_frags(st, 2, 0);
    mma(1);
    read_frags(st, 3, 1);
    mma(0);
    // every wave's reads of this stage and every thread's loads of tile kt+1
    // are complete past this barrier
    wait_lgkm0();
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + 1 < nk) read_frags(smem + ((kt + 1) & 1) * STAGE, 0, 0);
    mma(1);
  }
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
  static_assert(BM * PITCH <= SMEM, "staging tile must fit in LDS");
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


inline int ragged_max_entries(int64_t R, int E) { return ceil_div(R, kBM) + E; }


// Forward tile shapes.  The default is 256 x 256 with 8 waves (2 x 4, each
// 128 x 64, two waves per SIMD so one wave's MFMAs cover the other's waits).
// 256 x 256 with 4 waves and 128 x 512 with 4 waves remain selectable through
// LAEP_GEMM_TILE=256x256 / 128x512 for tuning comparisons.
enum FwdTile { TILE_128x512 = 0, TILE_256x256 = 1, TILE_256x256_W8 = 2, TILE_256x256_W8_DS = 3, TILE_K64_W8 = 4, TILE_K64_W4 = 5 };

FwdTile pick_fwd_tile(int64_t R, int E) {
  static const char* env = getenv("LAEP_GEMM_TILE");
  if (env && strcmp(env, "128x512") == 0) return TILE_128x512;
  if (env && strcmp(env, "256x256") == 0) return TILE_256x256;
  if (env && strcmp(env, "256x256w8") == 0) return TILE_256x256_W8;
  if (env && strcmp(env, "256x256w8ds") == 0) return TILE_256x256_W8_DS;
  if (env && strcmp(env, "k64w8") == 0) return TILE_K64_W8;
  if (env && strcmp(env, "k64w4") == 0) return TILE_K64_W4;
  (void)R;
  (void)E;
  return TILE_256x256_W8;
}

template <int BM, int BN, int NWM, int NWN, int NS, int SCHED, int EPI, bool GU>
hipError_t launch_pipe(const GemmParams& p, int grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_nt_pipe_kernel<BM, BN, NWM, NWN, NS, EPI, GU, SCHED>), dim3(round8(grid)),
                     dim3(64 * NWM * NWN), 0, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int NWM, int NWN, int EPI, bool GU>
hipError_t launch_k64(const GemmParams& p, int grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_nt_k64_kernel<BM, BN, NWM, NWN, EPI, GU>), dim3(round8(grid)),
                     dim3(64 * NWM * NWN), 0, s, p);
  return hipGetLastError();
}

template <int BM, int BN, int NWM, int NWN, int NS, int SCHED>
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
  hipError_t err;
  if constexpr (NS == 2)
    err = launch_k64<BM, BN, NWM, NWN, EPI_GU, true>(g, max_entries * g.n_tiles_n, s);
  else
    err = launch_pipe<BM, BN, NWM, NWN, NS, SCHED, EPI_GU, true>(g, max_entries * g.n_tiles_n, s);
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
  if constexpr (NS == 2)
    return launch_k64<BM, BN, NWM, NWN, EPI_STORE, false>(g, max_entries * g.n_tiles_n, s);
  else
    return launch_pipe<BM, BN, NWM, NWN, NS, SCHED, EPI_STORE, false>(g, max_entries * g.n_tiles_n, s);
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
    return ffn_fwd_pipe<256, 256, 2, 4, 5, 0>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                              y_perm, act_save, ws, s);
  if (tile == TILE_K64_W8)
    return ffn_fwd_pipe<256, 256, 2, 4, 2, 0>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                              y_perm, act_save, ws, s);
  if (tile == TILE_K64_W4)
    return ffn_fwd_pipe<256, 256, 2, 2, 2, 0>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                              y_perm, act_save, ws, s);
  if (tile == TILE_256x256_W8_DS)
    return ffn_fwd_pipe<256, 256, 2, 4, 5, 1>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                              y_perm, act_save, ws, s);
  if (tile == TILE_256x256)
    return ffn_fwd_pipe<256, 256, 2, 2, 5, 0>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R,
                                        y_perm, act_save, ws, s);
  return ffn_fwd_pipe<128, 512, 1, 4, 4, 0>(x_perm, w_gu, w_d, offsets, expert_map, E, d, f, R, y_perm,
                                      act_save, ws, s);
}

}  // namespace laep
