// Forward grouped bf16 GEMMs of the SwiGLU expert FFN (moe_grouped_ffn_fwd)
// on the gfx950 matrix cores:
//   gate/up   A = X_e [M_e, d]  x W_gu[p]^T [2f, d]  -> SwiGLU epilogue (H, act_save)
//   down      A = H_e [M_e, f]  x W_d[p]^T  [d, f]   -> Y
// Both operands are K-contiguous, so global -> LDS moves are LDS-DMA
// (buffer_load_dwordx4 with the LDS flag, no register staging): one wave instruction fills
// 1 KB of LDS contiguously, lane i at +16 i, so any LDS swizzle is applied on
// the global side (each lane fetches the chunk that belongs in its slot).
//
// MFMA v_mfma_f32_32x32x16_bf16 is issued with the operands swapped
// (weights as the "A" input, tokens as the "B" input), so each lane ends up
// owning one output row and 4 consecutive output columns per register quad:
// acc[tm][tn][4q + i] = C[m = tm*32 + lane%32][n = tn*32 + 8q + 4(lane/32) + i].
//
// Ragged expert rows come from a device-side tile table built from the
// expert offsets, so the host never learns the per-expert row counts.
// Workgroup ids are remapped so that each of the 8 XCDs walks a contiguous
// range of tiles (same expert, same weight blocks -> its own L2).
//
// Main loop: 256 x 256 tiles, 8 waves (2 x 4, each 128 x 64), k-steps of 64,
// so every row segment a step loads is one whole 128-byte line.  The L2 -> CU
// feed is bound by cache-line requests (about half a line per clock per CU,
// measured with LDS-DMA), so whole lines double the bytes per request against
// the 64-byte half lines of 32-wide k-steps.  One operand's k-step is a 32 KB
// "half"; the LDS is a ring of five halves (A0 B0 A1 B1 A2 | B2 A3 ...), so
// while step i computes, the B half of step i+1 and the A half of step i+2
// are in flight: every half has at least one whole k-step (2048 MFMA cycles
// per SIMD) to land.
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"
#include "tiles.hpp"
#include "gemm_common.hpp"


namespace laep {
namespace {

// fourth word of a raw buffer resource: 32-bit data format, no swizzle
constexpr int kBufferFlags = 0x00020000;

// Global -> LDS copy of NC 16-byte chunks per thread through buffer loads
// with the LDS flag: chunk i of this thread is at byte voff[i] + soff of the
// operand's buffer.  (The global-segment form of the same copy makes the
// compiler drain every outstanding LDS read, lgkmcnt(0), before each fragment
// use in the loop; with the buffer form it counts them in order.)  A device
// function, not a lambda: the host pass of a kernel must not see the LDS-DMA
// builtin inside a lambda, or the kernel's launch stub is dropped.
template <int NC, int NT>
__device__ __forceinline__ void dma_chunks(char* dst, __amdgpu_buffer_rsrc_t rsrc,
                                           const uint32_t* voff, int soff, int wave) {
#pragma unroll
  for (int i = 0; i < NC; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)(dst + (i * NT + wave * 64) * 16),
                                             16, voff[i], soff, 0, 0);
}

// Tile of the XCD-contiguous schedule owned by this workgroup, or -1.
__device__ __forceinline__ int xcd_tile(const GemmParams& p) {
  const int n_valid = (*p.n_entries) * p.tiles_per_entry;
  const int per = (n_valid + 7) >> 3;
  const int slot = blockIdx.x >> 3;
  if (slot >= per) return -1;
  const int L = (blockIdx.x & 7) * per + slot;
  return L < n_valid ? L : -1;
}

// Weight row feeding B-tile row r of output block nt.  Gate/up: the tile's
// BN rows are BN/2 f-columns of W_gate and the same BN/2 of W_up, interleaved
// per 32 (rows 64g .. 64g+31 gate, 64g+32 .. 64g+63 up), so the SwiGLU pairs
// sit in one wave's accumulators.
template <int BN, bool GU_ROWS>
__device__ __forceinline__ int weight_row(const GemmParams& p, int nt, int r) {
  if (GU_ROWS) {
    const int grp = r >> 6, w = r & 63;
    int fcol = nt * (BN / 2) + grp * 32 + (w & 31);
    fcol = fcol < p.f ? fcol : p.f - 1;
    return (w < 32) ? fcol : p.f + fcol;
  }
  const int row = nt * BN + r;
  return row < p.N ? row : p.N - 1;
}

// ---------------------------------------------------------------------------
// Epilogues: stage the tile in LDS, then write whole rows.  Each lane holds
// one row and 4 consecutive columns per register quad, so a direct store
// scatters 16 bytes into each of 32 rows; staging through the (idle) LDS lets
// every store instruction write 4 rows of 256 contiguous bytes instead.
// ---------------------------------------------------------------------------
template <int BM, int BN, int NWM, int NWN, int EPI>
__device__ __forceinline__ void fwd_epilogue(const GemmParams& p, const TileEntry& te, int nt,
                                             f32x16_t (&acc)[BM / NWM / 32][BN / NWN / 32],
                                             char* smem) {
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int PITCH = BN * 2 + 16;  // bytes per staged row
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;
  const int lrow = lane & 31;
  const int lcol = (lane >> 5) * 4;
  // staged [BM][BN] bf16 -> global rows: staged columns [scol0, scol0 + ncols)
  // go to dst + row * ld (rows < te.rows only).  NCMAX (>= ncols) fixes the
  // trip count, so all of a thread's LDS reads are issued before one wait.
  auto flush = [&](auto ncmax_tag, bf16_t* dst, long long ld, int ncols, int scol0) {
    constexpr int CPR = decltype(ncmax_tag)::value / 8;
    constexpr int ITERS = BM * CPR / NT;
    static_assert(BM * CPR % NT == 0, "flush chunks must divide over the threads");
    u32x4_t v[ITERS];
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * NT + tid;
      const int r = c / CPR, cc = c % CPR;
      v[it] = *reinterpret_cast<const u32x4_t*>(smem + r * PITCH + (scol0 + cc * 8) * 2);
    }
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * NT + tid;
      const int r = c / CPR, cc = c % CPR;
      if (r < te.rows && cc * 8 < ncols)
        *reinterpret_cast<u32x4_t*>(dst + (te.row0 + r) * ld + cc * 8) = v[it];
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
      flush(std::integral_constant<int, BN / 2>{}, p.out2 + fbase, 2LL * f, fcols, 0);
      flush(std::integral_constant<int, BN / 2>{}, p.out2 + f + fbase, 2LL * f, fcols, BN / 2);
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
    flush(std::integral_constant<int, BN / 2>{}, p.out + fbase, f, fcols, 0);
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
    const int ncols = min(BN, p.N - nt * BN);
    if (!p.out_tok) {
      flush(std::integral_constant<int, BN>{}, p.out + nt * BN, p.ldo, ncols, 0);
      return;
    }
    // scatter: routed row r also goes to its token's row of out_tok, times its
    // gate, with the combine's arithmetic (fp32 0 + g * y, one rounding); y
    // rows are written too when p.out is set (the backward reads them)
    constexpr int CPR = BN / 8, ITERS = BM * CPR / NT;
    u32x4_t v[ITERS];
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * NT + tid;
      v[it] = *reinterpret_cast<const u32x4_t*>(smem + (c / CPR) * PITCH + (c % CPR) * 16);
    }
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * NT + tid;
      const int r = c / CPR, cc = c % CPR;
      if (r < te.rows && cc * 8 < ncols) {
        const long long row = (long long)te.row0 + r;
        if (p.out) *reinterpret_cast<u32x4_t*>(p.out + row * p.ldo + nt * BN + cc * 8) = v[it];
        const int src = p.row_src[row];
        const float g = p.gate[src];
        u32x4_t o;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          float lo = 0.0f, hi = 0.0f;
          lo += g * lo_bf16(v[it][w]);
          hi += g * hi_bf16(v[it][w]);
          o[w] = pack_bf16x2(lo, hi);
        }
        *reinterpret_cast<u32x4_t*>(p.out_tok + (long long)(src / p.slots_k) * p.ldo + nt * BN +
                                    cc * 8) = o;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Ring main loop: 256 x 256 tiles, 8 waves (2 x 4, each 128 x 64), k-steps
// of 64 through a ring of five 32 KB halves.
// ---------------------------------------------------------------------------
template <int NWM, int NWN, int EPI, bool GU_ROWS, bool GATHER>
__global__ __launch_bounds__(64 * NWM * NWN) void gemm_nt_ring_kernel(GemmParams p) {
  constexpr int BM = 256, BN = 256;
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int ROWB = 128;                 // bytes per LDS row (64 k)
  constexpr int HALF = BM * ROWB;           // one operand's k-step, 32 KB
  constexpr int NSLOT = 5;
  constexpr int NH = BM * 8 / NT;           // 16-byte chunks per thread per half
  constexpr int SMEM = NSLOT * HALF;
  static_assert(BM == BN, "ring slots hold either operand");
  static_assert(BM * (BN * 2 + 16) <= SMEM, "staging tile must fit in LDS");
  static_assert(EPI != EPI_GU || (TN % 2 == 0), "SwiGLU epilogue pairs gate/up blocks");
  static_assert(TM == 4, "the ragged-tile dispatch below covers 0..4 row blocks");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int L = xcd_tile(p);
  if (L < 0) return;
  const TileEntry te = p.table[L];  // per-tile list (tiles_per_entry == 1)
  const int nt = te.nt;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;

  // per-thread byte offset of each LDS chunk it fills (k-step 0) within the
  // operand's buffer: A from the tile's first row (gathered rows: from x),
  // B from the expert's weight matrix
  const char* a_base = GATHER ? reinterpret_cast<const char*>(p.A)
                              : reinterpret_cast<const char*>(p.A + (long long)te.row0 * p.lda);
  const char* b_base = reinterpret_cast<const char*>(p.B + (long long)te.phys * p.strideB);
  uint32_t a_voff[NH], b_voff[NH];
#pragma unroll
  for (int i = 0; i < NH; ++i) {
    const int q = i * NT + tid;
    const int r = q >> 3;
    const int lc = (q & 7) ^ swz8(r);
    const int rr = r < te.rows ? r : te.rows - 1;  // rows past the expert: any valid row
    // gathered rows: the token row of routed row te.row0 + rr (dispatch folded in)
    const long long arow = GATHER ? (long long)(p.row_src[te.row0 + rr] / p.slots_k) : rr;
    a_voff[i] = (uint32_t)((arow * p.lda + lc * 8) * 2);
    b_voff[i] = (uint32_t)(((long long)weight_row<BN, GU_ROWS>(p, nt, r) * p.ldb + lc * 8) * 2);
  }
  const __amdgpu_buffer_rsrc_t a_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a_base), 0, -1, kBufferFlags);
  const __amdgpu_buffer_rsrc_t b_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(b_base), 0, -1, kBufferFlags);
  const int nk = p.K / 64;
  // half h: A of k-step h/2 (h even) or B (h odd), in slot h % 5.  Past the
  // end the last k-step is loaded again (never read), so every iteration
  // issues the same number of loads and one constant vmcnt serves every wait.
  auto issue_half = [&](int h) {
    const int ks = min(h >> 1, nk - 1);
    char* dst = smem + (h % NSLOT) * HALF;
    if (h & 1) dma_chunks<NH, NT>(dst, b_rsrc, b_voff, ks * 128, wave);
    else dma_chunks<NH, NT>(dst, a_rsrc, a_voff, ks * 128, wave);
  };

  // fragment LDS byte offsets within a half for k16 sub-step 0; sub-step s
  // reads logical chunk 2s + lane/32, i.e. byte offset ^ (32 s)
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
    b_off[j] = r * ROWB + ((lc0 ^ swz8(r)) << 4);
  }
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // The main loop, for a wave whose first TMV 32-row MFMA blocks hold rows of
  // the expert (a ragged last tile leaves the others empty: their MFMAs and
  // A-fragment reads are skipped, the loads and barriers are not).
  auto main_loop = [&](auto tmv_tag) {
    constexpr int TMV = decltype(tmv_tag)::value;
    constexpr int NRD = TMV > 0 ? TMV + TN : 0;  // DS reads per k16 sub-step
    constexpr int NMM = TMV * TN;                // MFMAs per k16 sub-step
    u32x4_t fa0[TM], fb0[TN], fa1[TM], fb1[TN];
    // reads in the order the MFMAs consume them (B0 A0 B1 A1 ...)
    auto read_frags = [&](const char* sa, const char* sb, int s, u32x4_t* fa, u32x4_t* fb) {
      if (TMV == 0) return;
#pragma unroll
      for (int i = 0; i < (TMV > TN ? TMV : TN); ++i) {
        if (i < TN) fb[i] = *reinterpret_cast<const u32x4_t*>(sb + (b_off[i] ^ (s << 5)));
        if (i < TMV) fa[i] = *reinterpret_cast<const u32x4_t*>(sa + (a_off[i] ^ (s << 5)));
      }
    };
    auto mma_step = [&](const u32x4_t* fa, const u32x4_t* fb) {
#pragma unroll
      for (int i = 0; i < TMV; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, fb[j]), __builtin_bit_cast(bf16x8_t, fa[i]), acc[i][j],
              0, 0, 0);
    };
    // the next sub-step's fragment reads alternate with this one's MFMAs
    auto interleave = [&]() {
      constexpr int NP = NRD < NMM ? NRD : NMM;
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
      }
      if (NMM > NP) __builtin_amdgcn_sched_group_barrier(0x008, NMM - NP, 0);
      if (NRD > NP) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NP, 0);
    };

    // prologue: halves 0 .. 4 in flight, step 0 (halves 0, 1) landed
#pragma unroll
    for (int h = 0; h < NSLOT; ++h) issue_half(h);
    wait_vmcnt<3 * NH>();
    __builtin_amdgcn_s_barrier();
    int ia = 0, ib = 1;  // slots of the current step's A and B halves
    read_frags(smem, smem + HALF, 0, fa0, fb0);

    for (int kt = 0; kt < nk; ++kt) {
      const char* sa = smem + ia * HALF;
      const char* sb = smem + ib * HALF;
      read_frags(sa, sb, 1, fa1, fb1);
      mma_step(fa0, fb0);
      interleave();
      read_frags(sa, sb, 2, fa0, fb0);
      mma_step(fa1, fb1);
      interleave();
      read_frags(sa, sb, 3, fa1, fb1);
      mma_step(fa0, fb0);
      interleave();
      // step boundary: this thread's reads of step kt are in registers and its
      // loads of step kt+1 have landed (only the A half of step kt+2 may still
      // be in flight); past the barrier the same holds for every thread, so the
      // two halves of step kt are free: they receive B of kt+2 and A of kt+3.
      wait_vmcnt_lgkm0<NH>();
      __builtin_amdgcn_s_barrier();
      issue_half(2 * kt + 5);
      issue_half(2 * kt + 6);
      ia = ia + 2 >= NSLOT ? ia + 2 - NSLOT : ia + 2;
      ib = ib + 2 >= NSLOT ? ib + 2 - NSLOT : ib + 2;
      read_frags(smem + ia * HALF, smem + ib * HALF, 0, fa0, fb0);
      mma_step(fa1, fb1);
      interleave();
    }
  };
  // wave-uniform count of this wave's 32-row blocks that hold expert rows
  const int tmv = min(TM, max(0, (te.rows - wm * WTM + 31) >> 5));
  if (tmv >= TM) main_loop(std::integral_constant<int, TM>{});
  else if (tmv == 3) main_loop(std::integral_constant<int, 3>{});
  else if (tmv == 2) main_loop(std::integral_constant<int, 2>{});
  else if (tmv == 1) main_loop(std::integral_constant<int, 1>{});
  else main_loop(std::integral_constant<int, 0>{});
  // no LDS-DMA may still be writing when the LDS is reused or the workgroup retires
  wait_vmcnt<0>();
  wait_lgkm0();
  __builtin_amdgcn_s_barrier();
  fwd_epilogue<BM, BN, NWM, NWN, EPI>(p, te, nt, acc, smem);
}

// ---------------------------------------------------------------------------
// Persistent variant: one workgroup per CU walks its XCD's contiguous tile
// range, taking tiles from a per-XCD counter (so uneven tiles balance as the
// hardware dispatcher would, without a workgroup launch per tile).  When a
// tile's k-loop ends, the first three halves of the next tile (k-step 0 and
// the A half of k-step 1) go by LDS-DMA into ring slots 0-2 while the
// epilogue stages the finished tile through slots 3-4 (64 KB, one wave row
// of 128 rows per pass); slots 3-4 receive the next tile's halves 3 and 4
// once the epilogue has read them back.  So the next tile's operand latency
// runs under the epilogue instead of after it.
// ---------------------------------------------------------------------------
// Epilogue staged through 64 KB at `stage` (forward only: no act_save).  The
// down product's 256-column Y takes one wave row of 128 rows per pass as
// 512-byte rows; the gate/up product's 128-column H takes all 256 rows in one
// pass as 256-byte rows.  The 16-byte chunks of a staged row are
// XOR-swizzled by row, which spreads a wave's 32 rows over the banks without
// padding.  mid() runs once, after the last staging is published and before
// its flush, when no accumulator is live any more (the caller issues the next
// tile's first copies there).
template <int BM, int BN, int NWM, int NWN, int EPI, typename Mid>
__device__ __forceinline__ void fwd_epilogue_split(const GemmParams& p, const TileEntry& te,
                                                   int nt,
                                                   f32x16_t (&acc)[BM / NWM / 32][BN / NWN / 32],
                                                   char* stage, Mid&& mid) {
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  static_assert(BM == 256 && BN == 256 && NWM == 2, "one wave row of 128 rows per pass");
  constexpr int PROWS = WTM;  // rows per wide pass
  static_assert(PROWS * 512 <= 65536 && BM * 256 <= 65536, "stagings fit the 64 KB");
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;
  const int lrow = lane & 31;
  const int lcol = (lane >> 5) * 4;
  auto st_wide = [&](int r, int col, float a, float b, float c, float d) {
    u32x2_t w = {pack_bf16x2(a, b), pack_bf16x2(c, d)};
    *reinterpret_cast<u32x2_t*>(stage + r * 512 + (((col >> 3) ^ (r & 31)) << 4) + (col & 7) * 2) =
        w;
  };
  auto ld_wide = [&](int r, int cc) {
    return *reinterpret_cast<const u32x4_t*>(stage + r * 512 + ((cc ^ (r & 31)) << 4));
  };
  auto st_h = [&](int r, int col, float a, float b, float c, float d) {
    u32x2_t w = {pack_bf16x2(a, b), pack_bf16x2(c, d)};
    *reinterpret_cast<u32x2_t*>(stage + r * 256 + (((col >> 3) ^ (r & 15)) << 4) + (col & 7) * 2) =
        w;
  };
  auto ld_h = [&](int r, int cc) {
    return *reinterpret_cast<const u32x4_t*>(stage + r * 256 + ((cc ^ (r & 15)) << 4));
  };
  // staged rows [0, ROWS) (global rows row_base + r of the tile), chunks
  // cc0 .. cc0 + CPR - 1 of each, to dst + (te.row0 + row_base + r) * ldd
  // (rows < te.rows, columns < ncols); LDS reads in batches of 4 per wait
  auto flush = [&](auto rows_tag, auto cpr_tag, auto ld, int row_base, bf16_t* dst, long long ldd,
                   int ncols, int cc0) {
    constexpr int ROWS = decltype(rows_tag)::value;
    constexpr int CPR = decltype(cpr_tag)::value;
    constexpr int ITERS = ROWS * CPR / NT;
    constexpr int B = ITERS < 4 ? ITERS : 4;
    static_assert(ROWS * CPR % NT == 0 && ITERS % B == 0, "flush chunks must divide over the threads");
#pragma unroll
    for (int b0 = 0; b0 < ITERS; b0 += B) {
      u32x4_t v[B];
#pragma unroll
      for (int it = 0; it < B; ++it) {
        const int c = (b0 + it) * NT + tid;
        v[it] = ld(c / CPR, cc0 + c % CPR);
      }
#pragma unroll
      for (int it = 0; it < B; ++it) {
        const int c = (b0 + it) * NT + tid;
        const int r = row_base + c / CPR, cc = c % CPR;
        if (r < te.rows && cc * 8 < ncols)
          *reinterpret_cast<u32x4_t*>(dst + (te.row0 + r) * ldd + cc * 8) = v[it];
      }
    }
  };
  auto sync = [&]() {
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
  };
  // the last staging published: every accumulator is in LDS
  auto publish_last = [&]() {
    sync();
    mid();
  };
  using R128 = std::integral_constant<int, PROWS>;
  if (EPI == EPI_GU) {
    const int f = p.f;
    const int fbase = nt * (BN / 2);
    const int fcols = min(BN / 2, f - fbase);
    auto stage_h = [&](int row_off) {  // H = silu(gate) * up of this wave's rows
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = row_off + i * 32 + lrow;
#pragma unroll
        for (int pp = 0; pp < TN / 2; ++pp) {
          const int grp = (wn * WTN) / 64 + pp;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float h[4];
#pragma unroll
            for (int c = 0; c < 4; ++c)
              h[c] = fast_silu(acc[i][2 * pp][q * 4 + c]) * acc[i][2 * pp + 1][q * 4 + c];
            st_h(r, grp * 32 + q * 8 + lcol, h[0], h[1], h[2], h[3]);
          }
        }
      }
    };
    // forward only (act_save takes the ring kernel): all of H in one pass
    stage_h(wm * WTM);
    publish_last();
    flush(std::integral_constant<int, BM>{}, std::integral_constant<int, BN / 16>{}, ld_h, 0,
          p.out + fbase, f, fcols, 0);
    sync();
  } else {
    const int ncols = min(BN, p.N - nt * BN);
    for (int pass = 0; pass < NWM; ++pass) {
      if (wm == pass) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = i * 32 + lrow;
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
              st_wide(r, wn * WTN + j * 32 + q * 8 + lcol, acc[i][j][q * 4], acc[i][j][q * 4 + 1],
                      acc[i][j][q * 4 + 2], acc[i][j][q * 4 + 3]);
        }
      }
      if (pass == NWM - 1) publish_last();
      else sync();
      if (!p.out_tok) {
        flush(R128{}, std::integral_constant<int, BN / 8>{}, ld_wide, pass * PROWS,
              p.out + nt * BN, p.ldo, ncols, 0);
      } else {
        // scatter: routed row r also goes to its token's row of out_tok, times
        // its gate, with the combine's arithmetic (fp32 0 + g * y, one rounding)
        constexpr int CPR = BN / 8, ITERS = PROWS * CPR / NT;
        u32x4_t v[ITERS];
#pragma unroll
        for (int it = 0; it < ITERS; ++it) {
          const int c = it * NT + tid;
          v[it] = ld_wide(c / CPR, c % CPR);
        }
#pragma unroll
        for (int it = 0; it < ITERS; ++it) {
          const int c = it * NT + tid;
          const int r = pass * PROWS + c / CPR, cc = c % CPR;
          if (r < te.rows && cc * 8 < ncols) {
            const long long row = (long long)te.row0 + r;
            if (p.out)
              *reinterpret_cast<u32x4_t*>(p.out + row * p.ldo + nt * BN + cc * 8) = v[it];
            const int src = p.row_src[row];
            const float g = p.gate[src];
            u32x4_t o;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              float lo = 0.0f, hi = 0.0f;
              lo += g * lo_bf16(v[it][w]);
              hi += g * hi_bf16(v[it][w]);
              o[w] = pack_bf16x2(lo, hi);
            }
            *reinterpret_cast<u32x4_t*>(p.out_tok + (long long)(src / p.slots_k) * p.ldo +
                                        nt * BN + cc * 8) = o;
          }
        }
      }
      sync();
    }
  }
}

template <int NWM, int NWN, int EPI, bool GU_ROWS, bool GATHER>
__global__ __launch_bounds__(64 * NWM * NWN) void gemm_nt_persist_kernel(GemmParams p) {
  constexpr int BM = 256, BN = 256;
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int ROWB = 128;                 // bytes per LDS row (64 k)
  constexpr int HALF = BM * ROWB;           // one operand's k-step, 32 KB
  constexpr int NSLOT = 5;
  constexpr int NH = BM * 8 / NT;           // 16-byte chunks per thread per half
  constexpr int SMEM = NSLOT * HALF;
  constexpr int NPRE = 3;                   // halves of the next tile issued before the epilogue
  static_assert(BM == BN, "ring slots hold either operand");
  static_assert(EPI != EPI_GU || (TN % 2 == 0), "SwiGLU epilogue pairs gate/up blocks");
  static_assert(TM == 4, "the ragged-tile dispatch below covers 0..4 row blocks");
  static_assert((NSLOT - NPRE) * HALF >= 65536, "the epilogue stages through the free slots");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  // thread 0's value to every thread through the first LDS word, while no copy
  // is in flight; the second barrier keeps it until every thread has read it.
  // The result is made wave-uniform (readfirstlane), so the tile's table
  // entry is a scalar load and its buffer descriptors stay in SGPRs (a
  // per-lane descriptor would put every LDS-DMA in a waterfall loop).
  auto bcast = [&](int v) {
    if (tid == 0) *reinterpret_cast<volatile int*>(smem) = v;
    __syncthreads();
    const int r = *reinterpret_cast<volatile int*>(smem);
    __syncthreads();
    return __builtin_amdgcn_readfirstlane(r);
  };

  // this XCD's contiguous range of the tile list (block i runs on XCD i % 8)
  const int n_valid = *p.n_entries;  // one tile per entry
  const int per = (n_valid + 7) >> 3;
  const int xcd = blockIdx.x & 7;
  const int t_lo = xcd * per, t_hi = min(t_lo + per, n_valid);
  int* const ctr = p.tile_ctr + xcd;
  // the first tile and the one after it
  const int L = t_lo + bcast(tid == 0 ? atomicAdd(ctr, 1) : 0);
  if (L >= t_hi) return;  // (uniform)

  // per-tile operand addressing, in two steps: the tile's rows (through
  // row_src for gathered A rows; rows past the expert: any valid row), then,
  // once they have arrived, the copies' offsets and descriptors
  TileEntry te;
  uint32_t a_voff[NH], b_voff[NH];
  __amdgpu_buffer_rsrc_t a_rsrc, b_rsrc;
  auto load_rows = [&](const TileEntry& t, uint32_t* raw) {
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      const int r = (i * NT + tid) >> 3;
      const int rr = r < t.rows ? r : t.rows - 1;
      raw[i] = GATHER ? (uint32_t)p.row_src[t.row0 + rr] : (uint32_t)rr;
    }
  };
  auto finish_tile = [&](const uint32_t* raw) {
    const char* a_base = GATHER ? reinterpret_cast<const char*>(p.A)
                                : reinterpret_cast<const char*>(p.A + (long long)te.row0 * p.lda);
    const char* b_base = reinterpret_cast<const char*>(p.B + (long long)te.phys * p.strideB);
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      const int q = i * NT + tid;
      const int r = q >> 3;
      const int lc = (q & 7) ^ swz8(r);
      const long long arow = GATHER ? (long long)(raw[i] / (uint32_t)p.slots_k) : (long long)raw[i];
      a_voff[i] = (uint32_t)((arow * p.lda + lc * 8) * 2);
      b_voff[i] = (uint32_t)(((long long)weight_row<BN, GU_ROWS>(p, te.nt, r) * p.ldb + lc * 8) * 2);
    }
    a_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a_base), 0, -1, kBufferFlags);
    b_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(b_base), 0, -1, kBufferFlags);
  };
  const int nk = p.K / 64;
  // half h of the current tile: A of k-step h/2 (h even) or B (h odd), in
  // slot h % 5.  Past the end the last k-step is loaded again (never read),
  // so every iteration issues the same number of loads and one constant
  // vmcnt serves every wait.
  auto issue_half = [&](int h) {
    const int ks = min(h >> 1, nk - 1);
    char* dst = smem + (h % NSLOT) * HALF;
    if (h & 1) dma_chunks<NH, NT>(dst, b_rsrc, b_voff, ks * 128, wave_s);
    else dma_chunks<NH, NT>(dst, a_rsrc, a_voff, ks * 128, wave_s);
  };

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
    b_off[j] = r * ROWB + ((lc0 ^ swz8(r)) << 4);
  }
  f32x16_t acc[TM][TN];

  // The k-loop of one tile, its halves 0 .. 4 already issued, for a wave
  // whose first TMV 32-row blocks hold rows of the expert.  Thread 0 takes
  // the next tile from the counter at its start (the reply is read after the
  // loop; the loop's in-order waits only grow stricter for an older load).
  int next_raw = 0;
  auto main_loop = [&](auto tmv_tag) {
    constexpr int TMV = decltype(tmv_tag)::value;
    constexpr int NRD = TMV > 0 ? TMV + TN : 0;
    constexpr int NMM = TMV * TN;
    u32x4_t fa0[TM], fb0[TN], fa1[TM], fb1[TN];
    auto read_frags = [&](const char* sa, const char* sb, int s, u32x4_t* fa, u32x4_t* fb) {
      if (TMV == 0) return;
#pragma unroll
      for (int i = 0; i < (TMV > TN ? TMV : TN); ++i) {
        if (i < TN) fb[i] = *reinterpret_cast<const u32x4_t*>(sb + (b_off[i] ^ (s << 5)));
        if (i < TMV) fa[i] = *reinterpret_cast<const u32x4_t*>(sa + (a_off[i] ^ (s << 5)));
      }
    };
    auto mma_step = [&](const u32x4_t* fa, const u32x4_t* fb) {
#pragma unroll
      for (int i = 0; i < TMV; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, fb[j]), __builtin_bit_cast(bf16x8_t, fa[i]), acc[i][j],
              0, 0, 0);
    };
    auto interleave = [&]() {
      constexpr int NP = NRD < NMM ? NRD : NMM;
#pragma unroll
      for (int i = 0; i < NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
      }
      if (NMM > NP) __builtin_amdgcn_sched_group_barrier(0x008, NMM - NP, 0);
      if (NRD > NP) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NP, 0);
    };
    // the fragment offsets are made opaque here, so the offsets each
    // instantiation derives from them are not hoisted out of the tile loop
    // (five instantiations' worth would stay live across every tile)
#pragma unroll
    for (int i = 0; i < TM; ++i) asm volatile("" : "+v"(a_off[i]));
#pragma unroll
    for (int j = 0; j < TN; ++j) asm volatile("" : "+v"(b_off[j]));
    // halves 0 and 1 (step 0) landed: all but the last three halves issued
    wait_vmcnt<3 * NH>();
    __builtin_amdgcn_s_barrier();
    if (tid == 0) next_raw = atomicAdd(ctr, 1);
    int ia = 0, ib = 1;
    read_frags(smem, smem + HALF, 0, fa0, fb0);
    for (int kt = 0; kt < nk; ++kt) {
      const char* sa = smem + ia * HALF;
      const char* sb = smem + ib * HALF;
      read_frags(sa, sb, 1, fa1, fb1);
      mma_step(fa0, fb0);
      interleave();
      read_frags(sa, sb, 2, fa0, fb0);
      mma_step(fa1, fb1);
      interleave();
      read_frags(sa, sb, 3, fa1, fb1);
      mma_step(fa0, fb0);
      interleave();
      wait_vmcnt_lgkm0<NH>();
      __builtin_amdgcn_s_barrier();
      issue_half(2 * kt + 5);
      issue_half(2 * kt + 6);
      ia = ia + 2 >= NSLOT ? ia + 2 - NSLOT : ia + 2;
      ib = ib + 2 >= NSLOT ? ib + 2 - NSLOT : ib + 2;
      read_frags(smem + ia * HALF, smem + ib * HALF, 0, fa0, fb0);
      mma_step(fa1, fb1);
      interleave();
    }
  };

  // One tile ahead: thread 0 asks the counter for the next tile at the start
  // of each k-loop; after the loop its index reaches every thread, its entry
  // and row ids load while this tile's accumulators are staged, and its first
  // three halves go out once the last staging is published (no accumulator
  // live).  Loading the entry and rows during the k-loop instead (vector loads
  // at the first two step boundaries) measured no faster: the chain already
  // overlaps the staging.
  uint32_t raw[NH];
  te = p.table[L];
  load_rows(te, raw);
  finish_tile(raw);

#pragma unroll
  for (int h = 0; h < NSLOT; ++h) issue_half(h);
  while (true) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    const int tmv = min(TM, max(0, (te.rows - wm * WTM + 31) >> 5));
    if (tmv >= TM) main_loop(std::integral_constant<int, TM>{});
    else if (tmv == 3) main_loop(std::integral_constant<int, 3>{});
    else if (tmv == 2) main_loop(std::integral_constant<int, 2>{});
    else if (tmv == 1) main_loop(std::integral_constant<int, 1>{});
    else main_loop(std::integral_constant<int, 0>{});
    // every copy into the ring has landed and every fragment read is done:
    // publish the tile after next, start the next tile's first three halves,
    // then stage and write this one
    wait_vmcnt<0>();
    wait_lgkm0();
    const TileEntry cur = te;
    const int next = t_lo + bcast(next_raw);
    const bool more = next < t_hi;
    if (more) {
      te = p.table[next];
      load_rows(te, raw);
    }
    fwd_epilogue_split<BM, BN, NWM, NWN, EPI>(p, cur, cur.nt, acc, smem + NPRE * HALF, [&]() {
      if (!more) return;
      finish_tile(raw);
#pragma unroll
      for (int h = 0; h < NPRE; ++h) issue_half(h);
    });
    if (!more) break;
#pragma unroll
    for (int h = NPRE; h < NSLOT; ++h) issue_half(h);
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
// The products run persistent (one workgroup per CU, a multiple of 8 so
// every XCD gets the same number, each walking its XCD's tile range through
// p.tile_ctr), except the gate/up product that also writes act_save for the
// backward: its wider epilogue does not fit beside the next tile's first
// copies without spilling, so it keeps one workgroup per tile (ring kernel).
template <int EPI, bool GU, bool GATHER = false>
hipError_t launch_fwd(const GemmParams& p, int max_tiles, hipStream_t s) {
  if (max_tiles <= 0) return hipSuccess;
  if constexpr (EPI == EPI_GU) {
    if (p.out2) {
      hipLaunchKernelGGL((gemm_nt_ring_kernel<2, 4, EPI, GU, GATHER>), dim3(round8(max_tiles)),
                         dim3(512), 0, s, p);
      return hipGetLastError();
    }
  }
  int dev = 0, cus = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err == hipSuccess) err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (err != hipSuccess) return err;
  const int grid = max(8, cus / 8 * 8);
  hipLaunchKernelGGL((gemm_nt_persist_kernel<2, 4, EPI, GU, GATHER>), dim3(grid), dim3(512), 0, s,
                     p);
  return hipGetLastError();
}

constexpr int kFwdBM = 256, kFwdBN = 256;

}  // namespace

// bf16 workspace: H [R, f], then the per-tile lists of the two products
namespace {
inline int fwd_list_max(int64_t R, int E, int n_tiles) { return (ceil_div(R, kFwdBM) + E) * n_tiles; }
}  // namespace

size_t ffn_fwd_ws_bytes(int64_t R, int E, int d, int f, int dtype) {
  if (dtype == kDtypeBf16)
    return align_up((size_t)R * f * 2, 256) +
           table_bytes(fwd_list_max(R, E, ceil_div(f, kFwdBN / 2))) +
           table_bytes(fwd_list_max(R, E, ceil_div(d, kFwdBN)));
  // fp32: H, then one entry per 64-row tile
  return align_up((size_t)R * f * 4, 256) + table_bytes(ceil_div(R, 64) + E);
}

namespace {

// the two products of the forward FFN (and the tile lists), on s
hipError_t launch_ffn_fwd_products(const void* x_perm, const void* w_gu, const void* w_d,
                                   const int32_t* offsets, const int32_t* expert_map, int E,
                                   int d, int f, int64_t R, void* y_perm, void* act_save,
                                   bf16_t* H, void* ws, hipStream_t s, const int32_t* row_src,
                                   int slots_k, const float* gate, void* out_tok) {
  const int nt_gu = ceil_div(f, kFwdBN / 2), nt_d = ceil_div(d, kFwdBN);
  const int max_gu = fwd_list_max(R, E, nt_gu), max_d = fwd_list_max(R, E, nt_d);
  char* tables = static_cast<char*>(ws) + align_up((size_t)R * f * 2, 256);
  TableWs tgu = carve_table(tables, max_gu);
  TableWs td = carve_table(tables + table_bytes(max_gu), max_d);
  const int group = kFwdTileGroup;
  TileList lgu = {nt_gu, group, max_gu, tgu.n_entries, tgu.table};
  TileList ld = {nt_d, group, max_d, td.n_entries, td.table};
  const int list_blocks = ceil_div(max_gu > max_d ? max_gu : max_d, kTableThreads);
  hipLaunchKernelGGL(build_tile_lists_kernel, dim3(list_blocks), dim3(kTableThreads), 0, s,
                     offsets, expert_map, E, kFwdBM, lgu, ld);
  GemmParams g = {};
  g.table = tgu.table;
  g.n_entries = tgu.n_entries;
  g.tile_ctr = tgu.n_entries + kTileCtrOffset;
  g.f = f;
  // gate/up + SwiGLU: B rows interleaved gate/up per 32, BN/2 f-columns per tile
  g.A = static_cast<const bf16_t*>(x_perm);
  g.lda = d;
  g.B = static_cast<const bf16_t*>(w_gu);
  g.ldb = d;
  g.strideB = (long long)2 * f * d;
  g.N = 2 * f;
  g.K = d;
  g.n_tiles_n = nt_gu;
  g.tiles_per_entry = 1;
  g.out = H;
  g.ldo = f;
  g.out2 = static_cast<bf16_t*>(act_save);
  g.row_src = row_src;
  g.slots_k = slots_k;
  hipError_t err = row_src ? launch_fwd<EPI_GU, true, true>(g, max_gu, s)
                           : launch_fwd<EPI_GU, true>(g, max_gu, s);
  if (err != hipSuccess) return err;
  // down projection
  g.table = td.table;
  g.n_entries = td.n_entries;
  g.tile_ctr = td.n_entries + kTileCtrOffset;
  g.A = H;
  g.lda = f;
  g.B = static_cast<const bf16_t*>(w_d);
  g.ldb = f;
  g.strideB = (long long)d * f;
  g.N = d;
  g.K = f;
  g.n_tiles_n = nt_d;
  g.tiles_per_entry = 1;
  g.out = static_cast<bf16_t*>(y_perm);
  g.ldo = d;
  g.out2 = nullptr;
  g.row_src = out_tok ? row_src : nullptr;  // the scatter's token rows (A is H here)
  g.gate = gate;
  g.out_tok = static_cast<bf16_t*>(out_tok);
  return launch_fwd<EPI_STORE, false>(g, max_d, s);
}

}  // namespace

hipError_t launch_ffn_fwd_bf16(const void* x_perm, const void* w_gu, const void* w_d,
                               const int32_t* offsets, const int32_t* expert_map, int E, int d,
                               int f, int64_t R, void* y_perm, void* act_save, void* ws,
                               hipStream_t s, const int32_t* row_src, int slots_k,
                               const float* gate, void* out_tok, void* x_perm_out) {
  bf16_t* H = static_cast<bf16_t*>(ws);
  // x_perm for the weight gradient: written on the side stream beside the FFN
  // (HBM-bound copy against MFMA-bound products), joined before returning
  std::unique_lock<std::mutex> lock;
  SideStream* side = nullptr;
  if (x_perm_out && row_src) {
    hipError_t e = side_stream_acquire(side, lock);
    if (e == hipSuccess) e = side_stream_fork(*side, s);
    if (e == hipSuccess) e = launch_gather_rows(x_perm, row_src, slots_k, R, d, 2, x_perm_out,
                                                side->stream);
    if (e != hipSuccess) {
      if (side) side_stream_join(*side, s);
      return e;
    }
  }
  const hipError_t err = launch_ffn_fwd_products(x_perm, w_gu, w_d, offsets, expert_map, E, d, f,
                                                 R, y_perm, act_save, H, ws, s, row_src, slots_k,
                                                 gate, out_tok);
  if (side) {
    const hipError_t jerr = side_stream_join(*side, s);
    return err != hipSuccess ? err : jerr;
  }
  return err;
}

}  // namespace laep
