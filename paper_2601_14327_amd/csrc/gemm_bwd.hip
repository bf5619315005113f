// Backward grouped GEMMs of the SwiGLU expert FFN (moe_grouped_ffn_bwd) on
// the gfx950 matrix cores:
//   dgrad 1   dH = dY W_d[p]        (A = dY rows, K contiguous; B = W_d [K=d][N=f]),
//             stored as bf16; then an elementwise pass computes the SwiGLU
//             backward at the saved pre-activations: dA, H_b
//             (a fused epilogue that read the pre-activations there cost about
//             55 us per tile: every CU reads and writes ~640 KB at once)
//   dgrad 2   dX = dA W_gu[p]       (A = dA rows; B = W_gu [K=2f][N=d])
//   wgrad     dW_d[p]  = dY^T H_b   (both operands [K = routed rows][features])
//             dW_gu[p] = dA^T X     -> fp32 weight gradients, one tile per expert
//             and output block, the reduction running over the expert's rows.
//
// Same pipeline as the forward kernels: 256 x 256 tiles, 8 waves (2 x 4, each
// 128 x 64), k-steps of 64 through a ring of five 32 KB halves (one operand's
// k-step each), LDS-DMA loads, one barrier per k-step.  A K-contiguous
// operand is stored as in the forward ([256 rows][64 k], 128-byte rows).
// Operands whose K is the strided global dimension are stored as
// [64 k][256 features] rows (512 contiguous bytes per global row segment, so
// every request is a whole line) and turned into MFMA operands with
// ds_read_b64_tr_b16: within each 16-lane group, lane j receives feature j of
// four consecutive k-rows, so two such reads give a lane the same 8
// consecutive k values a ds_read_b128 gives for a K-contiguous operand.  The
// 32-byte block b of k-row r is stored at b ^ ((r & 7) << 1), so the four
// k-rows a group reads fall in different banks.  Rows past the end of an
// expert (the ragged reduction of the weight gradient) fall outside the
// buffer range of the k-step's load and read as zeros.  The epilogues write
// with streaming (non-temporal) stores: every output (dA, H_b, dX, the fp32
// weight gradients) is far larger than the caches (measured 3 % faster on the
// backward call).
//
// Gathered X (the dispatch folded into the weight gradient): dW_gu = dA^T X
// can read X's routed row r straight from token row row_src[r] / k of x, so
// x_perm is never written.  The k-rows of a k-step are then different token
// rows at every step: each thread loads the row_src entries of its 4 k-rows
// one k-step ahead, issued before that iteration's LDS-DMA halves, so the
// in-order vmcnt waits of the ring still cover them.  Rows past the expert's
// end get an offset beyond x's buffer range and read as zeros.
//
// dY formed on load (the gate scaling of the combine backward folded into
// data-gradient 1 and dW_d): their A operand dY = round(g * dout) is read from
// dout's token rows (routed row r: token row row_src[r] / k, times
// gate[row_src[r]], one fp32 product rounded to bf16, exactly as
// moe_combine_bwd forms dy_perm), so dy_perm is never written.  The A halves
// are LDS-DMA'd from dout's token rows through row_src as usual (a gather, as
// in the forward), and each thread scales its own chunks in place just before
// the step boundary at which that half has landed: the ring's prefetch depth
// is unchanged, and the transform's LDS round trip overlaps the last
// sub-step's MFMAs.
#include <type_traits>

#include "gemm_common.hpp"

namespace laep {
namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int kRingRowB = 128;              // K-contiguous half: bytes per row (64 k)
constexpr int kRingHalf = 256 * kRingRowB;   // one operand's k-step: 32 KB
constexpr int kRingSlots = 5;
constexpr int kTrRowB = 512;                 // K-strided half: bytes per k-row (256 features)
constexpr int kTrCpr = kTrRowB / 16;         // 16-byte chunks per k-row
// fourth word of a raw buffer resource: 32-bit data format, no swizzle
constexpr int kBufferFlags = 0x00020000;

// LDS slot q of a TR tile -> (k-row, element column within the tile)
__device__ __forceinline__ void tr_slot(int q, int cpr, int& r, int& col) {
  r = q / cpr;
  const int pc = q % cpr;
  const int lblock = (pc >> 1) ^ ((r & 7) << 1);
  col = lblock * 16 + (pc & 1) * 8;
}

// byte offset, within a TR tile, of the 8 bytes a lane reads in a
// ds_read_b64_tr_b16 for k-row r (fragment column base mf, lane in group i,
// group column half gh)
__device__ __forceinline__ int tr_off(int r, int mf, int gh, int i) {
  const int lblock = (mf >> 4) + gh;
  return r * 512 + ((lblock ^ ((r & 7) << 1)) << 5) + ((i & 3) << 3);
}

// The transposed read through a restrict-qualified pointer, so the read
// carries alias-scope information.  Without it the compiler cannot tell the
// read from the LDS-DMA writes in flight and drains every outstanding load
// (vmcnt(0)) before the first read of each k-step, which serialises the
// ring's prefetch.  The ring's explicit vmcnt waits and barriers already
// order a slot's DMA writes before its reads (as for the plain reads of the
// K-contiguous fragments, which never drew that wait).
__device__ __forceinline__ s16x4_t ds_read_tr(lds_s16x4_t* __restrict__ p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(p);
}

__device__ __forceinline__ u32x4_t read_tr_frag(const char* st, int off1, int off2) {
  const s16x4_t a = ds_read_tr((lds_s16x4_t*)(st + off1));
  const s16x4_t b = ds_read_tr((lds_s16x4_t*)(st + off2));
  const u32x2_t ua = __builtin_bit_cast(u32x2_t, a);
  const u32x2_t ub = __builtin_bit_cast(u32x2_t, b);
  u32x4_t v = {ua[0], ua[1], ub[0], ub[1]};
  return v;
}

// One half (one operand's k-step) of LDS-DMA loads, through buffer loads with
// the LDS flag: NC 16-byte chunks per thread, chunk i of thread tid in LDS
// slot i * NT + tid, at byte voff[i] of the k-step's buffer.  The buffer
// starts at the k-step's first element and ends where the operand's valid
// rows end, so loads past that (the weight gradient's rows past the end of
// the expert) return zeros.  (The global-segment form of this copy makes the
// compiler drain every outstanding LDS read, lgkmcnt(0), before each fragment
// use in the loop; with the buffer form it counts them in order.)  A device
// function, not a lambda: the host pass must not see the LDS-DMA builtin
// inside a lambda.
template <int NC, int NT>
__device__ __forceinline__ void dma_half(char* dst, const char* base, uint32_t extent,
                                         const uint32_t* voff, int wave) {
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, (int)extent, kBufferFlags);
#pragma unroll
  for (int i = 0; i < NC; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)(dst + (i * NT + wave * 64) * 16),
                                             16, voff[i], 0, 0, 0);
}

// 8 bf16 values times g, each an fp32 product rounded to bf16
__device__ __forceinline__ u32x4_t scale_bf16x8(const u32x4_t v, float g) {
  u32x4_t o;
#pragma unroll
  for (int w = 0; w < 4; ++w) o[w] = pack_bf16x2(g * lo_bf16(v[w]), g * hi_bf16(v[w]));
  return o;
}

template <int BM, int BN, int NWM, int NWN, int EPI, bool A_TR, bool B_GATHER, bool A_DY>
__global__ __launch_bounds__(64 * NWM * NWN) void gemm_bwd_kernel(GemmParams p) {
  static_assert(!B_GATHER || EPI == EPI_WGRAD, "only the weight gradient gathers its B rows");
  static_assert(!(A_DY && B_GATHER), "dY on load and gathered B are separate products");
  constexpr int NT = 64 * NWM * NWN;
  constexpr int WTM = BM / NWM, WTN = BN / NWN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int NH = kRingHalf / 16 / NT;  // 16-byte chunks per thread per half
  static_assert(BM == 256 && BN == 256 && NT == 512, "ring halves are 256 x 64 / 64 x 256");
  static_assert(NWM == 2, "the staged epilogues process one wave row per pass");
  constexpr int PITCH16 = BN * 2 + 16;   // bf16 staging pitch
  constexpr int PITCH32 = BN * 4 + 16;   // fp32 staging pitch
  constexpr int EPI_BYTES = (EPI == EPI_WGRAD) ? 128 * PITCH32 : BM * PITCH16;
  constexpr int RING = kRingSlots * kRingHalf;
  constexpr int SMEM = RING > EPI_BYTES ? RING : EPI_BYTES;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  // ---- tile schedule --------------------------------------------------------
  // Row-tile products: tiles of one expert share weight blocks, so each XCD
  // takes a contiguous range of the table.  Weight gradients: the table is
  // ordered longest expert first and tile costs follow the expert's rows, so
  // the tiles of each expert are dealt round-robin over the XCDs (block i
  // runs on XCD i % 8) to keep the eight XCDs equally loaded.
  const int n_valid = (*p.n_entries) * p.tiles_per_entry;
  int L;
  if (EPI == EPI_WGRAD) {
    L = blockIdx.x;
  } else {
    const int per = (n_valid + 7) >> 3;
    const int slot = blockIdx.x >> 3;
    if (slot >= per) return;
    L = (blockIdx.x & 7) * per + slot;
  }
  if (L >= n_valid) return;
  // Tiles are rasterised in groups of p.group row tiles (column blocks in
  // the middle, the group's row tiles innermost), so the workgroups running
  // together touch few operand panels: row-tile products over the table's
  // row-tile entries, weight gradients over each expert's output tiles.
  int entry, mt, nt;
  if (EPI == EPI_WGRAD) {
    entry = L / p.tiles_per_entry;
    const int within = L % p.tiles_per_entry;
    const int MT = p.tiles_per_entry / p.n_tiles_n;   // output row blocks of the expert
    int m, n;
    if (p.xcd_gm > 0) {
      // block i runs on XCD i % 8, and tiles_per_entry % 8 == 0: XCD x takes
      // block (x / gn, x % gn) of the expert's MT x NT tile grid, so each
      // operand panel is fetched by gn (A) or gm (B) XCDs instead of all 8,
      // and every XCD gets the same share of every expert
      const int gm = p.xcd_gm, gn = 8 / gm;
      const int x = within & 7, j = within >> 3;
      const int bm = MT / gm, bn = p.n_tiles_n / gn;
      int mm, nn;
      grouped_tile(j, bm, bn, p.group, mm, nn);
      m = (x / gn) * bm + mm;
      n = (x % gn) * bn + nn;
    } else {
      grouped_tile(within, MT, p.n_tiles_n, p.group, m, n);
    }
    mt = m;
    nt = n;
  } else {
    int m, n;
    grouped_tile(L, *p.n_entries, p.n_tiles_n, p.group, m, n);
    entry = m;
    mt = 0;
    nt = n;
  }
  const TileEntry te = p.table[entry];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave / NWN, wn = wave % NWN;

  // reduction extent of this tile (a multiple of 64 for the data gradients)
  const int kext = (EPI == EPI_WGRAD) ? te.rows : p.K;
  const int nk = (kext + 63) / 64;

  // ---- per-thread DMA offsets within a k-step's buffer ----------------------------
  // A: weight gradient [routed rows][Mw] (k = row, feature = mt*BM + col), or
  // the data gradient's expert rows (K contiguous), from the tile's first row
  uint32_t a_voff[NH];
#pragma unroll
  for (int i = 0; i < NH; ++i) {
    const int q = i * NT + tid;
    if (A_TR) {
      int r, col;
      tr_slot(q, kTrCpr, r, col);
      int c = mt * BM + col;
      c = c < p.Mw ? c : p.Mw - 8;  // columns past Mw: any valid column (not stored)
      a_voff[i] = (uint32_t)(((long long)r * p.lda + c) * 2);
    } else {
      const int r = q >> 3;
      const int lc = (q & 7) ^ swz8(r);
      const int rr = r < te.rows ? r : te.rows - 1;  // rows past the expert: any valid row
      if (A_DY) {  // dY on load: the token row of routed row te.row0 + rr in dout
        const uint32_t s = (uint32_t)p.row_src[te.row0 + rr];
        a_voff[i] = (s / (uint32_t)p.slots_k) * (uint32_t)p.lda * 2u + (uint32_t)(lc * 16);
      } else {
        a_voff[i] = (uint32_t)(((long long)rr * p.lda + lc * 8) * 2);
      }
    }
  }
  const char* a_tile = reinterpret_cast<const char*>(
      A_DY ? p.A : p.A + (long long)te.row0 * p.lda);
  const long long a_kstep = A_TR ? 128LL * p.lda : 128LL;  // bytes per k-step
  // B is K-strided in every backward product: [K][N] rows, feature nt*BN + col
  // (clamped to the last valid column block)
  uint32_t b_voff[NH];
  int b_kr[NH];   // gathered B: k-row of chunk i within a k-step, and its column bytes
  uint32_t b_cb[NH];
#pragma unroll
  for (int i = 0; i < NH; ++i) {
    const int q = i * NT + tid;
    int r, col;
    tr_slot(q, kTrCpr, r, col);
    int c = nt * BN + col;
    c = c < p.N ? c : p.N - 8;
    b_voff[i] = (uint32_t)(((long long)r * p.ldb + c) * 2);
    b_kr[i] = r;
    b_cb[i] = (uint32_t)(c * 2);
  }
  const char* b_tile = reinterpret_cast<const char*>(
      B_GATHER ? p.B
               : (EPI == EPI_WGRAD) ? p.B + (long long)te.row0 * p.ldb
                                    : p.B + (long long)te.phys * p.strideB);
  const long long b_kstep = 128LL * p.ldb;
  // half h: A of k-step h/2 (h even) or B (h odd), in slot h % 5.  Past the
  // end the last k-step is loaded again (never read), so every iteration
  // issues the same number of loads and one constant vmcnt serves every wait.
  // A K-strided operand of the weight gradient ends with the expert's rows.
  auto extent = [&](int ks, int ld) -> uint32_t {
    if (EPI != EPI_WGRAD) return 0xffffffffu;
    const int rem = kext - ks * 64;
    return rem > 0 ? (uint32_t)((long long)min(rem, 64) * ld * 2) : 0u;
  };
  auto issue_half = [&](int h) {
    const int ks = min(h >> 1, nk - 1);
    char* dst = smem + (h % kRingSlots) * kRingHalf;
    if (h & 1) dma_half<NH, NT>(dst, b_tile + b_kstep * ks, extent(ks, p.ldb), b_voff, wave);
    else dma_half<NH, NT>(dst, a_tile + a_kstep * ks, A_TR ? extent(ks, p.lda) : 0xffffffffu,
                          a_voff, wave);
  };
  // gathered B: the row_src entries of this thread's k-rows of step ks and a
  // mask of the valid ones (rows past the expert, and the reloads past the
  // last step, are not); then the DMA offsets they give (invalid rows fall
  // outside x's buffer range).  Branch-free, and the loaded entries are only
  // used at the next k-step, so no wait follows the loads: every load reads
  // an entry of the expert's rows, and the validity is applied at use.
  auto gather_idx = [&](int ks, uint32_t* raw, uint32_t& okm) {
    okm = 0;
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      const int kr = ks * 64 + b_kr[i];
      const bool ok = ks < nk && kr < kext;
      raw[i] = (uint32_t)p.row_src[te.row0 + (ok ? kr : 0)];
      okm |= ok ? (1u << i) : 0u;
    }
  };
  auto gather_voff = [&](const uint32_t* raw, uint32_t okm, uint32_t* v) {
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      const uint32_t off = (raw[i] / (uint32_t)p.slots_k) * (uint32_t)p.ldb * 2u + b_cb[i];
      v[i] = (okm >> i) & 1u ? off : 0x80000000u;
    }
  };
  auto issue_b_gathered = [&](int h, const uint32_t* raw, uint32_t okm) {
    uint32_t v[NH];
    gather_voff(raw, okm, v);
    dma_half<NH, NT>(smem + (h % kRingSlots) * kRingHalf, b_tile, p.b_extent, v, wave);
  };

  // ---- dY formed on load (A_DY) ---------------------------------------------------
  // data gradient 1: the tile's rows are fixed, so each chunk's token-row
  // offset (a_voff, above) and its row's gate are loaded once; dW_d: the
  // k-rows change every step, so (as for a gathered B) each thread loads the
  // row_src entries of its k-rows one step ahead of that step's A half, and the
  // gates with the half
  float ady_g[NH];
  int ady_kr[NH];
  uint32_t ady_cb[NH];
  if constexpr (A_DY && A_TR) {
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      int r, col;
      tr_slot(i * NT + tid, kTrCpr, r, col);
      int c = mt * BM + col;
      c = c < p.Mw ? c : p.Mw - 8;
      ady_kr[i] = r;
      ady_cb[i] = (uint32_t)(c * 2);
    }
  }
  auto ady_idx = [&](int ks, uint32_t* raw, uint32_t& okm) {
    okm = 0;
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      const int kr = ks * 64 + ady_kr[i];
      const bool ok = ks < nk && kr < kext;
      raw[i] = (uint32_t)p.row_src[te.row0 + (ok ? kr : 0)];
      okm |= ok ? (1u << i) : 0u;
    }
  };
  // dW_d: the gathered A half of step ks (rows marked invalid fall outside
  // dout's buffer range and read as zeros), and the gates of its k-rows
  auto ady_issue_tr = [&](int ks, const uint32_t* raw, uint32_t okm, float* g) {
    uint32_t v[NH];
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      const uint32_t off = (raw[i] / (uint32_t)p.slots_k) * (uint32_t)p.lda * 2u + ady_cb[i];
      v[i] = (okm >> i) & 1u ? off : 0x80000000u;
      g[i] = p.gate[raw[i]];
    }
    dma_half<NH, NT>(smem + ((2 * ks) % kRingSlots) * kRingHalf, a_tile, p.a_extent, v, wave);
  };
  // this thread's chunks of the A half of step ks, scaled in place (its own
  // copies have landed; the next barrier publishes the result)
  auto ady_scale = [&](int ks, const float* g) {
    char* slot = smem + ((2 * ks) % kRingSlots) * kRingHalf;
#pragma unroll
    for (int i = 0; i < NH; ++i) {
      u32x4_t* c = reinterpret_cast<u32x4_t*>(slot + (i * NT + tid) * 16);
      *c = scale_bf16x8(*c, g[i]);
    }
  };

  // ---- fragment offsets within a half, k16 sub-step 0 -------------------------------
  const int lc0 = lane >> 5;
  const int gh = (lane >> 4) & 1;
  const int li = lane & 15;
  const int rk = (lane >> 5) * 8 + (li >> 2);  // first k-row of the lane's TR reads
  int a_o1[TM], a_o2[TM], b_o1[TN], b_o2[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    if (A_TR) {
      const int mf = wm * WTM + i * 32;
      a_o1[i] = tr_off(rk, mf, gh, li);
      a_o2[i] = tr_off(rk + 4, mf, gh, li);
    } else {
      const int r = wm * WTM + i * 32 + (lane & 31);
      a_o1[i] = r * kRingRowB + ((lc0 ^ swz8(r)) << 4);
      a_o2[i] = 0;
    }
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int mf = wn * WTN + j * 32;
    b_o1[j] = tr_off(rk, mf, gh, li);
    b_o2[j] = tr_off(rk + 4, mf, gh, li);
  }

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // The main loop, for a wave whose first TMV 32-row MFMA blocks hold rows of
  // the tile (the data gradients' ragged last row tile leaves the others
  // empty: their MFMAs and A-fragment reads are skipped, loads and barriers
  // are not).  Weight-gradient tiles are always full.
  auto main_loop = [&](auto tmv_tag) {
    constexpr int TMV = decltype(tmv_tag)::value;
    u32x4_t fa0[TM], fb0[TN], fa1[TM], fb1[TN];
    // k16 sub-step s of a k-step: K-contiguous fragments flip the logical
    // chunk by 2 (byte offset ^ 32 s); TR fragments move down 16 k-rows
    auto read_frags = [&](const char* sa, const char* sb, int s, u32x4_t* fa, u32x4_t* fb) {
      if (TMV == 0) return;
#pragma unroll
      for (int i = 0; i < (TMV > TN ? TMV : TN); ++i) {
        if (i < TN) fb[i] = read_tr_frag(sb, b_o1[i] + s * 16 * kTrRowB, b_o2[i] + s * 16 * kTrRowB);
        if (i < TMV) {
          if (A_TR) fa[i] = read_tr_frag(sa, a_o1[i] + s * 16 * kTrRowB, a_o2[i] + s * 16 * kTrRowB);
          else fa[i] = *reinterpret_cast<const u32x4_t*>(sa + (a_o1[i] ^ (s << 5)));
        }
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

    // prologue: halves 0 .. 4 in flight, step 0 (halves 0, 1) landed
    uint32_t idx_next[NH], ok_next = 0;  // gathered B: row_src of the next B half to issue
    // dY on load: the gates of the A halves landed or in flight (dW_d: of
    // steps kt+1 and kt+2 at step kt's boundary) and the row_src entries of the
    // next A half to issue
    float ady_g1[NH], ady_g2[NH];
    uint32_t ady_src[NH], ady_ok = 0;
    if constexpr (A_DY) {
      float g0[NH];
      if constexpr (A_TR) {
        uint32_t s0[NH], s1[NH], s2[NH], ok0, ok1, ok2;
        ady_idx(0, s0, ok0);
        ady_idx(1, s1, ok1);
        ady_idx(2, s2, ok2);
        ady_idx(3, ady_src, ady_ok);
        ady_issue_tr(0, s0, ok0, g0);
        issue_half(1);
        ady_issue_tr(1, s1, ok1, ady_g1);
        issue_half(3);
        ady_issue_tr(2, s2, ok2, ady_g2);
      } else {
#pragma unroll
        for (int i = 0; i < NH; ++i) {   // data gradient 1: the chunk rows' gates, once
          const int rr = min((i * NT + tid) >> 3, te.rows - 1);
          ady_g[i] = p.gate[p.row_src[te.row0 + rr]];
          g0[i] = ady_g[i];
        }
#pragma unroll
        for (int h = 0; h < kRingSlots; ++h) issue_half(h);
      }
      wait_vmcnt<3 * NH>();
      ady_scale(0, g0);
      wait_lgkm0();
    } else if constexpr (B_GATHER) {
      uint32_t idx0[NH], idx1[NH], ok0, ok1;
      gather_idx(0, idx0, ok0);
      gather_idx(1, idx1, ok1);
      gather_idx(2, idx_next, ok_next);
      issue_half(0);
      issue_b_gathered(1, idx0, ok0);
      issue_half(2);
      issue_b_gathered(3, idx1, ok1);
      issue_half(4);
    } else {
#pragma unroll
      for (int h = 0; h < kRingSlots; ++h) issue_half(h);
    }
    if constexpr (!A_DY) wait_vmcnt<3 * NH>();
    __builtin_amdgcn_s_barrier();
    int ia = 0, ib = 1;  // slots of the current step's A and B halves
    read_frags(smem, smem + kRingHalf, 0, fa0, fb0);
    for (int kt = 0; kt < nk; ++kt) {
      const char* sa = smem + ia * kRingHalf;
      const char* sb = smem + ib * kRingHalf;
      read_frags(sa, sb, 1, fa1, fb1);
      mma_step(fa0, fb0);
      read_frags(sa, sb, 2, fa0, fb0);
      mma_step(fa1, fb1);
      if constexpr (A_DY) {
        // dY on load: this thread's copies of the A half of step kt+1 have
        // landed once only the halves issued after it may be in flight (two
        // iterations' worth: 2 or, for dW_d with its row_src and gate loads, 4
        // groups of NH); scale them here, beside the MFMAs, so the LDS round
        // trip stays off the step boundary (the boundary's lgkmcnt(0) and
        // barrier publish them)
        wait_vmcnt<(A_TR ? 8 : 4) * NH>();
        ady_scale(kt + 1, A_TR ? ady_g1 : ady_g);
      }
      read_frags(sa, sb, 3, fa1, fb1);
      mma_step(fa0, fb0);
      // step boundary: this thread's reads of step kt are in registers and its
      // loads of step kt+1 have landed (only the A half of step kt+2 may still
      // be in flight); past the barrier the same holds for every thread, so the
      // two halves of step kt are free: they receive B of kt+2 and A of kt+3.
      wait_vmcnt_lgkm0<NH>();
      __builtin_amdgcn_s_barrier();
      if constexpr (A_DY && A_TR) {
        // dW_d: the gates move down a step; the A half of kt+3 (row_src loaded
        // last iteration) with its gates; the row_src entries of kt+4 first,
        // so the next boundary's wait covers them
#pragma unroll
        for (int i = 0; i < NH; ++i) ady_g1[i] = ady_g2[i];
        uint32_t src3[NH];
#pragma unroll
        for (int i = 0; i < NH; ++i) src3[i] = ady_src[i];
        const uint32_t ok3 = ady_ok;
        ady_idx(kt + 4, ady_src, ady_ok);
        issue_half(2 * kt + 5);
        ady_issue_tr(kt + 3, src3, ok3, ady_g2);
      } else if constexpr (B_GATHER) {
        // the offsets of B(kt + 2) from the entries loaded last iteration; the
        // entries of step kt + 3 are loaded before this iteration's halves,
        // so the next boundary's wait covers them
        uint32_t v[NH];
        gather_voff(idx_next, ok_next, v);
        gather_idx(kt + 3, idx_next, ok_next);
        dma_half<NH, NT>(smem + ((2 * kt + 5) % kRingSlots) * kRingHalf, b_tile, p.b_extent, v,
                         wave);
      } else {
        issue_half(2 * kt + 5);
      }
      if constexpr (!(A_DY && A_TR)) issue_half(2 * kt + 6);
      ia = ia + 2 >= kRingSlots ? ia + 2 - kRingSlots : ia + 2;
      ib = ib + 2 >= kRingSlots ? ib + 2 - kRingSlots : ib + 2;
      read_frags(smem + ia * kRingHalf, smem + ib * kRingHalf, 0, fa0, fb0);
      mma_step(fa1, fb1);
    }
    // no LDS-DMA may still be writing when the LDS is reused for staging
    wait_vmcnt<0>();
  };

  if (nk > 0) {
    if (EPI == EPI_WGRAD) {
      main_loop(std::integral_constant<int, TM>{});
    } else {
      static_assert(EPI == EPI_WGRAD || TM == 4, "the ragged-tile dispatch covers 0..4 blocks");
      const int tmv = min(TM, max(0, (te.rows - wm * WTM + 31) >> 5));
      if (tmv >= TM) main_loop(std::integral_constant<int, TM>{});
      else if (tmv == 3) main_loop(std::integral_constant<int, 3>{});
      else if (tmv == 2) main_loop(std::integral_constant<int, 2>{});
      else if (tmv == 1) main_loop(std::integral_constant<int, 1>{});
      else main_loop(std::integral_constant<int, 0>{});
    }
  }

  // ---- epilogues (staged through LDS) -------------------------------------------
  wait_lgkm0();
  __builtin_amdgcn_s_barrier();
  const int lrow = lane & 31;
  const int lcol = (lane >> 5) * 4;

  if (EPI == EPI_WGRAD) {
    // fp32 dW tile, 128 rows (one wave row) per pass
    float* W = p.wout + (long long)te.phys * p.strideW;
    const int ncols = min(BN, p.N - nt * BN);
    for (int pass = 0; pass < 2; ++pass) {
      if (wm == pass) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int r = i * 32 + lrow;
              const int c = wn * WTN + j * 32 + q * 8 + lcol;
              f32x4_t v = {acc[i][j][q * 4], acc[i][j][q * 4 + 1], acc[i][j][q * 4 + 2],
                           acc[i][j][q * 4 + 3]};
              *reinterpret_cast<f32x4_t*>(smem + r * PITCH32 + c * 4) = v;
            }
      }
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      // fixed trip count (BN columns): every LDS read of a thread before one wait
      constexpr int CPR = BN / 4, ITERS = 128 * CPR / NT;
      const int cpr = ncols / 4;
      f32x4_t v[ITERS];
#pragma unroll
      for (int it = 0; it < ITERS; ++it) {
        const int c = it * NT + tid;
        v[it] = *reinterpret_cast<const f32x4_t*>(smem + (c / CPR) * PITCH32 + (c % CPR) * 16);
      }
#pragma unroll
      for (int it = 0; it < ITERS; ++it) {
        const int c = it * NT + tid;
        const int r = c / CPR, cc = c % CPR;
        const int row = mt * BM + pass * 128 + r;
        if (row < p.Mw && cc < cpr) {
          f32x4_t* dst = reinterpret_cast<f32x4_t*>(W + (long long)row * p.N + nt * BN + cc * 4);
          if (p.accumulate) v[it] += *dst;
          st_stream(dst, v[it]);
        }
      }
      wait_lgkm0();
      __builtin_amdgcn_s_barrier();
    }
  } else {  // EPI_STORE (bf16 rows: dH, dX)
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int r = wm * WTM + i * 32 + lrow;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = wn * WTN + j * 32 + q * 8 + lcol;
          u32x2_t w = {pack_bf16x2(acc[i][j][q * 4], acc[i][j][q * 4 + 1]),
                       pack_bf16x2(acc[i][j][q * 4 + 2], acc[i][j][q * 4 + 3])};
          *reinterpret_cast<u32x2_t*>(smem + r * PITCH16 + c * 2) = w;
        }
    }
    wait_lgkm0();
    __syncthreads();
    const int ncols = min(BN, p.N - nt * BN);
    const int cpr = ncols / 8;
    constexpr int CPR = BN / 8, ITERS = BM * CPR / NT;
    u32x4_t v[ITERS];
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * NT + tid;
      v[it] = *reinterpret_cast<const u32x4_t*>(smem + (c / CPR) * PITCH16 + (c % CPR) * 16);
    }
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int c = it * NT + tid;
      const int r = c / CPR, cc = c % CPR;
      if (r < te.rows && cc < cpr) {
        bf16_t* dst = p.out + (long long)(te.row0 + r) * p.ldo + nt * BN + cc * 8;
        st_stream(reinterpret_cast<u32x4_t*>(dst), v[it]);
      }
    }
  }
}

// SwiGLU backward at the saved pre-activations, one 8-column vector of one
// routed row per thread: with s = sigmoid(A_g),
//   dA_g = dH A_u s (1 + A_g (1 - s)),  dA_u = dH silu(A_g),  H_b = silu(A_g) A_u.
// dH arrives in the H_b buffer and is replaced there by H_b (write_h), or left
// (the weight gradient then uses the forward's H).  Streaming accesses: every
// element is read and written once.
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const u32x4_t* __restrict__ act,
                                                         int64_t R, int f,
                                                         u32x4_t* __restrict__ dA,
                                                         u32x4_t* __restrict__ hb, int write_h) {
  const int vpr = f / 8;  // vectors per row of dH / H_b
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= R * vpr) return;
  const long long r = i / vpr;
  const int v = (int)(i % vpr);
  const u32x4_t dh = ld_stream(hb + i);
  const u32x4_t g = ld_stream(act + r * 2 * vpr + v);
  const u32x4_t u = ld_stream(act + r * 2 * vpr + vpr + v);
  u32x4_t og, ou, oh;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float dag[2], dau[2], h[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float d = e ? hi_bf16(dh[w]) : lo_bf16(dh[w]);
      const float ag = e ? hi_bf16(g[w]) : lo_bf16(g[w]);
      const float au = e ? hi_bf16(u[w]) : lo_bf16(u[w]);
      const float sg = fast_sigmoid(ag);
      const float sl = ag * sg;
      dag[e] = d * au * sg * (1.0f + ag * (1.0f - sg));
      dau[e] = d * sl;
      h[e] = sl * au;
    }
    og[w] = pack_bf16x2(dag[0], dag[1]);
    ou[w] = pack_bf16x2(dau[0], dau[1]);
    oh[w] = pack_bf16x2(h[0], h[1]);
  }
  st_stream(dA + r * 2 * vpr + v, og);
  st_stream(dA + r * 2 * vpr + vpr + v, ou);
  if (write_h) st_stream(hb + i, oh);
}

constexpr int kBwdBM = 256, kBwdBN = 256;

// The XCD blocking of a weight gradient's tile grid (MT x NT tiles per
// expert; A has Mw features, B N): the split gm x gn = 8 with gm | MT and
// gn | NT that fetches the fewest panel bytes (A panels gn times, B panels gm
// times), or 0 when none divides.
int wgrad_xcd_gm(int MT, int NT, int Mw, int N) {
  int best = 0;
  long long best_cost = 0;
  for (int gm = 1; gm <= 8; gm *= 2) {
    const int gn = 8 / gm;
    if (MT % gm || NT % gn) continue;
    const long long cost = (long long)gn * Mw + (long long)gm * N;
    if (!best || cost < best_cost) {
      best = gm;
      best_cost = cost;
    }
  }
  return best;
}

template <int EPI, bool A_TR, bool B_GATHER = false, bool A_DY = false>
hipError_t launch_bwd(const GemmParams& p, int grid, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_bwd_kernel<kBwdBM, kBwdBN, 2, 4, EPI, A_TR, B_GATHER, A_DY>),
                     dim3(round8(grid)), dim3(512), 0, s, p);
  return hipGetLastError();
}

}  // namespace

size_t ffn_bwd_hb_offset(int64_t R, int f, int dtype) {
  const size_t elem = dtype == kDtypeBf16 ? 2 : 4;
  return align_up((size_t)R * 2 * f * elem, 256);
}

size_t ffn_bwd_ws_bytes(int64_t R, int E, int d, int f, int dtype) {
  (void)d;
  const size_t elem = dtype == kDtypeBf16 ? 2 : 4;
  return ffn_bwd_hb_offset(R, f, dtype) + align_up((size_t)R * f * elem, 256) +
         table_bytes(ceil_div(R, kBwdBM) + E) + table_bytes(E);
}

hipError_t launch_ffn_bwd_bf16(const void* dy, const void* x_perm, const void* act_save,
                               const void* h_fwd, const void* w_gu, const void* w_d,
                               const int32_t* offsets, const int32_t* expert_map, int E, int d,
                               int f, int64_t R, void* dx_perm, float* dw_gu, float* dw_d,
                               int accumulate, void* ws, hipStream_t s, const int32_t* row_src,
                               int slots_k, int64_t x_rows, const void* dout,
                               const float* gate) {
  // dy == NULL: data gradient 1 and dW_d form dY on load from dout and the gates
  const bool dy_on_load = dy == nullptr;
  char* base = static_cast<char*>(ws);
  bf16_t* dA = reinterpret_cast<bf16_t*>(base);
  bf16_t* Hb = reinterpret_cast<bf16_t*>(base + ffn_bwd_hb_offset(R, f, kDtypeBf16));
  char* tables = base + ffn_bwd_hb_offset(R, f, kDtypeBf16) + align_up((size_t)R * f * 2, 256);
  const int max_ragged = ceil_div(R, kBwdBM) + E;
  TableWs tr = carve_table(tables, max_ragged);
  TableWs te = carve_table(tables + table_bytes(max_ragged), E);
  hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, expert_map,
                     E, kBwdBM, 0, max_ragged, tr.n_entries, tr.table);
  hipLaunchKernelGGL(build_table_kernel, dim3(1), dim3(kTableThreads), 0, s, offsets, expert_map,
                     E, kBwdBM, 1, E, te.n_entries, te.table);

  const int group = kBwdTileGroup;
  // weight gradients: dW_d[p] [d, f] = dY^T H over the expert's rows (H: the
  // forward's when given, else H_b), dW_gu[p] [2f, d] = dA^T X
  GemmParams wd = {};
  wd.group = group;
  wd.table = te.table;
  wd.n_entries = te.n_entries;
  wd.f = f;
  wd.A = static_cast<const bf16_t*>(dy_on_load ? dout : dy);
  wd.lda = d;
  wd.row_src = row_src;
  wd.slots_k = slots_k;
  wd.gate = gate;
  wd.a_extent = (uint32_t)(x_rows * d * 2);
  wd.B = h_fwd ? static_cast<const bf16_t*>(h_fwd) : Hb;
  wd.ldb = f;
  wd.Mw = d;
  wd.N = f;
  wd.n_tiles_n = ceil_div(f, kBwdBN);
  wd.tiles_per_entry = ceil_div(d, kBwdBM) * wd.n_tiles_n;
  wd.wout = dw_d;
  wd.strideW = (long long)d * f;
  wd.accumulate = accumulate;
  wd.xcd_gm = wgrad_xcd_gm(ceil_div(d, kBwdBM), wd.n_tiles_n, d, f);
  GemmParams wg = wd;
  wg.A = dA;
  wg.lda = 2 * f;
  wg.B = static_cast<const bf16_t*>(x_perm);   // token rows x when gathering
  wg.ldb = d;
  wg.row_src = row_src;
  wg.slots_k = slots_k;
  wg.b_extent = (uint32_t)(x_rows * d * 2);
  wg.Mw = 2 * f;
  wg.N = d;
  wg.n_tiles_n = ceil_div(d, kBwdBN);
  wg.tiles_per_entry = ceil_div(2 * f, kBwdBM) * wg.n_tiles_n;
  wg.wout = dw_gu;
  wg.strideW = (long long)2 * f * d;
  wg.xcd_gm = wgrad_xcd_gm(ceil_div(2 * f, kBwdBM), wg.n_tiles_n, 2 * f, d);

  // The weight gradients run on the side stream, concurrently with the data
  // gradients: dW_d from the start when it uses the forward's H, else after
  // the SwiGLU backward like dW_gu; joined back (also after an error) before
  // the call returns.
  std::unique_lock<std::mutex> lock;
  SideStream* side = nullptr;
  hipError_t err = side_stream_acquire(side, lock);
  if (err != hipSuccess) return err;
  const hipStream_t s2 = side->stream;
  auto fork = [&]() { return side_stream_fork(*side, s); };
  if ((err = fork()) != hipSuccess) return err;
  auto launch_dw_d = [&]() {
    return dy_on_load ? launch_bwd<EPI_WGRAD, true, false, true>(wd, E * wd.tiles_per_entry, s2)
                      : launch_bwd<EPI_WGRAD, true>(wd, E * wd.tiles_per_entry, s2);
  };
  if (h_fwd) err = launch_dw_d();

  // dgrad 1: dH = dY W_d (bf16, into the H_b buffer), then the SwiGLU backward -> dA (, H_b)
  GemmParams g = {};
  g.group = group;
  g.table = tr.table;
  g.n_entries = tr.n_entries;
  g.f = f;
  g.A = static_cast<const bf16_t*>(dy_on_load ? dout : dy);
  g.lda = d;
  g.row_src = row_src;
  g.slots_k = slots_k;
  g.gate = gate;
  g.a_extent = (uint32_t)(x_rows * d * 2);
  g.B = static_cast<const bf16_t*>(w_d);
  g.ldb = f;
  g.strideB = (long long)d * f;
  g.N = f;
  g.K = d;
  g.n_tiles_n = ceil_div(f, kBwdBN);
  g.tiles_per_entry = g.n_tiles_n;
  g.out = Hb;
  g.ldo = f;
  if (err == hipSuccess)
    err = dy_on_load ? launch_bwd<EPI_STORE, false, false, true>(g, max_ragged * g.n_tiles_n, s)
                     : launch_bwd<EPI_STORE, false>(g, max_ragged * g.n_tiles_n, s);
  if (err == hipSuccess && R > 0) {
    const long long n_vec = R * (long long)(f / 8);
    hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)((n_vec + 255) / 256)), dim3(256), 0, s,
                       static_cast<const u32x4_t*>(act_save), (int64_t)R, f,
                       reinterpret_cast<u32x4_t*>(dA), reinterpret_cast<u32x4_t*>(Hb),
                       h_fwd ? 0 : 1);
    err = hipGetLastError();
  }
  // dA (and H_b) ready: the remaining weight gradients on the side stream
  if (err == hipSuccess) err = fork();
  if (err == hipSuccess && !h_fwd) err = launch_dw_d();
  if (err == hipSuccess)
    err = row_src ? launch_bwd<EPI_WGRAD, true, true>(wg, E * wg.tiles_per_entry, s2)
                  : launch_bwd<EPI_WGRAD, true>(wg, E * wg.tiles_per_entry, s2);

  // dgrad 2: dX = dA W_gu
  g.A = dA;
  g.lda = 2 * f;
  g.B = static_cast<const bf16_t*>(w_gu);
  g.ldb = d;
  g.strideB = (long long)2 * f * d;
  g.N = d;
  g.K = 2 * f;
  g.n_tiles_n = ceil_div(d, kBwdBN);
  g.tiles_per_entry = g.n_tiles_n;
  g.out = static_cast<bf16_t*>(dx_perm);
  g.ldo = d;
  if (err == hipSuccess) err = launch_bwd<EPI_STORE, false>(g, max_ragged * g.n_tiles_n, s);
  const hipError_t jerr = side_stream_join(*side, s);
  return err != hipSuccess ? err : jerr;
}

}  // namespace laep
