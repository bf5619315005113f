// C-ABI entry points (include/laep_moe.h): argument validation, workspace
// sizing and kernel dispatch.  Validation is pure host code and runs before
// any HIP call, so an invalid call enqueues nothing.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "../../include/laep_moe.h"
#include "../../include/laep_calib.h"
#include "internal.hpp"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return LAEP_OK;
}

int hip_status(hipError_t e, const char* where) {
  if (e != hipSuccess) return fail(LAEP_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE(cond, code, ...) \
  do {                           \
    if (!(cond)) return fail(code, __VA_ARGS__); \
  } while (0)

int check_dtype(int dtype) {
  if (dtype != LAEP_F32 && dtype != LAEP_BF16)
    return fail(LAEP_ERR_UNSUPPORTED, "dtype %d is not LAEP_F32 (0) or LAEP_BF16 (1)", dtype);
  return LAEP_OK;
}

int check_experts(int E, int k) {
  REQUIRE(E >= 1 && E <= LAEP_MAX_EXPERTS, LAEP_ERR_INVALID_ARG, "E=%d outside [1, %d]", E,
          LAEP_MAX_EXPERTS);
  REQUIRE(k >= 1 && k <= E, LAEP_ERR_INVALID_ARG, "k=%d outside [1, E=%d]", k, E);
  return LAEP_OK;
}

int check_rows(int T, int k, int d_model) {
  REQUIRE(T >= 0, LAEP_ERR_INVALID_ARG, "T=%d < 0", T);
  REQUIRE(d_model > 0 && d_model % 8 == 0, LAEP_ERR_INVALID_ARG,
          "d_model=%d must be a positive multiple of 8", d_model);
  REQUIRE((long long)T * k <= 0x7FFFFFFFll, LAEP_ERR_INVALID_ARG, "T*k=%lld exceeds int32",
          (long long)T * k);
  return LAEP_OK;
}

size_t elem_bytes(int dtype) { return dtype == LAEP_BF16 ? 2 : 4; }

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// extent of a buffer the bf16 GEMMs address with 32-bit byte offsets
constexpr int64_t kMaxBufferBytes = (int64_t)1 << 31;

int check_ffn_shape(int dtype, int E, int d_model, int d_ff, int64_t R) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  REQUIRE(E >= 1 && E <= LAEP_MAX_EXPERTS, LAEP_ERR_INVALID_ARG, "E=%d outside [1, %d]", E,
          LAEP_MAX_EXPERTS);
  REQUIRE(R >= 0 && R <= 0x7FFFFFFFll, LAEP_ERR_INVALID_ARG, "R=%lld outside [0, 2^31)",
          (long long)R);
  REQUIRE(d_model > 0 && d_ff > 0, LAEP_ERR_INVALID_ARG, "d_model=%d, d_ff=%d must be > 0",
          d_model, d_ff);
  REQUIRE(d_model % 64 == 0 && d_ff % 64 == 0, LAEP_ERR_UNSUPPORTED,
          "d_model=%d and d_ff=%d must be multiples of 64", d_model, d_ff);
  // the bf16 GEMMs address one expert's weights with 32-bit byte offsets
  REQUIRE(dtype != LAEP_BF16 || (int64_t)4 * d_ff * d_model < kMaxBufferBytes,
          LAEP_ERR_UNSUPPORTED, "bf16: one expert's w_gate_up (2*d_ff*d_model) must be under 2 GiB");
  return LAEP_OK;
}

}  // namespace

extern "C" {

const char* laep_last_error(void) { return g_err; }

size_t moe_workspace_bytes(int which_call, int T, int k, int E, int d_model, int d_ff) {
  if (T < 0 || k < 1 || E < 1 || E > LAEP_MAX_EXPERTS) return 0;
  const int64_t R = (int64_t)T * k;
  switch (which_call) {
    case LAEP_CALL_ROUTE:
      return 0;
    case LAEP_CALL_COUNTS:
      return laep::counts_ws_bytes(T, k, E);
    case LAEP_CALL_FFN_FWD: {
      // large enough for either dtype
      const size_t a = laep::ffn_fwd_ws_bytes(R, E, d_model, d_ff, laep::kDtypeF32);
      const size_t b = laep::ffn_fwd_ws_bytes(R, E, d_model, d_ff, laep::kDtypeBf16);
      return a > b ? a : b;
    }
    case LAEP_CALL_FFN_BWD:
      return laep::ffn_bwd_ws_bytes(R, E, d_model, d_ff, laep::kDtypeBf16);
    case LAEP_CALL_ROUTE_BWD:
      return laep::route_bwd_ws_bytes(T, k, E, d_model < 0 ? 0 : d_model);
    default:
      return 0;
  }
}

size_t laep_ws_hb_offset(int64_t R, int d_ff, int dtype) {
  return laep::ffn_bwd_hb_offset(R, d_ff, dtype);
}

int moe_route(const void* x, const void* w_router, const float* bias, const uint8_t* alive,
              int dtype, int T, int d_model, int E, int k, int renorm, float* logits,
              int32_t* topk_idx, float* topk_gate, void* ws, size_t ws_bytes, void* stream) {
  (void)ws;
  (void)ws_bytes;
  int rc = check_dtype(dtype);
  if (rc) return rc;
  if ((rc = check_experts(E, k))) return rc;
  if ((rc = check_rows(T, k, d_model))) return rc;
  if (T == 0) return ok();
  REQUIRE(x && w_router && topk_idx && topk_gate, LAEP_ERR_INVALID_ARG,
          "moe_route: x, w_router, topk_idx and topk_gate must be non-null");
  REQUIRE(aligned16(x) && aligned16(w_router), LAEP_ERR_INVALID_ARG,
          "moe_route: x and w_router must be 16-byte aligned");
  return hip_status(laep::launch_route(x, w_router, bias, alive, dtype, T, d_model, E, k,
                                       renorm != 0, logits, topk_idx, topk_gate, nullptr,
                                       as_stream(stream)),
                    "moe_route");
}

int moe_expert_counts(const int32_t* topk_idx, int T, int k, int E, int32_t* counts,
                      int32_t* offsets, int32_t* dest_row, int32_t* row_src, int64_t* etn_accum,
                      void* ws, size_t ws_bytes, void* stream) {
  int rc = check_experts(E, k);
  if (rc) return rc;
  REQUIRE(T >= 0, LAEP_ERR_INVALID_ARG, "T=%d < 0", T);
  REQUIRE((long long)T * k <= 0x7FFFFFFFll, LAEP_ERR_INVALID_ARG, "T*k exceeds int32");
  REQUIRE(counts && offsets, LAEP_ERR_INVALID_ARG,
          "moe_expert_counts: counts and offsets must be non-null");
  REQUIRE(T == 0 || (topk_idx && dest_row), LAEP_ERR_INVALID_ARG,
          "moe_expert_counts: topk_idx and dest_row must be non-null");
  const size_t need = laep::counts_ws_bytes(T, k, E);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE, "moe_expert_counts: workspace %zu < %zu bytes",
          ws_bytes, need);
  REQUIRE(need == 0 || ws, LAEP_ERR_INVALID_ARG, "moe_expert_counts: ws must be non-null");
  return hip_status(laep::launch_counts(topk_idx, T, k, E, counts, offsets, dest_row, row_src,
                                        etn_accum, ws, as_stream(stream)),
                    "moe_expert_counts");
}

}  // extern "C"

namespace {

// argument checks shared by moe_route_count and moe_route_count_noalloc
int check_route_count(const char* name, const void* x, const void* w_router, int dtype, int T,
                      int d_model, int E, int k, const int32_t* topk_idx, const float* topk_gate,
                      const int32_t* counts, const int32_t* offsets, const int32_t* dest_row) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  if ((rc = check_experts(E, k))) return rc;
  if ((rc = check_rows(T, k, d_model))) return rc;
  REQUIRE(counts && offsets, LAEP_ERR_INVALID_ARG, "%s: counts and offsets must be non-null",
          name);
  if (T > 0) {
    REQUIRE(x && w_router && topk_idx && topk_gate && dest_row, LAEP_ERR_INVALID_ARG,
            "%s: x, w_router, topk_idx, topk_gate and dest_row must be non-null", name);
    REQUIRE(aligned16(x) && aligned16(w_router), LAEP_ERR_INVALID_ARG,
            "%s: x and w_router must be 16-byte aligned", name);
  }
  return LAEP_OK;
}

// the launches of the fused route + count call, on a checked workspace
int route_count_launch(const char* name, const void* x, const void* w_router, const float* bias,
                       const uint8_t* alive, int dtype, int T, int d_model, int E, int k,
                       int renorm, float* logits, int32_t* topk_idx, float* topk_gate,
                       int32_t* counts, int32_t* offsets, int32_t* dest_row, int32_t* row_src,
                       int64_t* etn_accum, void* ws, void* stream) {
  const hipStream_t s = as_stream(stream);
  hipError_t e = laep::launch_route(x, w_router, bias, alive, dtype, T, d_model, E, k,
                                    renorm != 0, logits, topk_idx, topk_gate,
                                    T > 0 ? laep::counts_masks(ws) : nullptr, s);
  if (e == hipSuccess)
    e = laep::launch_counts(topk_idx, T, k, E, counts, offsets, dest_row, row_src, etn_accum, ws,
                            s, /*masks_ready=*/true);
  return hip_status(e, name);
}

}  // namespace

extern "C" {

int moe_route_count(const void* x, const void* w_router, const float* bias, const uint8_t* alive,
                    int dtype, int T, int d_model, int E, int k, int renorm, float* logits,
                    int32_t* topk_idx, float* topk_gate, int32_t* counts, int32_t* offsets,
                    int32_t* dest_row, int32_t* row_src, int64_t* etn_accum, void* ws,
                    size_t ws_bytes, void* stream) {
  int rc = check_route_count("moe_route_count", x, w_router, dtype, T, d_model, E, k, topk_idx,
                             topk_gate, counts, offsets, dest_row);
  if (rc) return rc;
  const size_t need = laep::counts_ws_bytes(T, k, E);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE, "moe_route_count: workspace %zu < %zu bytes",
          ws_bytes, need);
  REQUIRE(need == 0 || ws, LAEP_ERR_INVALID_ARG, "moe_route_count: ws must be non-null");
  return route_count_launch("moe_route_count", x, w_router, bias, alive, dtype, T, d_model, E, k,
                            renorm, logits, topk_idx, topk_gate, counts, offsets, dest_row,
                            row_src, etn_accum, ws, stream);
}

static_assert(laep::kNoAllocScratchBytes == LAEP_NOALLOC_SCRATCH_BYTES,
              "the header states the scratch array's size");

int moe_route_count_noalloc(const void* x, const void* w_router, const float* bias,
                            const uint8_t* alive, int dtype, int T, int d_model, int E, int k,
                            int renorm, float* logits, int32_t* topk_idx, float* topk_gate,
                            int32_t* counts, int32_t* offsets, int32_t* dest_row,
                            int32_t* row_src, int64_t* etn_accum, void* stream) {
  int rc = check_route_count("moe_route_count_noalloc", x, w_router, dtype, T, d_model, E, k,
                             topk_idx, topk_gate, counts, offsets, dest_row);
  if (rc) return rc;
  const size_t need = laep::counts_ws_bytes(T, k, E);
  REQUIRE(need <= laep::kNoAllocScratchBytes, LAEP_ERR_WORKSPACE,
          "moe_route_count_noalloc: T=%d, E=%d need %zu bytes of scratch, more than the "
          "library's %zu-byte array (use moe_route_count with a workspace)",
          T, E, need, laep::kNoAllocScratchBytes);
  void* ws = nullptr;
  if (need > 0) {
    const hipError_t e = laep::noalloc_scratch(&ws);
    if (e != hipSuccess) return hip_status(e, "moe_route_count_noalloc: scratch lookup");
  }
  return route_count_launch("moe_route_count_noalloc", x, w_router, bias, alive, dtype, T,
                            d_model, E, k, renorm, logits, topk_idx, topk_gate, counts, offsets,
                            dest_row, row_src, etn_accum, ws, stream);
}

int laep_prune_mask(const int32_t* counts, int E, int64_t total, double alpha, double beta,
                    uint8_t* alive, int32_t* n_pruned, void* stream) {
  REQUIRE(E >= 1 && E <= LAEP_MAX_EXPERTS, LAEP_ERR_INVALID_ARG, "E=%d outside [1, %d]", E,
          LAEP_MAX_EXPERTS);
  REQUIRE(counts && alive && n_pruned, LAEP_ERR_INVALID_ARG,
          "laep_prune_mask: counts, alive and n_pruned must be non-null");
  REQUIRE(total >= 0, LAEP_ERR_INVALID_ARG, "laep_prune_mask: total=%lld < 0", (long long)total);
  REQUIRE(!std::isnan(alpha) && !std::isnan(beta) && alpha >= 0 && beta >= 0,
          LAEP_ERR_INVALID_ARG, "laep_prune_mask: alpha and beta must be >= 0 (got %g, %g)",
          alpha, beta);
  return hip_status(
      laep::launch_prune(counts, E, total, alpha, beta, alive, n_pruned, as_stream(stream)),
      "laep_prune_mask");
}

int laep_expert_pruning(const int64_t* etn, int ITER, int L, int E, int64_t total,
                        const double* alpha, double beta, uint8_t* alive, int32_t* n_pruned,
                        int32_t* marker, void* stream) {
  REQUIRE(E >= 1 && E <= LAEP_MAX_EXPERTS, LAEP_ERR_INVALID_ARG, "E=%d outside [1, %d]", E,
          LAEP_MAX_EXPERTS);
  REQUIRE(L >= 1 && L <= LAEP_MAX_LAYERS, LAEP_ERR_INVALID_ARG, "L=%d outside [1, %d]", L,
          LAEP_MAX_LAYERS);
  REQUIRE(ITER >= 1, LAEP_ERR_INVALID_ARG, "laep_expert_pruning: ITER=%d < 1", ITER);
  REQUIRE(etn && alpha && alive && n_pruned, LAEP_ERR_INVALID_ARG,
          "laep_expert_pruning: etn, alpha, alive and n_pruned must be non-null");
  REQUIRE(total >= 0, LAEP_ERR_INVALID_ARG, "laep_expert_pruning: total=%lld < 0",
          (long long)total);
  REQUIRE(!std::isnan(beta) && beta >= 0, LAEP_ERR_INVALID_ARG,
          "laep_expert_pruning: beta must be >= 0 (got %g)", beta);
  for (int l = 0; l < L; ++l)
    REQUIRE(!std::isnan(alpha[l]) && alpha[l] >= 0, LAEP_ERR_INVALID_ARG,
            "laep_expert_pruning: alpha[%d] must be >= 0 (got %g)", l, alpha[l]);
  return hip_status(laep::launch_expert_pruning(etn, ITER, L, E, total, alpha, beta, alive,
                                                n_pruned, marker, as_stream(stream)),
                    "laep_expert_pruning");
}

int laep_compact_experts(const uint8_t* alive, int L, int E, int32_t* expert_map,
                         int32_t* n_alive, void* stream) {
  REQUIRE(E >= 1 && E <= LAEP_MAX_EXPERTS, LAEP_ERR_INVALID_ARG, "E=%d outside [1, %d]", E,
          LAEP_MAX_EXPERTS);
  REQUIRE(L >= 1, LAEP_ERR_INVALID_ARG, "laep_compact_experts: L=%d < 1", L);
  REQUIRE(alive && expert_map && n_alive, LAEP_ERR_INVALID_ARG,
          "laep_compact_experts: alive, expert_map and n_alive must be non-null");
  return hip_status(laep::launch_expert_map(alive, L, E, expert_map, n_alive, as_stream(stream)),
                    "laep_compact_experts");
}

int laep_repack_experts(const int32_t* expert_map, int E, int n_out, int dtype, int d_model,
                        int d_ff, const void* w_router, const float* bias, const void* w_gate_up,
                        const void* w_down, void* w_router_out, float* bias_out,
                        void* w_gate_up_out, void* w_down_out, void* stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  REQUIRE(E >= 1 && E <= LAEP_MAX_EXPERTS, LAEP_ERR_INVALID_ARG, "E=%d outside [1, %d]", E,
          LAEP_MAX_EXPERTS);
  REQUIRE(n_out >= 0, LAEP_ERR_INVALID_ARG, "laep_repack_experts: n_out=%d < 0", n_out);
  REQUIRE(expert_map, LAEP_ERR_INVALID_ARG, "laep_repack_experts: expert_map must be non-null");
  REQUIRE(d_model > 0 && d_model % 8 == 0, LAEP_ERR_INVALID_ARG,
          "laep_repack_experts: d_model=%d must be a positive multiple of 8", d_model);
  REQUIRE(!!w_router == !!w_router_out && !!bias == !!bias_out &&
              !!w_gate_up == !!w_gate_up_out && !!w_down == !!w_down_out,
          LAEP_ERR_INVALID_ARG,
          "laep_repack_experts: each source and its destination must be both set or both NULL");
  REQUIRE(!(w_gate_up || w_down) || d_ff > 0, LAEP_ERR_INVALID_ARG,
          "laep_repack_experts: d_ff=%d must be positive", d_ff);
  const void* ptrs[] = {w_router, w_router_out, w_gate_up, w_gate_up_out, w_down, w_down_out};
  for (const void* q : ptrs)
    REQUIRE(aligned16(q), LAEP_ERR_INVALID_ARG,
            "laep_repack_experts: weight pointers must be 16-byte aligned");
  if (n_out == 0) return ok();
  const size_t es = elem_bytes(dtype);
  const hipStream_t s = as_stream(stream);
  hipError_t e = hipSuccess;
  if (w_router)
    e = laep::launch_repack(expert_map, E, n_out, w_router, w_router_out, d_model * es, s);
  if (e == hipSuccess && bias)
    e = laep::launch_repack_scalar(expert_map, E, n_out, bias, bias_out, s);
  if (e == hipSuccess && w_gate_up)
    e = laep::launch_repack(expert_map, E, n_out, w_gate_up, w_gate_up_out,
                            (size_t)2 * d_ff * d_model * es, s);
  if (e == hipSuccess && w_down)
    e = laep::launch_repack(expert_map, E, n_out, w_down, w_down_out,
                            (size_t)d_model * d_ff * es, s);
  return hip_status(e, "laep_repack_experts");
}

int moe_route_bwd(const float* dgate, const int32_t* topk_idx, const float* topk_gate,
                  const float* logits, const uint8_t* alive, const void* x, const void* w_router,
                  const int32_t* offsets, const int32_t* row_src, int dtype, int T, int d_model,
                  int E, int k, int renorm, float* dlogits, float* dw_router, float* dbias,
                  void* dx, int accumulate_dx, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  if ((rc = check_experts(E, k))) return rc;
  if ((rc = check_rows(T, k, d_model))) return rc;
  REQUIRE(w_router, LAEP_ERR_INVALID_ARG, "moe_route_bwd: w_router must be non-null");
  REQUIRE(dw_router || !dbias, LAEP_ERR_INVALID_ARG,
          "moe_route_bwd: dbias needs dw_router (they are computed together)");
  REQUIRE(aligned16(w_router) && aligned16(dw_router), LAEP_ERR_INVALID_ARG,
          "moe_route_bwd: w_router and dw_router must be 16-byte aligned");
  if (T > 0) {
    REQUIRE(dgate && topk_idx && topk_gate && x && ws, LAEP_ERR_INVALID_ARG,
            "moe_route_bwd: dgate, topk_idx, topk_gate, x and ws must be non-null");
    REQUIRE(aligned16(x) && aligned16(dx), LAEP_ERR_INVALID_ARG,
            "moe_route_bwd: x and dx must be 16-byte aligned");
    if (renorm)
      REQUIRE(offsets && row_src, LAEP_ERR_INVALID_ARG,
              "moe_route_bwd: renorm = 1 needs offsets and row_src from moe_expert_counts");
    else
      REQUIRE(logits, LAEP_ERR_INVALID_ARG, "moe_route_bwd: renorm = 0 needs the logits");
    const size_t need = laep::route_bwd_ws_bytes(T, k, E, d_model);
    REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE, "moe_route_bwd: workspace %zu < %zu bytes",
            ws_bytes, need);
  }
  return hip_status(laep::launch_route_bwd(dgate, topk_idx, topk_gate, logits, alive, x, w_router,
                                           offsets, row_src, dtype, T, d_model, E, k, renorm,
                                           dlogits, dw_router, dbias, dx, accumulate_dx, ws,
                                           as_stream(stream)),
                    "moe_route_bwd");
}

int moe_permute(const void* x, int dtype, const int32_t* dest_row, int T, int k, int d_model,
                void* x_perm, void* stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  REQUIRE(k >= 1, LAEP_ERR_INVALID_ARG, "k=%d < 1", k);
  if ((rc = check_rows(T, k, d_model))) return rc;
  if (T == 0) return ok();
  REQUIRE(x && dest_row && x_perm, LAEP_ERR_INVALID_ARG,
          "moe_permute: x, dest_row and x_perm must be non-null");
  REQUIRE(aligned16(x) && aligned16(x_perm), LAEP_ERR_INVALID_ARG,
          "moe_permute: x and x_perm must be 16-byte aligned");
  return hip_status(laep::launch_permute(x, (int)elem_bytes(dtype), dest_row, T, k, d_model,
                                         x_perm, as_stream(stream)),
                    "moe_permute");
}

int moe_grouped_ffn_fwd(const void* x_perm, const void* w_gate_up, const void* w_down,
                        const int32_t* offsets, const int32_t* expert_map, int dtype, int E,
                        int d_model, int d_ff, int64_t R, void* y_perm, void* act_save, void* ws,
                        size_t ws_bytes, void* stream) {
  int rc = check_ffn_shape(dtype, E, d_model, d_ff, R);
  if (rc) return rc;
  REQUIRE(offsets, LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_fwd: offsets must be non-null");
  if (R == 0) return ok();
  REQUIRE(x_perm && w_gate_up && w_down && y_perm && ws, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd: x_perm, w_gate_up, w_down, y_perm and ws must be non-null");
  REQUIRE(aligned16(x_perm) && aligned16(w_gate_up) && aligned16(w_down) && aligned16(y_perm) &&
              aligned16(act_save) && aligned16(ws),
          LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_fwd: buffers must be 16-byte aligned");
  const size_t need = laep::ffn_fwd_ws_bytes(R, E, d_model, d_ff, dtype);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE, "moe_grouped_ffn_fwd: workspace %zu < %zu bytes",
          ws_bytes, need);
  hipError_t e =
      dtype == LAEP_BF16
          ? laep::launch_ffn_fwd_bf16(x_perm, w_gate_up, w_down, offsets, expert_map, E, d_model,
                                      d_ff, R, y_perm, act_save, ws, as_stream(stream))
          : laep::launch_ffn_fwd_f32(x_perm, w_gate_up, w_down, offsets, expert_map, E, d_model,
                                     d_ff, R, y_perm, act_save, ws, as_stream(stream));
  return hip_status(e, "moe_grouped_ffn_fwd");
}

int moe_grouped_ffn_fwd_gather(const void* x, const int32_t* row_src, int T, int k,
                               const void* w_gate_up, const void* w_down, const int32_t* offsets,
                               const int32_t* expert_map, int dtype, int E, int d_model, int d_ff,
                               int64_t R, void* y_perm, void* act_save, void* x_perm_out,
                               void* ws, size_t ws_bytes, void* stream) {
  int rc = check_ffn_shape(dtype, E, d_model, d_ff, R);
  if (rc) return rc;
  REQUIRE(dtype == LAEP_BF16, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_fwd_gather: only LAEP_BF16 is supported");
  REQUIRE(T >= 0 && k >= 1, LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_fwd_gather: T=%d, k=%d", T, k);
  REQUIRE(R <= (int64_t)T * k, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather: R=%lld exceeds T*k", (long long)R);
  REQUIRE((int64_t)T * d_model * 2 < kMaxBufferBytes, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_fwd_gather: x (T*d_model bf16) must be under 2 GiB");
  REQUIRE(offsets, LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_fwd_gather: offsets must be non-null");
  if (R == 0) return ok();
  REQUIRE(x && row_src && w_gate_up && w_down && y_perm && ws, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather: x, row_src, w_gate_up, w_down, y_perm and ws must be "
          "non-null");
  REQUIRE(aligned16(x) && aligned16(w_gate_up) && aligned16(w_down) && aligned16(y_perm) &&
              aligned16(act_save) && aligned16(x_perm_out) && aligned16(ws),
          LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_fwd_gather: buffers must be 16-byte aligned");
  REQUIRE(x_perm_out != x && x_perm_out != y_perm, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather: x_perm_out must not alias x or y_perm");
  const size_t need = laep::ffn_fwd_ws_bytes(R, E, d_model, d_ff, dtype);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE,
          "moe_grouped_ffn_fwd_gather: workspace %zu < %zu bytes", ws_bytes, need);
  return hip_status(laep::launch_ffn_fwd_bf16(x, w_gate_up, w_down, offsets, expert_map, E,
                                              d_model, d_ff, R, y_perm, act_save, ws,
                                              as_stream(stream), row_src, k, nullptr, nullptr,
                                              x_perm_out),
                    "moe_grouped_ffn_fwd_gather");
}

int moe_grouped_ffn_fwd_gather_combine(const void* x, const int32_t* row_src, int T, int k,
                                       const void* w_gate_up, const void* w_down,
                                       const int32_t* offsets, const int32_t* expert_map,
                                       const float* topk_gate, int dtype, int E, int d_model,
                                       int d_ff, int64_t R, void* out, void* y_perm,
                                       void* act_save, void* x_perm_out, void* ws,
                                       size_t ws_bytes, void* stream) {
  int rc = check_ffn_shape(dtype, E, d_model, d_ff, R);
  if (rc) return rc;
  REQUIRE(dtype == LAEP_BF16, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_fwd_gather_combine: only LAEP_BF16 is supported");
  REQUIRE(k == 1, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_fwd_gather_combine: k=%d, only one slot per token is supported", k);
  REQUIRE(T >= 0, LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_fwd_gather_combine: T=%d < 0", T);
  REQUIRE(R <= (int64_t)T, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather_combine: R=%lld exceeds T", (long long)R);
  REQUIRE((int64_t)T * d_model * 2 < kMaxBufferBytes, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_fwd_gather_combine: x and out (T*d_model bf16) must be under 2 GiB");
  REQUIRE(offsets, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather_combine: offsets must be non-null");
  if (R == 0) return ok();
  REQUIRE(x && row_src && w_gate_up && w_down && topk_gate && out && ws, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather_combine: x, row_src, w_gate_up, w_down, topk_gate, out "
          "and ws must be non-null");
  REQUIRE(aligned16(x) && aligned16(w_gate_up) && aligned16(w_down) && aligned16(out) &&
              aligned16(y_perm) && aligned16(act_save) && aligned16(x_perm_out) && aligned16(ws),
          LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather_combine: buffers must be 16-byte aligned");
  REQUIRE(out != y_perm && out != x && out != x_perm_out, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather_combine: out must not alias x, y_perm or x_perm_out");
  REQUIRE(x_perm_out == nullptr || (x_perm_out != x && x_perm_out != y_perm),
          LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_fwd_gather_combine: x_perm_out must not alias x or y_perm");
  const size_t need = laep::ffn_fwd_ws_bytes(R, E, d_model, d_ff, dtype);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE,
          "moe_grouped_ffn_fwd_gather_combine: workspace %zu < %zu bytes", ws_bytes, need);
  return hip_status(laep::launch_ffn_fwd_bf16(x, w_gate_up, w_down, offsets, expert_map, E,
                                              d_model, d_ff, R, y_perm, act_save, ws,
                                              as_stream(stream), row_src, k, topk_gate, out,
                                              x_perm_out),
                    "moe_grouped_ffn_fwd_gather_combine");
}

int moe_grouped_ffn_bwd(const void* dy_perm, const void* x_perm, const void* act_save,
                        const void* h_fwd, const void* w_gate_up, const void* w_down,
                        const int32_t* offsets,
                        const int32_t* expert_map, int dtype, int E, int d_model, int d_ff,
                        int64_t R, void* dx_perm, float* dw_gate_up, float* dw_down,
                        int accumulate, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_ffn_shape(dtype, E, d_model, d_ff, R);
  if (rc) return rc;
  REQUIRE(dtype == LAEP_BF16, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_bwd: only LAEP_BF16 is supported");
  REQUIRE(offsets && dw_gate_up && dw_down && ws, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_bwd: offsets, dw_gate_up, dw_down and ws must be non-null");
  REQUIRE(R == 0 || (dy_perm && x_perm && act_save && w_gate_up && w_down && dx_perm),
          LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_bwd: activation pointers must be non-null");
  REQUIRE(aligned16(dy_perm) && aligned16(x_perm) && aligned16(act_save) && aligned16(h_fwd) &&
              aligned16(w_gate_up) && aligned16(w_down) && aligned16(dx_perm) &&
              aligned16(dw_gate_up) && aligned16(dw_down) && aligned16(ws),
          LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_bwd: buffers must be 16-byte aligned");
  const size_t need = laep::ffn_bwd_ws_bytes(R, E, d_model, d_ff, dtype);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE, "moe_grouped_ffn_bwd: workspace %zu < %zu bytes",
          ws_bytes, need);
  return hip_status(laep::launch_ffn_bwd_bf16(dy_perm, x_perm, act_save, h_fwd, w_gate_up, w_down,
                                              offsets, expert_map, E, d_model, d_ff, R, dx_perm,
                                              dw_gate_up, dw_down, accumulate != 0, ws,
                                              as_stream(stream)),
                    "moe_grouped_ffn_bwd");
}

int moe_grouped_ffn_bwd_gather(const void* dy_perm, const void* dout, const float* topk_gate,
                               const void* x, const int32_t* row_src, int T,
                               int k, const void* act_save, const void* h_fwd,
                               const void* w_gate_up, const void* w_down, const int32_t* offsets,
                               const int32_t* expert_map, int dtype, int E, int d_model, int d_ff,
                               int64_t R, void* dx_perm, float* dw_gate_up, float* dw_down,
                               int accumulate, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_ffn_shape(dtype, E, d_model, d_ff, R);
  if (rc) return rc;
  REQUIRE(dtype == LAEP_BF16, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_bwd_gather: only LAEP_BF16 is supported");
  REQUIRE(T >= 0 && k >= 1, LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_bwd_gather: T=%d, k=%d", T, k);
  REQUIRE(R <= (int64_t)T * k, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_bwd_gather: R=%lld exceeds T*k", (long long)R);
  REQUIRE((int64_t)T * d_model * 2 < kMaxBufferBytes, LAEP_ERR_UNSUPPORTED,
          "moe_grouped_ffn_bwd_gather: x (T*d_model bf16) must be under 2 GiB");
  REQUIRE(offsets && dw_gate_up && dw_down && ws, LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_bwd_gather: offsets, dw_gate_up, dw_down and ws must be non-null");
  REQUIRE(R == 0 || (x && row_src && act_save && w_gate_up && w_down && dx_perm),
          LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_bwd_gather: activation pointers and row_src must be non-null");
  REQUIRE(R == 0 || dy_perm || (dout && topk_gate), LAEP_ERR_INVALID_ARG,
          "moe_grouped_ffn_bwd_gather: without dy_perm, dout and topk_gate must be non-null");
  REQUIRE(aligned16(dy_perm) && aligned16(dout) && aligned16(x) && aligned16(act_save) &&
              aligned16(h_fwd) &&
              aligned16(w_gate_up) && aligned16(w_down) && aligned16(dx_perm) &&
              aligned16(dw_gate_up) && aligned16(dw_down) && aligned16(ws),
          LAEP_ERR_INVALID_ARG, "moe_grouped_ffn_bwd_gather: buffers must be 16-byte aligned");
  const size_t need = laep::ffn_bwd_ws_bytes(R, E, d_model, d_ff, dtype);
  REQUIRE(ws_bytes >= need, LAEP_ERR_WORKSPACE,
          "moe_grouped_ffn_bwd_gather: workspace %zu < %zu bytes", ws_bytes, need);
  return hip_status(laep::launch_ffn_bwd_bf16(dy_perm, x, act_save, h_fwd, w_gate_up, w_down,
                                              offsets, expert_map, E, d_model, d_ff, R, dx_perm,
                                              dw_gate_up, dw_down, accumulate != 0, ws,
                                              as_stream(stream), row_src, k, T, dout, topk_gate),
                    "moe_grouped_ffn_bwd_gather");
}

int moe_combine(const void* y_perm, const float* topk_gate, const int32_t* dest_row, int T, int k,
                int d_model, int dtype, void* out, void* stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  REQUIRE(k >= 1, LAEP_ERR_INVALID_ARG, "k=%d < 1", k);
  if ((rc = check_rows(T, k, d_model))) return rc;
  if (T == 0) return ok();
  REQUIRE(y_perm && topk_gate && dest_row && out, LAEP_ERR_INVALID_ARG,
          "moe_combine: y_perm, topk_gate, dest_row and out must be non-null");
  REQUIRE(aligned16(y_perm) && aligned16(out), LAEP_ERR_INVALID_ARG,
          "moe_combine: y_perm and out must be 16-byte aligned");
  return hip_status(laep::launch_combine(y_perm, topk_gate, dest_row, T, k, d_model, dtype, out,
                                         as_stream(stream)),
                    "moe_combine");
}

int moe_combine_bwd(const void* dout, const void* y_perm, const float* topk_gate,
                    const int32_t* dest_row, int T, int k, int d_model, int dtype, void* dy_perm,
                    float* dgate, void* stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  REQUIRE(k >= 1, LAEP_ERR_INVALID_ARG, "k=%d < 1", k);
  if ((rc = check_rows(T, k, d_model))) return rc;
  if (T == 0) return ok();
  REQUIRE(dout && y_perm && topk_gate && dest_row && dgate, LAEP_ERR_INVALID_ARG,
          "moe_combine_bwd: pointers other than dy_perm must be non-null");
  REQUIRE(aligned16(dout) && aligned16(y_perm) && aligned16(dy_perm), LAEP_ERR_INVALID_ARG,
          "moe_combine_bwd: dout, y_perm and dy_perm must be 16-byte aligned");
  return hip_status(laep::launch_combine_bwd(dout, y_perm, topk_gate, dest_row, T, k, d_model,
                                             dtype, dy_perm, dgate, as_stream(stream)),
                    "moe_combine_bwd");
}

int moe_permute_bwd(const void* dx_perm, const int32_t* dest_row, int T, int k, int d_model,
                    int dtype, void* dx, void* stream) {
  int rc = check_dtype(dtype);
  if (rc) return rc;
  REQUIRE(k >= 1, LAEP_ERR_INVALID_ARG, "k=%d < 1", k);
  if ((rc = check_rows(T, k, d_model))) return rc;
  if (T == 0) return ok();
  REQUIRE(dx_perm && dest_row && dx, LAEP_ERR_INVALID_ARG,
          "moe_permute_bwd: dx_perm, dest_row and dx must be non-null");
  REQUIRE(aligned16(dx_perm) && aligned16(dx), LAEP_ERR_INVALID_ARG,
          "moe_permute_bwd: dx_perm and dx must be 16-byte aligned");
  return hip_status(laep::launch_combine(dx_perm, nullptr, dest_row, T, k, d_model, dtype, dx,
                                         as_stream(stream)),
                    "moe_permute_bwd");
}

// ---- measurement kernels (laep_calib.h) ------------------------------------------
int laep_calib_copy(const void* src, void* dst, size_t bytes, void* stream) {
  REQUIRE(src && dst && aligned16(src) && aligned16(dst) && bytes % 16 == 0,
          LAEP_ERR_INVALID_ARG, "laep_calib_copy: null or misaligned pointer, or bytes %% 16 != 0");
  return hip_status(laep::launch_calib_copy(src, dst, bytes, as_stream(stream)), "laep_calib_copy");
}

int laep_calib_read(const void* src, size_t bytes, int block_bytes, float* out, void* stream) {
  REQUIRE(src && out && aligned16(src), LAEP_ERR_INVALID_ARG,
          "laep_calib_read: null or misaligned pointer");
  REQUIRE(block_bytes >= 8192 && block_bytes <= 131072 && block_bytes % 8192 == 0 &&
              bytes % (size_t)block_bytes == 0 && bytes / (size_t)block_bytes <= 0x7FFFFFFFu,
          LAEP_ERR_INVALID_ARG,
          "laep_calib_read: block_bytes must be a multiple of 8192 in [8192, 131072] that divides "
          "bytes");
  return hip_status(laep::launch_calib_read(src, bytes, block_bytes, out, as_stream(stream)),
                    "laep_calib_read");
}

int laep_calib_mfma(int n_workgroups, int iters, float* out, void* stream) {
  REQUIRE(out && n_workgroups >= 1 && iters >= 1, LAEP_ERR_INVALID_ARG,
          "laep_calib_mfma: null out, n_workgroups < 1 or iters < 1");
  return hip_status(laep::launch_calib_mfma(n_workgroups, iters, out, as_stream(stream)),
                    "laep_calib_mfma");
}

}  // extern "C"
