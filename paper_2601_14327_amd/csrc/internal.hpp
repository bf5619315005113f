// Host-side launch entry points of the kernels (internal to the library).
// Every launcher only enqueues work on `s`; arguments are validated by the
// C-ABI layer before these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

namespace laep {

constexpr int kDtypeF32 = 0;
constexpr int kDtypeBf16 = 1;

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Library-owned side streams of the current device (a pool of kSidePool,
// default priority) with their fork / join events, for work a call runs
// beside the caller's stream.  side_stream_acquire hands out the next pool
// entry round robin, locked: keep `lock` from acquisition through the call's
// join (the entry's events are reused by the next call that takes it).
// Concurrent calls from different caller streams take different entries, so
// their side work runs concurrently on the GPU.
constexpr int kSidePool = 4;
struct SideStream {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
hipError_t side_stream_acquire(SideStream*& out, std::unique_lock<std::mutex>& lock);
// the side stream waits for the work enqueued on s so far
hipError_t side_stream_fork(const SideStream& ss, hipStream_t s);
// s waits for the work enqueued on the side stream so far
hipError_t side_stream_join(const SideStream& ss, hipStream_t s);

hipError_t launch_route(const void* x, const void* w, const float* bias, const uint8_t* alive,
                        int dtype, int T, int d, int E, int k, int renorm, float* logits,
                        int32_t* idx, float* gate, uint32_t* masks32, hipStream_t s);

size_t counts_ws_bytes(int T, int k, int E);
// masks_ready: the router already wrote the expert masks into ws
hipError_t launch_counts(const int32_t* idx, int T, int k, int E, int32_t* counts,
                         int32_t* offsets, int32_t* dest_row, int32_t* row_src, int64_t* etn,
                         void* ws, hipStream_t s, bool masks_ready = false);
// the expert-mask area of the counting workspace (uint64 [ceil(T/64)][E])
uint32_t* counts_masks(void* ws);

// Scratch of the allocation-free route + count call: a static device array of
// this many bytes per GPU (csrc/noalloc.hip).  noalloc_scratch() returns its
// device address on the current device (looked up once per device).
constexpr size_t kNoAllocScratchBytes = size_t(8) << 20;
hipError_t noalloc_scratch(void** out);

hipError_t launch_prune(const int32_t* counts, int E, int64_t total, double alpha, double beta,
                        uint8_t* alive, int32_t* n_pruned, hipStream_t s);
constexpr int kMaxLayers = 256;
// alpha: host [L] (L <= kMaxLayers)
hipError_t launch_expert_pruning(const int64_t* etn, int iters, int L, int E, int64_t total,
                                 const double* alpha, double beta, uint8_t* alive,
                                 int32_t* n_pruned, int32_t* marker, hipStream_t s);
hipError_t launch_expert_map(const uint8_t* alive, int L, int E, int32_t* expert_map,
                             int32_t* n_alive, hipStream_t s);
hipError_t launch_repack(const int32_t* expert_map, int E, int n_out, const void* src, void* dst,
                         size_t bytes_per_expert, hipStream_t s);
hipError_t launch_repack_scalar(const int32_t* expert_map, int E, int n_out, const float* src,
                                float* dst, hipStream_t s);

hipError_t launch_permute(const void* x, int elem_bytes, const int32_t* dest_row, int T, int k,
                          int d, void* x_perm, hipStream_t s);
// x_perm[r] = x[row_src[r] / k] for the R routed rows
hipError_t launch_gather_rows(const void* x, const int32_t* row_src, int k, int64_t R, int d,
                              int elem_bytes, void* x_perm, hipStream_t s);
hipError_t launch_combine(const void* y, const float* gate, const int32_t* dest_row, int T, int k,
                          int d, int dtype, void* out, hipStream_t s);
hipError_t launch_combine_bwd(const void* dout, const void* y, const float* gate,
                              const int32_t* dest_row, int T, int k, int d, int dtype, void* dy,
                              float* dgate, hipStream_t s);

// Grouped SwiGLU FFN.
size_t ffn_fwd_ws_bytes(int64_t R, int E, int d, int f, int dtype);
// row_src != NULL: the gate/up A rows are gathered (row r = x_perm row row_src[r] / slots_k).
// out_tok != NULL (one slot per token): routed row r also goes to out_tok row
// row_src[r] / slots_k, times gate[row_src[r]]; y_perm may then be NULL.
// x_perm_out != NULL (with row_src): the gathered rows are also written there,
// on the side stream, beside the FFN.
hipError_t launch_ffn_fwd_bf16(const void* x_perm, const void* w_gu, const void* w_d,
                               const int32_t* offsets, const int32_t* expert_map, int E, int d,
                               int f, int64_t R, void* y_perm, void* act_save, void* ws,
                               hipStream_t s, const int32_t* row_src = nullptr, int slots_k = 1,
                               const float* gate = nullptr, void* out_tok = nullptr,
                               void* x_perm_out = nullptr);
hipError_t launch_ffn_fwd_f32(const void* x_perm, const void* w_gu, const void* w_d,
                              const int32_t* offsets, const int32_t* expert_map, int E, int d,
                              int f, int64_t R, void* y_perm, void* act_save, void* ws,
                              hipStream_t s);

size_t ffn_bwd_ws_bytes(int64_t R, int E, int d, int f, int dtype);
size_t ffn_bwd_hb_offset(int64_t R, int f, int dtype);
// h_fwd != NULL: dW_d uses the forward's H (and starts beside data-gradient 1);
// else H_b, recomputed at the saved pre-activations.
// row_src != NULL: x_perm is the token rows x [x_rows, d] and the weight
// gradient reads routed row r from token row row_src[r] / slots_k.
// dy == NULL (with row_src): dY is formed on load from dout [x_rows, d] and the
// flat gates [x_rows * slots_k], as round(gate[s] * dout[s / slots_k]).
hipError_t launch_ffn_bwd_bf16(const void* dy, const void* x_perm, const void* act_save,
                               const void* h_fwd, const void* w_gu, const void* w_d,
                               const int32_t* offsets,
                               const int32_t* expert_map, int E, int d, int f, int64_t R,
                               void* dx_perm, float* dw_gu, float* dw_d, int accumulate,
                               void* ws, hipStream_t s, const int32_t* row_src = nullptr,
                               int slots_k = 1, int64_t x_rows = 0, const void* dout = nullptr,
                               const float* gate = nullptr);

// Router backward.
size_t route_bwd_ws_bytes(int T, int k, int E, int d_model);
hipError_t launch_route_bwd(const float* dgate, const int32_t* idx, const float* gate,
                            const float* logits, const uint8_t* alive, const void* x,
                            const void* w_router, const int32_t* offsets, const int32_t* row_src,
                            int dtype, int T, int d, int E, int k, int renorm, float* dlogits,
                            float* dw_router, float* dbias, void* dx, int accumulate_dx, void* ws,
                            hipStream_t s);

// Measurement kernels (laep_calib.h).
hipError_t launch_calib_copy(const void* src, void* dst, size_t bytes, hipStream_t s);
hipError_t launch_calib_mfma(int n_workgroups, int iters, float* out, hipStream_t s);
hipError_t launch_calib_read(const void* src, size_t bytes, int block_bytes, float* out,
                             hipStream_t s);

}  // namespace laep
