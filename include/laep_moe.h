/*
 * laep_moe.h -- C ABI of one mixture-of-experts layer on one MI355X (gfx950),
 * the data-parallel hot path that Layer-Adaptive Expert Pruning (LAEP) acts on.
 *
 * The paper (arXiv 2601.14327) states the problem in these terms
 * (Section 3.2): E[i, j, l] = 1 iff token j of layer l is routed to expert i;
 * the load of expert i is sum_j E[i, j, l]; experts are pruned by an
 * individual-load threshold alpha (Eq. (1)) and a cumulative-load threshold
 * beta (Eq. (2)), as carried out by Algorithm 1 (Appendix); surviving
 * experts are placed on devices by Algorithm 2 (Section 3.3, Appendix).
 * The router, the gating function and the expert FFN are not spelled out in
 * the paper; this library implements a linear router, top-k softmax gating
 * and a SwiGLU expert FFN (three d x f matrices per expert, as the paper's
 * parameter counts imply).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Pointers marked "device" are HIP device (HBM) addresses; "host" ones are
 *    ordinary CPU memory.  The caller owns and allocates every buffer; the
 *    library allocates no device memory.  Scratch memory comes in through
 *    `ws` / `ws_bytes`, sized by moe_workspace_bytes(); its contents need no
 *    initialisation, and calls that may run concurrently (on different
 *    streams) need workspaces of their own.
 *  - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *    Every device call only enqueues work on `stream`: no host/device copy,
 *    no synchronisation.  Inputs must stay valid until that work completes.
 *  - `dtype` is LAEP_F32 or LAEP_BF16 and applies to activations and expert
 *    weights (x, w_router, w_gate_up, w_down, x_perm, y_perm, act_save, out
 *    and their gradients).  Router logits, gates, gate gradients and weight
 *    gradients are always float32.  Layouts are row-major; weight matrices
 *    are stored [out_features, in_features] (w_gate_up[e] stacks the gate
 *    rows [0, d_ff) over the up rows [d_ff, 2*d_ff)).
 *  - Activation and weight pointers must be 16-byte aligned.
 *  - Return value: LAEP_OK or an error code.  Arguments are validated on the
 *    host before any HIP call; an invalid call enqueues nothing.  The message
 *    of the last error of the calling thread is laep_last_error().
 *    A fault inside a kernel surfaces at the caller's next synchronisation.
 *  - Results are deterministic: identical inputs give identical bits (no
 *    floating-point atomics anywhere).
 *  - Calls are thread-safe; the only library state is the per-thread error
 *    message.
 */
#ifndef LAEP_MOE_H
#define LAEP_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* dtypes */
#define LAEP_F32 0
#define LAEP_BF16 1

/* return codes */
#define LAEP_OK 0
#define LAEP_ERR_INVALID_ARG 1 /* null pointer, bad size, misaligned pointer */
#define LAEP_ERR_UNSUPPORTED 2 /* dtype or shape the library does not handle */
#define LAEP_ERR_WORKSPACE 3   /* ws_bytes smaller than moe_workspace_bytes() */
#define LAEP_ERR_HIP 4         /* a HIP launch reported an error              */
#define LAEP_ERR_INFEASIBLE 5  /* the request cannot be met (e.g. capacity)   */

/* `which_call` of moe_workspace_bytes() */
#define LAEP_CALL_ROUTE 0
#define LAEP_CALL_COUNTS 1
#define LAEP_CALL_FFN_FWD 2
#define LAEP_CALL_FFN_BWD 3
#define LAEP_CALL_ROUTE_BWD 4

/* Limits of the library. */
#define LAEP_MAX_EXPERTS 256
#define LAEP_MAX_LAYERS 256

/*
 * moe_route -- router scoring and top-k gating (produces E[i, j, l] of
 * Section 3.2 in compact form: the k expert ids of each token).
 *
 *   logits[t, e] = sum_c x[t, c] * w_router[e, c] (+ bias[e])   (fp32 accumulation)
 *   dead experts (alive[e] == 0) are excluded;
 *   topk_idx[t, 0..k-1] = the k largest logits, descending, ties to the
 *                         lower expert index;
 *   topk_gate[t, j] = renorm ? softmax over the k selected logits
 *                            : softmax over all alive experts, at the k selected.
 *
 *   x        device [T, d_model] dtype        w_router device [E, d_model] dtype
 *   bias     device [E] fp32 or NULL          alive    device [E] uint8 or NULL (all alive)
 *   logits   device [T, E] fp32 or NULL (written when non-NULL; dead experts -inf)
 *   topk_idx device [T, k] int32              topk_gate device [T, k] fp32
 *   Constraints: 1 <= E <= 256, 1 <= k <= E, d_model % 8 == 0, T >= 0.
 *   If fewer than k experts are alive, every alive expert is selected and the
 *   remaining slots get topk_idx = -1 and topk_gate = 0 (such slots are not
 *   routed by the calls below).
 *   Workspace: none (ws may be NULL).
 */
int moe_route(const void* x, const void* w_router, const float* bias,
              const uint8_t* alive, int dtype, int T, int d_model, int E, int k,
              int renorm, float* logits, int32_t* topk_idx, float* topk_gate,
              void* ws, size_t ws_bytes, void* stream);

/*
 * moe_expert_counts -- per-expert token load (the left-hand side of Eq. (1);
 * ETN of Algorithm 1, Step 1, for one iteration and one layer), the expert
 * offsets and the stable dispatch permutation.
 *
 *   counts[e]   = #{(t, j) : topk_idx[t, j] == e}
 *   offsets     = exclusive prefix sum of counts, offsets[E] = routed rows
 *   dest_row[t*k + j] = offsets[e] + #{(t', j') : topk_idx[t', j'] == e, t' < t}
 *                 (rows grouped by expert, ordered by token); -1 for slots
 *                 with topk_idx == -1
 *   row_src[dest_row[s]] = s   (inverse map; optional)
 *   etn_accum[e] += counts[e]  (optional int64 running ETN row)
 *
 *   topk_idx device [T, k] int32, values in [0, E) or -1; the ids of one
 *   token are distinct (as moe_route writes them; a repeated id within a token
 *   is counted once and its slots share one row)
 *   counts device [E] int32, offsets device [E + 1] int32,
 *   dest_row device [T * k] int32, row_src device [T * k] int32 or NULL,
 *   etn_accum device [E] int64 or NULL.
 *   Workspace: moe_workspace_bytes(LAEP_CALL_COUNTS, T, k, E, 0, 0).
 */
int moe_expert_counts(const int32_t* topk_idx, int T, int k, int E,
                      int32_t* counts, int32_t* offsets, int32_t* dest_row,
                      int32_t* row_src, int64_t* etn_accum, void* ws,
                      size_t ws_bytes, void* stream);

/*
 * moe_route_count -- moe_route and moe_expert_counts in one call: the router
 * kernel also records, per 64-token tile and expert, which tokens chose the
 * expert, so the counting pass starts at its scan (one kernel and one read
 * of topk_idx fewer).  Outputs are bit-identical to moe_route followed by
 * moe_expert_counts on the same arguments.
 *
 *   Arguments as in moe_route (x .. topk_gate) and moe_expert_counts
 *   (counts .. etn_accum).  Workspace: moe_workspace_bytes(LAEP_CALL_COUNTS,
 *   T, k, E, 0, 0), the counting workspace.
 */
int moe_route_count(const void* x, const void* w_router, const float* bias,
                    const uint8_t* alive, int dtype, int T, int d_model, int E,
                    int k, int renorm, float* logits, int32_t* topk_idx,
                    float* topk_gate, int32_t* counts, int32_t* offsets,
                    int32_t* dest_row, int32_t* row_src, int64_t* etn_accum,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * moe_route_count_noalloc -- moe_route_count for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, minus the workspace; outputs are
 * bit-identical to moe_route_count's (the same kernels).
 *
 *   The counting scratch (moe_workspace_bytes(LAEP_CALL_COUNTS, T, k, E, 0, 0)
 *   bytes) lives in a library-owned device array of
 *   LAEP_NOALLOC_SCRATCH_BYTES bytes per GPU, held until the process ends.
 *   The call makes no allocation of any kind (its first call on a device
 *   only looks the array's address up).  The scratch is fully written before
 *   it is read, so stale contents from an earlier call do not matter.
 *   Errors: a shape whose scratch exceeds LAEP_NOALLOC_SCRATCH_BYTES ->
 *   LAEP_ERR_WORKSPACE before anything is enqueued (8 MiB hold the counting
 *   scratch of up to 691840 tokens at E = 64, 172928 at E = 256); otherwise
 *   as moe_route_count.
 *   Concurrency: every call on one GPU shares that GPU's array.  Calls that
 *   overlap in time on one GPU (different streams, or different host
 *   threads without ordering) race on it and give undefined results;
 *   serialise them, e.g. on one stream.
 */
#define LAEP_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
int moe_route_count_noalloc(const void* x, const void* w_router,
                            const float* bias, const uint8_t* alive, int dtype,
                            int T, int d_model, int E, int k, int renorm,
                            float* logits, int32_t* topk_idx, float* topk_gate,
                            int32_t* counts, int32_t* offsets,
                            int32_t* dest_row, int32_t* row_src,
                            int64_t* etn_accum, void* stream);

/*
 * laep_prune_mask -- the LAEP prune decision for one layer and one counted
 * batch (Section 3.2, Eqs. (1) and (2); Algorithm 1, Step 2 with ITER = 1).
 *
 *   Experts are ranked by (counts[e], e) ascending.  Walking that order with
 *   an inclusive running sum, an expert is pruned iff
 *       (double)running < (double)total * beta                    (Eq. (2))
 *   and (double)count   < ((double)total * alpha) / (double)E     (Eq. (1))
 *   (strict comparisons, as in Algorithm 1; alpha = INFINITY disables Eq. (1)).
 *   The pruned set is a prefix of that ranking.
 *
 *   counts device [E] int32 (>= 0); total = S * topK (tokens times k);
 *   alive device [E] uint8 (out: 1 = kept, 0 = pruned);
 *   n_pruned device int32 (out).
 *   The rule has no lower bound: it may prune below k survivors.
 */
int laep_prune_mask(const int32_t* counts, int E, int64_t total, double alpha,
                    double beta, uint8_t* alive, int32_t* n_pruned,
                    void* stream);

/*
 * laep_expert_pruning -- Algorithm 1 (Appendix) over a recorded window of
 * ITER training iterations and L layers: which experts each layer prunes.
 *
 *   Step 1 (recording) is the caller's: etn[it, l, :] holds the tokens each
 *   expert of layer l received in iteration it (moe_expert_counts adds them
 *   into an int64 row through etn_accum).
 *   Step 2: for every (it, l), the rule of laep_prune_mask on etn[it, l, :]
 *   with total and the layer's alpha[l] marks experts; Marker[l, e] counts
 *   the iterations that marked e, Exp_dis[l] all marks of the layer.
 *   Step 3: layer l prunes N_l = floor(Exp_dis[l] / ITER + 0.5) experts, the
 *   most marked, ties to the lower window load sum (equivalently the lower
 *   mean load), then to the lower index.
 *
 *   etn device [ITER, L, E] int64 (>= 0); total = S * topK per iteration;
 *   alpha host [L] double (>= 0, INFINITY disables Eq. (1)); a per-layer
 *   schedule such as 0.2 on the first and last sixth of the layers and 0.4
 *   in between (the ablation of Section 3.4, and the setting of the
 *   Section 4 pre-training run) is passed here;
 *   alive device [L, E] uint8 (out: 1 = kept); n_pruned device [L] int32
 *   (out: N_l); marker device [L, E] int32 (out, optional: Marker).
 *   1 <= L <= LAEP_MAX_LAYERS, 1 <= ITER.
 */
int laep_expert_pruning(const int64_t* etn, int ITER, int L, int E,
                        int64_t total, const double* alpha, double beta,
                        uint8_t* alive, int32_t* n_pruned, int32_t* marker,
                        void* stream);

/*
 * laep_compact_experts -- slot assignment for physical expert compaction
 * (Section 3.2: pruned experts leave the model).  Per layer, the surviving
 * experts keep their order and take consecutive slots:
 *   expert_map[l, e] = #{j < e : alive[l, j]} if alive[l, e], else -1
 *   n_alive[l]       = #{e : alive[l, e]}
 *
 *   alive device [L, E] uint8; expert_map device [L, E] int32 (out);
 *   n_alive device [L] int32 (out).  The map is also the expert_map of
 *   moe_grouped_ffn_fwd/bwd over the repacked weights.
 */
int laep_compact_experts(const uint8_t* alive, int L, int E, int32_t* expert_map,
                         int32_t* n_alive, void* stream);

/*
 * laep_repack_experts -- copy the surviving experts' parameters of one layer
 * into compact buffers of n_out slots.  For every e with
 * 0 <= p = expert_map[e] < n_out:
 *   w_router_out[p]  = w_router[e]       ([d_model] row)
 *   bias_out[p]      = bias[e]           (float32)
 *   w_gate_up_out[p] = w_gate_up[e]      ([2*d_ff, d_model])
 *   w_down_out[p]    = w_down[e]         ([d_model, d_ff])
 * Each (source, destination) pair may be NULL together to skip that tensor;
 * optimizer states of the same shapes are repacked by further calls with
 * dtype LAEP_F32.  Slots an expert map does not reach are left untouched.
 *
 *   expert_map device [E] int32 (from laep_compact_experts); the sources are
 *   device [E, ...] dtype, the destinations device [n_out, ...] dtype.
 *   d_model % 8 == 0.  Sources and destinations must not overlap.
 */
int laep_repack_experts(const int32_t* expert_map, int E, int n_out, int dtype,
                        int d_model, int d_ff, const void* w_router,
                        const float* bias, const void* w_gate_up,
                        const void* w_down, void* w_router_out, float* bias_out,
                        void* w_gate_up_out, void* w_down_out, void* stream);

/*
 * moe_route_bwd -- backward of moe_route's scoring and gating, with the
 * top-k selection held fixed (it is piecewise constant in the logits; the
 * paper trains through the router, Section 3.1, and does not define this
 * step further).  From dgate = dLoss/dgate:
 *
 *   renorm = 1 (softmax over the k selected logits), for e = topk_idx[t, j]:
 *     dl[t, e] = g_j * (dg_j - sum_i g_i dg_i),    0 for the other experts
 *   renorm = 0 (softmax over the alive experts, p = that softmax):
 *     dl[t, e] = p_e * (q_e - sum_j g_j dg_j) for alive e, 0 for dead ones,
 *     with q_e = dg_j where e = topk_idx[t, j], 0 elsewhere
 *   dlogits[t, e] = dl[t, e]                         (optional, float32)
 *   dw_router[e] = sum_t dl[t, e] x[t]                (float32, overwritten)
 *   dbias[e]     = sum_t dl[t, e]                     (optional, float32)
 *   dx[t]        = round(dx[t] + sum_e dl[t, e] W_r[e])  (accumulate_dx = 1)
 *                  round(sum_e dl[t, e] W_r[e])            (accumulate_dx = 0)
 *   Slots with topk_idx == -1 carry no gradient.  Sums are fp32 in a fixed
 *   order (deterministic, no atomics).
 *
 *   dgate, topk_gate device [T, k] float32; topk_idx device [T, k] int32
 *   (as moe_route wrote them); x device [T, d_model] dtype; w_router device
 *   [E, d_model] dtype; dx device [T, d_model] dtype.
 *   dx may be NULL (no data gradient) and dw_router may be NULL (no weight
 *   gradients; dbias must then be NULL too), so a training step can take the
 *   weight gradients as soon as dgate exists and dx once the expert path's dx
 *   does (two calls, two workspaces).
 *   renorm = 1 needs offsets [E + 1] and row_src [T * k] from
 *   moe_expert_counts on the same topk_idx (dw_router is summed over each
 *   expert's routed rows in that order); logits and alive may be NULL.
 *   renorm = 0 needs logits [T, E] (moe_route's float32 logits output) and
 *   the alive mask moe_route used (NULL = all alive).
 *   Workspace: moe_workspace_bytes(LAEP_CALL_ROUTE_BWD, T, k, E, d_model, 0).
 *   Two calls in flight at once (the two halves on two streams) need two
 *   workspaces.  T = 0: dw_router and dbias (when given) are zero-filled and
 *   nothing else is touched; the activation pointers may then be NULL.
 */
int moe_route_bwd(const float* dgate, const int32_t* topk_idx,
                  const float* topk_gate, const float* logits,
                  const uint8_t* alive, const void* x, const void* w_router,
                  const int32_t* offsets, const int32_t* row_src, int dtype,
                  int T, int d_model, int E, int k, int renorm, float* dlogits,
                  float* dw_router, float* dbias, void* dx, int accumulate_dx,
                  void* ws, size_t ws_bytes, void* stream);

/*
 * moe_permute -- dispatch (under expert parallelism, Section 3.3, the rows
 * sent to each expert's device): x_perm[dest_row[t*k + j]] = x[t] (a copy;
 * slots with dest_row == -1 are skipped).
 *   x device [T, d_model] dtype; dest_row device [T * k] int32;
 *   x_perm device [rows, d_model] dtype, rows = number of routed slots.
 *   d_model % 8 == 0.
 */
int moe_permute(const void* x, int dtype, const int32_t* dest_row, int T,
                int k, int d_model, void* x_perm, void* stream);

/*
 * moe_grouped_ffn_fwd -- SwiGLU expert FFN over the routed rows, as one
 * grouped GEMM pass over the experts that have rows (pruned experts have
 * none and cost nothing).
 *
 *   for each expert e with rows [offsets[e], offsets[e+1]) and weight slot
 *   p = expert_map ? expert_map[e] : e:
 *     A = X_e W_gu[p]^T                         (fp32 accumulation, [M_e, 2*d_ff])
 *     act_save = A rounded to dtype             (optional, for the backward)
 *     H = round(silu(A[:, :d_ff]) * A[:, d_ff:])
 *     Y_e = round(H W_d[p]^T)                   -> y_perm rows of expert e
 *
 *   x_perm device [R, d_model]; w_gate_up device [E_phys, 2*d_ff, d_model];
 *   w_down device [E_phys, d_model, d_ff]; offsets device [E + 1] int32
 *   (offsets[E] <= R); expert_map device [E] int32 or NULL (identity), -1 =
 *   pruned (such experts must have no rows; the map must not repeat a slot);
 *   y_perm device [R, d_model]; act_save device [R, 2*d_ff] or NULL.
 *   Constraints: d_model % 64 == 0, d_ff % 64 == 0, R < 2^31; bf16: one
 *   expert's w_gate_up under 2 GiB (4*d_ff*d_model bytes), since the GEMMs
 *   address it with 32-bit offsets (LAEP_ERR_UNSUPPORTED otherwise).
 *   LAEP_BF16 runs on the bf16 matrix cores (fp32 accumulation).  LAEP_F32
 *   is a plain fp32 FMA loop (no matrix cores), meant for small parity
 *   layers, not for speed; its backward is not implemented.
 *   Workspace: moe_workspace_bytes(LAEP_CALL_FFN_FWD, R, 1, E, d_model, d_ff)
 *   (holds H, the tile tables and the products' tile counters, which the
 *   call's first kernel resets; on return H [R, d_ff] (dtype) is at byte
 *   offset 0, which moe_grouped_ffn_bwd can take as h_fwd).
 */
int moe_grouped_ffn_fwd(const void* x_perm, const void* w_gate_up,
                        const void* w_down, const int32_t* offsets,
                        const int32_t* expert_map, int dtype, int E,
                        int d_model, int d_ff, int64_t R, void* y_perm,
                        void* act_save, void* ws, size_t ws_bytes,
                        void* stream);

/*
 * moe_grouped_ffn_fwd_gather -- moe_permute followed by moe_grouped_ffn_fwd
 * in one pass: the gate/up product reads each routed row straight from the
 * token rows (x_perm is never written).  Routed row r is token
 * row_src[r] / k, as moe_expert_counts writes row_src (the inverse of
 * dest_row).  Results are bit-identical to the two calls.
 *
 *   x device [T, d_model] bf16; row_src device [R] int32 (every entry in
 *   [0, T*k)); the other arguments and the workspace are those of
 *   moe_grouped_ffn_fwd.  dtype must be LAEP_BF16 and x under 2 GiB
 *   (T*d_model*2 bytes: its rows are addressed with 32-bit offsets);
 *   LAEP_ERR_UNSUPPORTED otherwise.
 *   x_perm_out device [R, d_model] bf16 or NULL: when given, the dispatched
 *   rows (what moe_permute writes) are also written there, for the weight
 *   gradient, by a copy on the library's side stream (see
 *   moe_grouped_ffn_bwd) that runs beside the FFN and is joined back before
 *   the call ends on `stream`.  It must not alias x or y_perm.
 */
int moe_grouped_ffn_fwd_gather(const void* x, const int32_t* row_src, int T,
                               int k, const void* w_gate_up,
                               const void* w_down, const int32_t* offsets,
                               const int32_t* expert_map, int dtype, int E,
                               int d_model, int d_ff, int64_t R,
                               void* y_perm, void* act_save, void* x_perm_out,
                               void* ws, size_t ws_bytes, void* stream);

/*
 * moe_grouped_ffn_fwd_gather_combine -- moe_grouped_ffn_fwd_gather followed
 * by moe_combine, for one slot per token (k = 1: an expert-parallel rank's
 * local rows, Section 3.3, each returned to its sender scaled by its gate).  The down
 * projection's epilogue writes each routed row r straight to its token row:
 *   out[t] = round(topk_gate[t] * y_r)   with t = row_src[r] (k = 1),
 * where y_r is the rounded FFN output row, in the combine's arithmetic, so
 * out is bit-identical to the three calls.  y_perm is written too when
 * non-NULL (the backward's moe_combine_bwd reads it), else never.
 *
 *   topk_gate device [T] fp32; out device [T, d_model] bf16 (must not alias
 *   x, y_perm or x_perm_out); y_perm device [R, d_model] bf16 or NULL; the
 *   other arguments (x_perm_out included) and the workspace are those of
 *   moe_grouped_ffn_fwd_gather.
 *   Rows of out whose token has no routed row (topk_idx == -1, which with
 *   k = 1 happens only when no expert is alive) are not written; moe_combine
 *   would write zeros there.
 *   Errors: k != 1 or dtype != LAEP_BF16 -> LAEP_ERR_UNSUPPORTED.
 */
int moe_grouped_ffn_fwd_gather_combine(const void* x, const int32_t* row_src,
                                       int T, int k, const void* w_gate_up,
                                       const void* w_down, const int32_t* offsets,
                                       const int32_t* expert_map,
                                       const float* topk_gate, int dtype, int E,
                                       int d_model, int d_ff, int64_t R, void* out,
                                       void* y_perm, void* act_save, void* x_perm_out,
                                       void* ws, size_t ws_bytes, void* stream);

/*
 * moe_grouped_ffn_bwd -- backward of moe_grouped_ffn_fwd (data and weight
 * gradients), evaluated at the saved pre-activations act_save (Â):
 *
 *   dH   = dY W_d[p]          (stored in dtype between the two steps)
 *   dA_g = dH * Â_u * s * (1 + Â_g (1 - s)),  s = sigmoid(Â_g)
 *   dA_u = dH * silu(Â_g)                      dA = round([dA_g, dA_u])
 *   H_b  = round(silu(Â_g) * Â_u)
 *   dX   = round(dA W_gu[p])                   -> dx_perm
 *   dW_gu[p] (+)= dA^T X,   dW_d[p] (+)= dY^T H   (fp32; `accumulate` adds)
 *   where H is h_fwd, the H the forward computed and the down projection
 *   consumed (exact), or when h_fwd is NULL H_b recomputed at Â.
 *   Slots p of experts without rows get zero gradient (or keep their value
 *   when accumulating).
 *
 *   dy_perm, x_perm device [R, d_model]; act_save device [R, 2*d_ff];
 *   h_fwd device [R, d_ff] or NULL (moe_grouped_ffn_fwd leaves H in its
 *   workspace at byte offset 0); dx_perm device [R, d_model];
 *   dw_gate_up device fp32 [E_phys, 2*d_ff, d_model];
 *   dw_down device fp32 [E_phys, d_model, d_ff].
 *   Workspace: moe_workspace_bytes(LAEP_CALL_FFN_BWD, R, 1, E, d_model, d_ff).
 *   On return the workspace holds dA [R, 2*d_ff] (dtype) at byte offset 0 and,
 *   at byte offset laep_ws_hb_offset(R, d_ff, dtype), H_b [R, d_ff] (dtype)
 *   when h_fwd is NULL, else dH.
 *   Only LAEP_BF16 is supported (LAEP_F32 -> LAEP_ERR_UNSUPPORTED).
 *   Streams: the weight gradients run on a library-owned side stream of the
 *   current device (a pool of four per device, handed out round robin,
 *   created on first use, default priority, kept until the process ends; so
 *   calls on different caller streams overlap on the GPU), forked
 *   from `stream` (dW_d at the start when h_fwd is given, so it overlaps the
 *   first data gradient; otherwise after the SwiGLU backward) and joined back
 *   with events, so the call is ordered on `stream` as a whole and may be
 *   graph-captured.
 */
int moe_grouped_ffn_bwd(const void* dy_perm, const void* x_perm,
                        const void* act_save, const void* h_fwd,
                        const void* w_gate_up, const void* w_down,
                        const int32_t* offsets, const int32_t* expert_map,
                        int dtype, int E, int d_model, int d_ff, int64_t R,
                        void* dx_perm, float* dw_gate_up, float* dw_down,
                        int accumulate,
                        void* ws, size_t ws_bytes, void* stream);

/*
 * moe_grouped_ffn_bwd_gather -- moe_grouped_ffn_bwd with the expert-parallel
 * dispatch and return (Section 3.3) folded into the products:
 *   - dW_gu = dA^T X reads routed row r of X straight from token row
 *     row_src[r] / k of x, so the dispatched rows x_perm are never needed;
 *   - with dy_perm NULL, the first data gradient and dW_d form dY on load:
 *     routed row r is round(topk_gate[s] * dout[s / k]) with s = row_src[r],
 *     exactly what moe_combine_bwd writes into dy_perm (which it can then
 *     skip: pass it dy_perm NULL).
 * Results are bit-identical to moe_permute, moe_combine_bwd's dy_perm and
 * moe_grouped_ffn_bwd.
 *
 *   dy_perm device [R, d_model] bf16 or NULL; dout device [T, d_model] bf16
 *   and topk_gate device [T * k] fp32 (used when dy_perm is NULL);
 *   x device [T, d_model] bf16; row_src device [R] int32 (as
 *   moe_expert_counts writes it, every entry in [0, T*k)); the other
 *   arguments, the workspace and the streams are those of moe_grouped_ffn_bwd.
 *   dtype must be LAEP_BF16 and x and dout under 2 GiB (T*d_model*2 bytes:
 *   their rows are addressed with 32-bit offsets); LAEP_ERR_UNSUPPORTED
 *   otherwise.
 */
int moe_grouped_ffn_bwd_gather(const void* dy_perm, const void* dout,
                               const float* topk_gate, const void* x,
                               const int32_t* row_src, int T, int k,
                               const void* act_save, const void* h_fwd,
                               const void* w_gate_up, const void* w_down,
                               const int32_t* offsets, const int32_t* expert_map,
                               int dtype, int E, int d_model, int d_ff, int64_t R,
                               void* dx_perm, float* dw_gate_up, float* dw_down,
                               int accumulate, void* ws, size_t ws_bytes,
                               void* stream);

/* Byte offset of H_b inside the moe_grouped_ffn_bwd workspace. */
size_t laep_ws_hb_offset(int64_t R, int d_ff, int dtype);

/*
 * moe_combine -- gate-weighted combine (return path of the dispatch,
 * Section 3.3):
 *   out[t] = round(sum_j topk_gate[t, j] * y_perm[dest_row[t*k + j]])
 *   (fp32 accumulation in slot order; slots with dest_row == -1 skipped).
 *   y_perm device [rows, d_model]; topk_gate device [T, k] fp32;
 *   dest_row device [T * k] int32; out device [T, d_model].
 */
int moe_combine(const void* y_perm, const float* topk_gate,
                const int32_t* dest_row, int T, int k, int d_model, int dtype,
                void* out, void* stream);

/*
 * moe_combine_bwd -- backward of moe_combine:
 *   dgate[t, j]  = <dout[t], y_perm[row]>          (fp32 accumulation)
 *   dy_perm[row] = round(topk_gate[t, j] * dout[t]),  row = dest_row[t*k + j]
 *   dout device [T, d_model]; dy_perm device [rows, d_model] or NULL (then
 *   only dgate: moe_grouped_ffn_bwd_gather can form dY itself); dgate device
 *   [T, k] fp32 (0 for unrouted slots).
 */
int moe_combine_bwd(const void* dout, const void* y_perm,
                    const float* topk_gate, const int32_t* dest_row, int T,
                    int k, int d_model, int dtype, void* dy_perm, float* dgate,
                    void* stream);

/*
 * moe_permute_bwd -- backward of moe_permute:
 *   dx[t] = round(sum_j dx_perm[dest_row[t*k + j]])   (fp32 accumulation)
 */
int moe_permute_bwd(const void* dx_perm, const int32_t* dest_row, int T, int k,
                    int d_model, int dtype, void* dx, void* stream);

/* Workspace bytes a call needs (0 if none).  For the FFN calls pass T = R
 * (routed rows) and k = 1; the LAEP_CALL_FFN_FWD size covers both dtypes. */
size_t moe_workspace_bytes(int which_call, int T, int k, int E, int d_model,
                           int d_ff);

/*
 * laep_rearrange -- host utility: greedy placement of n experts into
 * n_groups device groups that balances their loads (Section 3.3;
 * Algorithm 2).  Experts are visited in descending load order (equal loads
 * by index) and each goes to the group with the smallest running sum that
 * still has room (ties to the lower group index).  Capacity per group is
 * ceil(n / n_groups) (the printed floor cannot place every expert when
 * n_groups does not divide n).
 *
 *   loads host [n]; group_of host [n] (out: group of each expert);
 *   order host [n] (out: the flattened group lists, In_flat);
 *   group_sums host [n_groups] (out: sum of loads per group).
 *   Returns LAEP_ERR_INVALID_ARG for n < 0, n_groups < 1 or null pointers.
 */
int laep_rearrange(const double* loads, int n, int n_groups, int32_t* group_of,
                   int32_t* order, double* group_sums);

/* Message of the calling thread's last error ("" if none). */
const char* laep_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LAEP_MOE_H */
