/*
 * moe_resident.h - C ABI of the resident-expert MoE layer on MI355X (gfx950).
 *
 * One worker's local training step through a mixture-of-experts layer in which
 * the worker holds only its resident subset S_m of the experts (arxiv
 * 2606.19025, Sec. 3.3 "Experts partitioning" and "Ghost Experts and
 * Skip-Token"; Alg. 2 "Simplified View").  The router is not partitioned: it
 * scores all E experts, the top-k is taken over all of them, and routes whose
 * expert is not resident ("ghost experts") are skipped - they contribute
 * nothing to the output and receive no gradient through an expert path.
 *
 * Conventions shared by every entry point:
 *  - Pointers are DEVICE pointers owned by the caller, unless stated
 *    otherwise.  Tensors are dense, row-major and contiguous.
 *  - dtype is MOE_F32 or MOE_BF16 and applies to activations, expert weights
 *    and router weights.  Logits, gate weights, their gradients, dz and every
 *    weight gradient are always fp32.  bf16 results are rounded to nearest
 *    even; all accumulation is fp32.
 *  - Arguments are validated on the host before anything is launched; a
 *    failed check returns a negative status and launches nothing.  The
 *    message for the last failure of the calling thread is moe_last_error().
 *  - Calls are asynchronous on `stream`: they never allocate, never
 *    synchronise the host, and never read device data back (data-dependent
 *    sizes, such as the number of executed routes, stay on the device).
 *  - The library keeps no state between calls and is reentrant.  Results are
 *    deterministic: the same inputs give the same bits on every call.
 *  - Non-finite inputs give unspecified (but in-bounds) results.
 */
#ifndef MOE_RESIDENT_H
#define MOE_RESIDENT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element types */
enum { MOE_F32 = 0, MOE_BF16 = 1 };

/* gate functions s_i(x) applied to the selected logits z (App. A; App. B.3.2):
 *  MOE_GATE_SOFTMAX_TOPK  softmax over all E experts renormalised over the
 *                         global top-k, i.e. softmax of the k selected logits;
 *                         the k weights of a token sum to 1 BEFORE masking and
 *                         are never renormalised over the surviving resident
 *                         routes (App. B.3.2: an unavailable expert must not
 *                         skew the weights of the available ones).
 *  MOE_GATE_SOFTMAX       raw softmax probability over all E experts.
 *  MOE_GATE_SIGMOID       independent logistic gate (the sigma-MoE gate). */
enum { MOE_GATE_SOFTMAX_TOPK = 0, MOE_GATE_SOFTMAX = 1, MOE_GATE_SIGMOID = 2 };

/* status codes */
enum { MOE_OK = 0, MOE_ERR_ARG = -1, MOE_ERR_UNSUPPORTED = -2, MOE_ERR_HIP = -3 };

/* Message for the last non-OK return on the calling thread ("" if none). */
const char* moe_last_error(void);

/* ABI version of this header (incremented on incompatible change). */
int moe_abi_version(void);

/*
 * Router scores, top-k selection, gate weights and ghost-expert mask
 * (App. A: T(x) = TopK of the router scores; Sec. 3.3: ghost experts).
 *
 *   z[t,e]        = (x[t,:] . w_router[e,:] + router_bias[e]) * inv_tau, all E
 *   topk_idx[t,j] = the k experts with the largest z[t,:], in descending z;
 *                   equal logits go to the lower expert id
 *   topk_w[t,j]   = gate weight of topk_idx[t,j] (see MOE_GATE_*)
 *   topk_local[t,j] = rank of topk_idx[t,j] in the sorted resident set, or -1
 *                   when that expert is not resident (a ghost route)
 *
 * x [T,d] dtype; w_router [E,d] dtype; router_bias [E] fp32 or NULL;
 * resident [E] uint8 (nonzero = resident on this worker);
 * logits [T,E] fp32 or NULL (not written when NULL);
 * topk_idx, topk_local [T,k] int32; topk_w [T,k] fp32.
 * Limits: 1 <= k <= E <= 256, T >= 0, d >= 1 (d % 8 == 0 for bf16).
 */
int moe_route_mask(const void* x, const void* w_router, const float* router_bias, int dtype,
                   int T, int d, int E, int k, float inv_tau, int gate,
                   const uint8_t* resident, float* logits, int32_t* topk_idx,
                   float* topk_w, int32_t* topk_local, hipStream_t stream);

/*
 * Backward of moe_route_mask with the top-k set held fixed.
 *
 *   dz[t,e]         = dL/dz[t,e] (fp32 [T,E], written in full; zero off the
 *                     top-k for the SOFTMAX_TOPK and SIGMOID gates)
 *   dw_router[e,:]  = inv_tau * sum_t dz[t,e] x[t,:]      (fp32 [E,d])
 *   d_bias[e]       = inv_tau * sum_t dz[t,e]             (fp32 [E] or NULL)
 *   dx[t,:]        (+)= inv_tau * sum_e dz[t,e] w_router[e,:]   (dtype [T,d])
 *
 * d_topk_w [T,k] fp32 is dL/dtopk_w (0 for ghost routes, as moe_combine_bwd
 * writes it).  logits is required for MOE_GATE_SOFTMAX and may be NULL
 * otherwise.  accumulate_dx != 0 adds into dx, else overwrites it.
 * ws: device workspace (16-byte aligned) of at least
 * moe_route_bwd_workspace_size(T, d, E) bytes; its contents on entry are
 * ignored.  In bf16 with E <= 64 and
 * d % 128 == 0 the fp32 dz enters the MFMA products as a bf16 pair hi + lo
 * (relative error <= 2^-17 per element); otherwise the sums run in fp32 FMA.
 * Every sum is taken in a fixed order, so results are run-to-run identical.
 */
size_t moe_route_bwd_workspace_size(int T, int d, int E);
int moe_route_bwd(const void* x, const void* w_router, int dtype, int T, int d, int E, int k,
                  float inv_tau, int gate, const int32_t* topk_idx, const float* topk_w,
                  const float* logits, const float* d_topk_w, float* dz, float* dw_router,
                  float* d_bias, void* dx, int accumulate_dx, void* ws, size_t ws_bytes,
                  hipStream_t stream);

/*
 * Dispatch: group the resident routes by local expert (tokens are processed
 * only by experts hosted on this worker, Sec. 3.3.2) and gather their rows.
 *
 *   counts[r]  = number of routes with topk_local == r            [E_r]
 *   offsets[r] = sum_{r' < r} counts[r'];  offsets[E_r] = n          [E_r+1]
 *   slots [offsets[r], offsets[r+1]) hold the routes of local expert r in
 *   ascending token order; perm[p] = t*k + j of the route in slot p
 *   inv_perm[t,j] = its slot, or -1 for a ghost route               [T,k]
 *   xp[p,:] = x[perm[p]/k, :]                                         [cap,d]
 *
 * cap = T * min(k, E_r) bounds n; perm and xp have cap rows, of which rows
 * n..cap-1 are left untouched.  ws: at least moe_dispatch_workspace_size()
 * bytes; its contents on entry are ignored.  Limits: E_r <= 256.
 */
size_t moe_dispatch_workspace_size(int T, int k, int E_r);
int moe_dispatch(const void* x, int dtype, int T, int d, int k, int E_r,
                 const int32_t* topk_local, int32_t* counts, int32_t* offsets,
                 int32_t* perm, int32_t* inv_perm, void* xp, void* ws, size_t ws_bytes,
                 hipStream_t stream);

/*
 * moe_dispatch without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, outputs, limits and results as
 * moe_dispatch; the workspace is a library-owned device array of
 * MOE_DISPATCH_NOALLOC_MAX_WS bytes per device, reserved from the library's
 * load until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); its first call on a device resolves
 * that device's array address.  Returns MOE_ERR_UNSUPPORTED when
 * moe_dispatch_workspace_size(T, k, E_r) exceeds MOE_DISPATCH_NOALLOC_MAX_WS
 * (for example E_r = 256 with T above 130816), MOE_ERR_HIP when the array
 * cannot be resolved.  All calls on one device share its array: calls that
 * overlap in time on one device (different streams, or host threads) race
 * and give undefined results; calls ordered on one stream are safe.
 */
#define MOE_DISPATCH_NOALLOC_MAX_WS ((size_t)1 << 20)
int moe_dispatch_noalloc(const void* x, int dtype, int T, int d, int k, int E_r,
                         const int32_t* topk_local, int32_t* counts, int32_t* offsets,
                         int32_t* perm, int32_t* inv_perm, void* xp, hipStream_t stream);

/*
 * Backward of the gather (un-permute):
 *   dx[t,:] (+)= sum_{j: inv_perm[t,j] >= 0} dxp[inv_perm[t,j], :]
 * A token whose routes are all ghosts gets exactly 0 (or keeps dx when
 * accumulate != 0).  dxp [cap,d], dx [T,d], both dtype.  Slots outside
 * [0, cap) are treated as ghost routes (cap = rows of dxp).
 */
int moe_dispatch_bwd(const void* dxp, int dtype, int T, int d, int k, int cap,
                     const int32_t* inv_perm, void* dx, int accumulate, hipStream_t stream);

/*
 * Grouped SwiGLU expert FFN, forward: the expert outputs E_i(x) of the
 * combine (App. A), evaluated only for the experts this worker hosts and only
 * on the rows routed to them (Sec. 3.3.3 "Ghost Experts and Skip-Token";
 * Alg. 2's local step).  The SwiGLU form is the one the layer workloads use;
 * MOE_ACT_SILU below selects the paper's own expert (App. B.3.1).  Group g is
 * rows [offsets[g], offsets[g+1]) of xp and uses expert g's weights:
 *   G = X Wg^T, U = X Wu^T, Hh = silu(G) * U, Y = Hh Wd^T   (no biases)
 * w_gate_up [n_groups, 2H, d]: rows 0..H-1 are Wg, rows H..2H-1 are Wu.
 * w_down    [n_groups, d, H].
 * Outputs (rows of each group only): gu [cap, 2H] = [G | U], h [cap, H] = Hh,
 * yp [cap, d].  Shared (always-active) experts are run through the same call
 * with n_groups = 1, offsets = {0, T}, xp = x; several shared experts on the
 * same input are one expert with their hidden units concatenated.
 * offsets is a device array of n_groups + 1 non-decreasing int32 values; each
 * group is clamped to [0, cap].
 * Limits: n_groups <= 256 (the GEMM kernels hold the group table in LDS),
 * H % 64 == 0; fp32: d % 8 == 0; bf16: d % 64 == 0 and each operand below
 * 4 GiB (2 cap max(d, 2H) and 2 n_groups 2H d bytes below 2^32 - 16: the
 * GEMMs address operands with 32-bit byte offsets); MOE_ERR_UNSUPPORTED
 * otherwise.
 */
int moe_grouped_ffn_fwd(const void* xp, const void* w_gate_up, const void* w_down, int dtype,
                        int cap, int d, int H, int n_groups, const int32_t* offsets,
                        void* gu, void* h, void* yp, hipStream_t stream);

/*
 * Grouped SwiGLU expert FFN, backward: the gradients of the resident
 * experts' parameters and of their input rows that the local step of Alg. 2
 * needs (the chain rule of the forward, per group; the SiLU form as stated
 * with MOE_ACT_SILU below):
 *   dHh = dY Wd;  dG = dHh * U * silu'(G);  dU = dHh * silu(G)
 *   dX  = dG Wg + dU Wu
 *   dWd = dY^T Hh;  dWg = dG^T X;  dWu = dU^T X           (fp32, per expert)
 * dyp [cap,d], xp [cap,d], gu [cap,2H], h [cap,H] as written by the forward.
 * Outputs: dgu [cap,2H] = [dG | dU] (dtype), dxp [cap,d] (dtype),
 * dw_gate_up [n_groups,2H,d] fp32, dw_down [n_groups,d,H] fp32 - written for
 * every group (zero for an empty group), or added to when accumulate_dw != 0.
 * Limits as for the forward, and 4 * 2H * d bytes of one expert's dw_gate_up
 * below 4 GiB.
 */
int moe_grouped_ffn_bwd(const void* dyp, const void* xp, const void* gu, const void* h,
                        const void* w_gate_up, const void* w_down, int dtype, int cap, int d,
                        int H, int n_groups, const int32_t* offsets, void* dgu, void* dxp,
                        float* dw_gate_up, float* dw_down, int accumulate_dw,
                        hipStream_t stream);

/*
 * Several expert sets in one call.  A set is a group of experts with one
 * hidden size and one input buffer: the routed resident experts (xp = the
 * dispatched rows, groups = the dispatch offsets) or the merged shared
 * experts (Sec. 3.2: dense, always active; xp = x, offsets = {0, T}).  The
 * sets' tiles of each GEMM share one launch, so the small routed groups and
 * the large shared group fill the GPU together; the results are those of one
 * moe_grouped_ffn_fwd / _bwd call per set.  Every field has the meaning and
 * layout of the matching argument of those calls; fields a direction does
 * not use may be NULL (forward: dyp, dgu, dxp, dw_gate_up, dw_down; backward:
 * yp).  gu and h are written by the forward and read by the backward.
 * n_sets is 1 or 2; all sets share dtype and d.
 */
/*
 * Expert form of a set.  MOE_ACT_SWIGLU: the SwiGLU expert above.
 * MOE_ACT_SILU: the paper's own expert (App. B.3.1), a projection to the
 * hidden size followed by SiLU and the projection back,
 *   A = X W1^T;  Hh = silu(A);  Y = Hh Wd^T
 * with backward dHh = dY Wd, dA = dHh * silu'(A), dX = dA W1, dW1 = dA^T X,
 * dWd = dY^T Hh.  Then w_gate_up holds W1 [n_groups, H, d], gu holds A
 * [cap, H], dgu holds dA [cap, H] and dw_gate_up is [n_groups, H, d]; every
 * other field is as for SwiGLU.
 */
enum { MOE_ACT_SWIGLU = 0, MOE_ACT_SILU = 1 };

typedef struct moe_ffn_set {
  const void* xp;          /* [cap, d] */
  const void* w_gate_up;   /* [n_groups, 2H, d] */
  const void* w_down;      /* [n_groups, d, H] */
  const int32_t* offsets;  /* device, [n_groups + 1] */
  int cap, H, n_groups;
  void* gu;                /* [cap, 2H] */
  void* h;                 /* [cap, H] */
  void* yp;                /* [cap, d] */
  const void* dyp;         /* [cap, d] */
  void* dgu;               /* [cap, 2H] */
  void* dxp;               /* [cap, d] */
  float* dw_gate_up;       /* [n_groups, 2H, d] fp32 */
  float* dw_down;          /* [n_groups, d, H] fp32 */
  int activation;          /* MOE_ACT_SWIGLU (0) or MOE_ACT_SILU; the same in every set */
} moe_ffn_set;

/*
 * ws: device workspace of at least moe_grouped_ffn_fwd_workspace_size(sets,
 * n_sets, dtype, d) bytes (which may be 0), 256-byte aligned, or NULL with
 * ws_bytes = 0.  Its contents on entry are ignored.  With a workspace (bf16)
 * the down projection may cut its reduction (the hidden units) into up to 8
 * parts when its output tiles are too few to fill the GPU (small groups,
 * e.g. few resident experts): each part writes fp32 partial rows, summed in
 * a fixed part order into yp afterwards.  The kernel chooses the parts from
 * the device-side group sizes; partials of at most 256 MiB per set are
 * reserved (none when two do not fit).  Results are run-to-run identical.
 */
size_t moe_grouped_ffn_fwd_workspace_size(const moe_ffn_set* sets, int n_sets, int dtype, int d);
int moe_grouped_ffn_fwd_sets(const moe_ffn_set* sets, int n_sets, int dtype, int d, void* ws,
                             size_t ws_bytes, hipStream_t stream);
/*
 * ws: device workspace of at least moe_grouped_ffn_bwd_workspace_size(sets,
 * n_sets, dtype, d) bytes, 256-byte aligned, or NULL with ws_bytes = 0.  Its
 * contents on entry are ignored.  With a workspace the weight-gradient GEMMs
 * hand out tiles dynamically (per-XCD counters) and a set with one large
 * group (the shared experts) may have its rows split into parts whose fp32
 * partial gradients are summed in a fixed order afterwards; dX may cut its
 * reduction (the 2H columns of [dG | dU]) into parts as the forward's down
 * projection does.  The size depends on the sets and on the device's
 * compute-unit count.  Results are run-to-run identical either way.
 */
size_t moe_grouped_ffn_bwd_workspace_size(const moe_ffn_set* sets, int n_sets, int dtype, int d);
int moe_grouped_ffn_bwd_sets(const moe_ffn_set* sets, int n_sets, int dtype, int d,
                             int accumulate_dw, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Weighted combine (App. A: y = sum_{i in T(x)} s_i(x) E_i(x)):
 *   y[t,:] = sum_{j: inv_perm[t,j] >= 0} topk_w[t,j] * yp[inv_perm[t,j], :]
 *            (+ y_add[t,:] when y_add != NULL, e.g. the shared experts' output)
 * Ghost routes are skipped; a token whose routes are all ghosts gets exactly
 * y_add[t,:] (exactly 0 when y_add == NULL).  yp [cap,d], y_add, y [T,d].
 * Slots outside [0, cap) are treated as ghost routes (cap = rows of yp).
 */
int moe_combine_fwd(const void* yp, int dtype, int T, int d, int k, int cap, const float* topk_w,
                    const int32_t* inv_perm, const void* y_add, void* y, hipStream_t stream);

/*
 * Backward of the combine:
 *   dyp[p,:]      = topk_w[t,j] * dy[t,:]         for p = inv_perm[t,j] >= 0
 *   d_topk_w[t,j] = <dy[t,:], yp[p,:]>  (fp32), 0 for a ghost route
 * yp, dyp [cap,d]; slots outside [0, cap) are treated as ghost routes.
 */
int moe_combine_bwd(const void* dy, const void* yp, int dtype, int T, int d, int k, int cap,
                    const float* topk_w, const int32_t* inv_perm, void* dyp, float* d_topk_w,
                    hipStream_t stream);

/*
 * Round boundary: expert-wise pseudo-gradient of the resident experts and its
 * average over the expert's replica group (Alg. 2, aggregation of the sparse
 * parameters within expert replica groups; Sec. 3.4 "Round structure").
 *   delta_local = theta_start - theta_now
 *   delta_avg   = (((delta_local + peers[0]) + peers[1]) + ...) * (1/(n_peers+1))
 * evaluated elementwise in fp32 in exactly that order (the reciprocal is the
 * fp32-rounded 1/(n_peers+1)), so the result is reproducible bit for bit.
 * peers is a HOST array of n_peers device pointers, each to n_params fp32
 * values (the other replicas' deltas).  delta_local may be NULL.
 * Limits: 0 <= n_peers <= 16.
 */
int moe_expert_delta(const float* theta_start, const float* theta_now,
                     const float* const* peers, int n_peers, size_t n_params,
                     float* delta_local, float* delta_avg, hipStream_t stream);

/*
 * Optimisers of the resident experts' fp32 master parameters (Sec. 3.4
 * "Outer optimization": AdamW on the worker's own parameters during the local
 * steps, with the state kept across rounds and only for its own experts; a
 * momentum outer step on the replica-group average at the round boundary;
 * App. F: AdamW weight decay 0, betas (0.9, 0.95), eps 1e-8, Nesterov outer
 * step with learning rate 0.7 and momentum 0.9, LocalAdamW averaging of the
 * moments).  All arrays are device fp32 [n] (theta_bf16: bf16 [n]), 16-byte
 * aligned, owned by the caller, updated in place.  Each element is computed
 * in fp32 one rounding at a time in the order written below (no fused
 * multiply-add; correctly rounded division and square root), so results are
 * reproducible bit for bit.  theta_bf16 (may be NULL) receives the updated
 * parameters rounded to bf16 (nearest even): the working copy the bf16
 * grouped GEMMs read (w_gate_up / w_down share the fp32 masters' layout).
 * Returns MOE_ERR_ARG for NULL required arrays or bad hyper-parameters,
 * MOE_ERR_UNSUPPORTED for misaligned arrays.
 *
 * moe_adamw_step, step t >= 1 (c1 = 1 - beta1^t, c2 = 1 - beta2^t, evaluated
 * in double and rounded to fp32):
 *   m = beta1 m + (1 - beta1) g;   v = beta2 v + (1 - beta2) (g g)
 *   theta = theta - lr ((m / c1) / (sqrt(v / c2) + eps) + weight_decay theta)
 */
int moe_adamw_step(float* theta, const float* grad, float* m, float* v, size_t n, int step,
                   float lr, float beta1, float beta2, float eps, float weight_decay,
                   void* theta_bf16, hipStream_t stream);

/*
 * moe_outer_nesterov: the outer step of a round on the replica-group average
 * delta_avg (from moe_expert_delta) with momentum buffer b (zero before the
 * first round):
 *   b = mu b + delta_avg;   theta = theta_start - lr (delta_avg + mu b)
 * and theta is written to theta_start and theta_now (where every replica
 * starts the next round) and, if non-NULL, to theta_bf16.
 */
int moe_outer_nesterov(float* theta_start, float* theta_now, const float* delta_avg,
                       float* momentum, size_t n, float lr, float mu, void* theta_bf16,
                       hipStream_t stream);

/*
 * moe_replica_mean: the replica-group average of a tensor (LocalAdamW's
 * moment synchronisation):
 *   out = (((local + peers[0]) + peers[1]) + ...) * fp32(1 / (n_peers + 1))
 * peers is a HOST array of n_peers device pointers; 0 <= n_peers <= 16; out
 * may alias local.
 */
int moe_replica_mean(const float* local, const float* const* peers, int n_peers, size_t n,
                     float* out, hipStream_t stream);

/*
 * Expert placement and migration (Alg. 1; Sec. 3.3 "Expert placement modes").
 * Every expert lives on exactly O_e of M workers and every worker holds
 * N_le = O_e N_e / M distinct experts; random placement redraws the map every
 * T rounds, after which a worker fetches the experts new to it (Delta_in),
 * keeps the optimiser state of the others and restarts that of the new ones
 * with a learning-rate warm-up (Sec. 3.4).
 *
 * moe_gen_placement (host only): sets [M, N_le] (host) receives each worker's
 * sorted expert ids.  The (expert, replica) slots in expert order are dealt
 * to the workers in turn - expert e on workers (e O_e + j) mod M, j < O_e -
 * after relabelling experts by expert_perm and workers by worker_perm (host
 * permutations of 0..N_e-1 and 0..M-1; NULL = identity, the fixed placement;
 * random placement passes uniformly drawn ones).  MOE_ERR_ARG unless
 * 1 <= O_e <= M, M divides N_e O_e and the permutations are valid.
 */
int moe_gen_placement(int N_e, int O_e, int M, const int32_t* expert_perm,
                      const int32_t* worker_perm, int32_t* sets);

/*
 * moe_migration_map (host only): for slot i of the new resident set (strictly
 * ascending ids), map[i] = the slot of the same expert in the previous set,
 * or -1 if the expert is new to the worker.
 */
int moe_migration_map(const int32_t* prev_set, int n_prev, const int32_t* new_set, int n_new,
                      int32_t* map);

/*
 * moe_copy_expert_rows: dst[dst_row[r], :] = src[src_row[r], :] for
 * src_row[r] >= 0, zeros for src_row[r] = -1, r < n_rows <= 256; rows of
 * row_len fp32 values (row_len % 4 == 0); src_row and dst_row are HOST arrays
 * (dst_row NULL = 0..n_rows-1, otherwise distinct).  The migration step:
 * weights of the new set from the global store, optimiser state from the
 * previous local layout by moe_migration_map (-1 = restarted), and the
 * resident rows back into the global store.  The rows read must not overlap
 * the rows written.  dst_bf16 (may be NULL) receives the written rows rounded
 * to bf16 (nearest even) in dst's layout: the working copy of migrated
 * weights.
 */
int moe_copy_expert_rows(const float* src, const int32_t* src_row, float* dst,
                         const int32_t* dst_row, int n_rows, size_t row_len, void* dst_bf16,
                         hipStream_t stream);

/*
 * moe_warmup_lr (host only): the learning rate of each resident expert under
 * the warm-up that Sec. 3.4 prescribes for experts new to a worker.  The
 * paper gives no shape; this library's reading is linear over warmup_steps
 * local steps counted from the (re)start of the expert's optimiser state, so
 * lr_out[r] = (float)(lr * min(1, steps[r] / warmup_steps)), evaluated in
 * double and rounded once; warmup_steps <= 0 gives lr to every row.  Experts
 * kept across a migration keep their count and so leave the warm-up on
 * schedule.  steps (each >= 0) and lr_out are HOST arrays of n_rows (>= 0);
 * MOE_ERR_ARG on a NULL array, a negative count or a non-finite lr.  The
 * rates feed moe_adamw_step_rows.
 */
int moe_warmup_lr(const int* steps, int n_rows, double lr, int warmup_steps, float* lr_out);

/*
 * moe_adamw_step_rows: moe_adamw_step over n_rows experts of row_len
 * parameters each, with expert r at its own step count steps[r] >= 1 (its
 * steps since its state was (re)started) and learning rate lr[r] (the
 * warm-up of reassigned experts); steps and lr are HOST arrays.  Row r is
 * bit-for-bit moe_adamw_step(row r, steps[r], lr[r]).  Rows that share
 * (step, lr) are updated by one launch.
 */
int moe_adamw_step_rows(float* theta, const float* grad, float* m, float* v, int n_rows,
                        size_t row_len, const int* steps, const float* lr, float beta1,
                        float beta2, float eps, float weight_decay, void* theta_bf16,
                        hipStream_t stream);

/*
 * Measurement support for benchmarks and profilers (not part of the layer).
 * moe_timing_enable(capacity > 0) creates a pool of 2*capacity HIP events on
 * the current device and from then on brackets every kernel this library
 * launches with an event pair on the launch's stream (launches beyond the
 * capacity are not recorded).  moe_timing_enable(0) stops recording and
 * releases the pool.  moe_timing_collect() waits for the recorded events,
 * sums the elapsed time per kernel name into out[0..*n_out) (at most max_out
 * entries; names are static strings owned by the library) and clears the
 * record.  Enabling is the one call that allocates (the event pool); it is
 * process-wide and must not race with launches on other threads.
 */
typedef struct {
  const char* name;
  int launches;
  float total_ms;
  float min_ms;
  float max_ms;
} moe_kernel_time;
int moe_timing_enable(int capacity);
int moe_timing_collect(moe_kernel_time* out, int max_out, int* n_out);

#ifdef __cplusplus
}
#endif
#endif /* MOE_RESIDENT_H */
