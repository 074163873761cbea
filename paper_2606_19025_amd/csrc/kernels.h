// Host-side launchers of the gfx950 kernels (internal; the public ABI is in
// include/moe_resident.h).  Each launcher assumes validated arguments and
// only enqueues work on `stream`; it returns hipGetLastError().
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "moe_resident.h"

namespace moe {

hipError_t launch_route_fwd(const void* x, const void* w, const float* bias, int bf16, int T,
                            int d, int E, int k, float inv_tau, int gate, const uint8_t* resident,
                            float* logits, int32_t* idx, float* tw, int32_t* local,
                            hipStream_t s);

size_t route_bwd_ws_bytes(int T, int d, int E);
hipError_t launch_route_bwd(const void* x, const void* w, int bf16, int T, int d, int E, int k,
                            float inv_tau, int gate, const int32_t* idx, const float* tw,
                            const float* logits, const float* dtw, float* dz, float* dw_router,
                            float* d_bias, void* dx, int accumulate_dx, void* ws,
                            hipStream_t s);

size_t dispatch_ws_bytes(int T, int k, int E_r);
hipError_t launch_dispatch(const void* x, int bf16, int T, int d, int k, int E_r,
                           const int32_t* local, int32_t* counts, int32_t* offsets,
                           int32_t* perm, int32_t* inv_perm, void* xp, void* ws, hipStream_t s);
// The same counting sort with its workspace in a library-owned device array
// of kDispatchScratchBytes (one per device); dispatch_ws_bytes() of the call
// must not exceed it.
constexpr size_t kDispatchScratchBytes = MOE_DISPATCH_NOALLOC_MAX_WS;
hipError_t launch_dispatch_noalloc(const void* x, int bf16, int T, int d, int k, int E_r,
                                   const int32_t* local, int32_t* counts, int32_t* offsets,
                                   int32_t* perm, int32_t* inv_perm, void* xp, hipStream_t s);
hipError_t launch_dispatch_bwd(const void* dxp, int bf16, int T, int d, int k, int cap,
                               const int32_t* inv_perm, void* dx, int accumulate, hipStream_t s);

hipError_t launch_combine_fwd(const void* yp, int bf16, int T, int d, int k, int cap,
                              const float* tw, const int32_t* inv_perm, const void* y_add, void* y,
                              hipStream_t s);
hipError_t launch_combine_bwd(const void* dy, const void* yp, int bf16, int T, int d, int k,
                              int cap, const float* tw, const int32_t* inv_perm, void* dyp,
                              float* dtw, hipStream_t s);

// Grouped SwiGLU FFN over 1 or 2 expert sets (moe_ffn_set of the public
// header), one launch per GEMM kind.  ws: NULL (no K parts) or
// ffn_fwd_ws_bytes() bytes, 256-byte aligned; its contents on entry are ignored.
size_t ffn_fwd_ws_bytes(const moe_ffn_set* sets, int n_sets, int bf16, int d);
hipError_t launch_ffn_fwd_sets(const moe_ffn_set* sets, int n_sets, int bf16, int d, void* ws,
                               hipStream_t s);
// ws: NULL (static tile dealing, no split-K) or ffn_bwd_ws_bytes() bytes,
// 256-byte aligned; its contents on entry are ignored.
size_t ffn_bwd_ws_bytes(const moe_ffn_set* sets, int n_sets, int bf16, int d);
hipError_t launch_ffn_bwd_sets(const moe_ffn_set* sets, int n_sets, int bf16, int d,
                               int accumulate_dw, void* ws, hipStream_t s);

constexpr int kMaxPeers = 16;
hipError_t launch_expert_delta(const float* start, const float* now, const float* const* peers,
                               int n_peers, size_t n, float* dl, float* avg, hipStream_t s);

// Optimisers (optim.hip); c1, c2 = the step's AdamW bias corrections.
hipError_t launch_adamw(float* theta, const float* grad, float* m, float* v, size_t n, float lr,
                        float beta1, float beta2, float eps, float wd, float c1, float c2,
                        void* theta_bf16, hipStream_t s);
hipError_t launch_outer_nesterov(float* start, float* now, const float* delta, float* mom,
                                 size_t n, float lr, float mu, void* theta_bf16, hipStream_t s);
hipError_t launch_replica_mean(const float* local, const float* const* peers, int n_peers,
                               size_t n, float* out, hipStream_t s);

// Placement and migration (placement.hip).  gen_placement: false when the
// constraints cannot be met.  launch_copy_expert_rows: src_row / dst_row are
// host arrays of n_rows <= 256 entries (dst_row NULL = 0..n_rows-1).
bool gen_placement(int N_e, int O_e, int M, const int32_t* expert_perm,
                   const int32_t* worker_perm, int32_t* sets);
hipError_t launch_copy_expert_rows(const float* src, const int32_t* src_row, float* dst,
                                   const int32_t* dst_row, int n_rows, size_t row_len,
                                   void* dst_bf16, hipStream_t s);

}  // namespace moe
