// C ABI of the resident-expert MoE layer: argument validation on the host,
// then the kernel launchers.  Declarations and contracts: moe_resident.h.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "moe_resident.h"
#include "timing.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return MOE_OK;
}

int hip_status(hipError_t e, const char* where) {
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE(cond, ...) \
  do {                     \
    if (!(cond)) return fail(MOE_ERR_ARG, __VA_ARGS__); \
  } while (0)
#define SUPPORT(cond, ...) \
  do {                     \
    if (!(cond)) return fail(MOE_ERR_UNSUPPORTED, __VA_ARGS__); \
  } while (0)

int check_dtype(int dtype) {
  SUPPORT(dtype == MOE_F32 || dtype == MOE_BF16, "unsupported dtype %d", dtype);
  return MOE_OK;
}

// row vectors of 16 bytes: d % 8 == 0 and 16-byte aligned base pointers
int check_rows16(int d, const char* name, const void* p) {
  SUPPORT(d % 8 == 0, "d = %d must be a multiple of 8", d);
  SUPPORT(p == nullptr || aligned16(p), "%s must be 16-byte aligned", name);
  return MOE_OK;
}

// ---------------------------------------------------------------- timing pool
std::mutex g_tmu;
std::atomic<bool> g_ton{false};
std::vector<hipEvent_t> g_pool;
struct TimingRec {
  const char* name;
  int ev;
};
std::vector<TimingRec> g_recs;
int g_next = 0;
thread_local int t_open = -1;

void release_pool() {
  for (hipEvent_t e : g_pool) (void)hipEventDestroy(e);
  g_pool.clear();
  g_recs.clear();
  g_next = 0;
}

}  // namespace

namespace moe {
bool timing_on() { return g_ton.load(std::memory_order_relaxed); }

void timing_begin(const char* name, hipStream_t s) {
  std::lock_guard<std::mutex> lock(g_tmu);
  t_open = -1;
  if (g_next + 2 > (int)g_pool.size()) return;
  const int ev = g_next;
  g_next += 2;
  if (hipEventRecord(g_pool[ev], s) != hipSuccess) return;
  g_recs.push_back({name, ev});
  t_open = ev;
}

void timing_end(hipStream_t s) {
  if (t_open < 0) return;
  std::lock_guard<std::mutex> lock(g_tmu);
  (void)hipEventRecord(g_pool[t_open + 1], s);
  t_open = -1;
}
}  // namespace moe

extern "C" {

int moe_timing_enable(int capacity) {
  REQUIRE(capacity >= 0, "capacity = %d must be >= 0", capacity);
  std::lock_guard<std::mutex> lock(g_tmu);
  g_ton.store(false);
  release_pool();
  if (capacity == 0) return ok();
  g_pool.resize(2 * (size_t)capacity);
  for (auto& e : g_pool) {
    if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
      release_pool();
      return fail(MOE_ERR_HIP, "hipEventCreate failed");
    }
  }
  g_recs.reserve(capacity);
  g_ton.store(true);
  return ok();
}

int moe_timing_collect(moe_kernel_time* out, int max_out, int* n_out) {
  REQUIRE(out && n_out && max_out >= 0, "out and n_out must not be NULL");
  std::lock_guard<std::mutex> lock(g_tmu);
  int n = 0;
  for (const TimingRec& r : g_recs) {
    hipError_t e = hipEventSynchronize(g_pool[r.ev + 1]);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, g_pool[r.ev], g_pool[r.ev + 1]);
    if (e != hipSuccess) {
      g_recs.clear();
      g_next = 0;
      return fail(MOE_ERR_HIP, "timing: %s", hipGetErrorString(e));
    }
    int i = 0;
    while (i < n && std::strcmp(out[i].name, r.name) != 0) ++i;
    if (i == n) {
      if (n == max_out) continue;
      out[n++] = moe_kernel_time{r.name, 0, 0.f, 1e30f, 0.f};
    }
    out[i].launches += 1;
    out[i].total_ms += ms;
    out[i].min_ms = std::min(out[i].min_ms, ms);
    out[i].max_ms = std::max(out[i].max_ms, ms);
  }
  g_recs.clear();
  g_next = 0;
  *n_out = n;
  return ok();
}

const char* moe_last_error(void) { return g_err.c_str(); }

int moe_abi_version(void) { return 3; }

int moe_route_mask(const void* x, const void* w_router, const float* router_bias, int dtype,
                   int T, int d, int E, int k, float inv_tau, int gate,
                   const uint8_t* resident, float* logits, int32_t* topk_idx, float* topk_w,
                   int32_t* topk_local, hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0, "T = %d must be >= 0", T);
  REQUIRE(d >= 1, "d = %d must be >= 1", d);
  REQUIRE(E >= 1 && E <= 256, "E = %d must be in [1, 256]", E);
  REQUIRE(k >= 1 && k <= E, "k = %d must be in [1, E = %d]", k, E);
  REQUIRE(gate >= MOE_GATE_SOFTMAX_TOPK && gate <= MOE_GATE_SIGMOID, "unknown gate %d", gate);
  REQUIRE(std::isfinite(inv_tau) && inv_tau > 0.f, "inv_tau must be finite and > 0");
  REQUIRE(w_router && resident, "w_router and resident must not be NULL");
  REQUIRE(T == 0 || (x && topk_idx && topk_w && topk_local), "x and the top-k outputs must not be NULL");
  if (dtype == MOE_BF16) {
    if ((r = check_rows16(d, "x", x)) != MOE_OK) return r;
    if ((r = check_rows16(d, "w_router", w_router)) != MOE_OK) return r;
  }
  return hip_status(moe::launch_route_fwd(x, w_router, router_bias, dtype == MOE_BF16, T, d, E, k,
                                          inv_tau, gate, resident, logits, topk_idx, topk_w,
                                          topk_local, stream),
                    "moe_route_mask");
}

size_t moe_route_bwd_workspace_size(int T, int d, int E) {
  if (T < 0 || d < 1 || E < 1) return 0;
  return moe::route_bwd_ws_bytes(T, d, E);
}

int moe_route_bwd(const void* x, const void* w_router, int dtype, int T, int d, int E, int k,
                  float inv_tau, int gate, const int32_t* topk_idx, const float* topk_w,
                  const float* logits, const float* d_topk_w, float* dz, float* dw_router,
                  float* d_bias, void* dx, int accumulate_dx, void* ws, size_t ws_bytes,
                  hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0 && d >= 1, "bad sizes T = %d, d = %d", T, d);
  REQUIRE(E >= 1 && E <= 256, "E = %d must be in [1, 256]", E);
  REQUIRE(k >= 1 && k <= E, "k = %d must be in [1, E = %d]", k, E);
  REQUIRE(gate >= MOE_GATE_SOFTMAX_TOPK && gate <= MOE_GATE_SIGMOID, "unknown gate %d", gate);
  REQUIRE(std::isfinite(inv_tau) && inv_tau > 0.f, "inv_tau must be finite and > 0");
  REQUIRE(w_router && dw_router, "w_router and dw_router must not be NULL");
  REQUIRE(T == 0 || (x && topk_idx && topk_w && d_topk_w && dz && dx),
          "x, topk_idx, topk_w, d_topk_w, dz and dx must not be NULL");
  REQUIRE(gate != MOE_GATE_SOFTMAX || T == 0 || logits, "logits are required for MOE_GATE_SOFTMAX");
  const size_t need = moe::route_bwd_ws_bytes(T, d, E);
  REQUIRE(ws && ws_bytes >= need, "workspace of %zu bytes needed (got %zu)", need, ws_bytes);
  if ((r = check_rows16(d, "x", x)) != MOE_OK) return r;
  if ((r = check_rows16(d, "dx", dx)) != MOE_OK) return r;
  if ((r = check_rows16(d, "w_router", w_router)) != MOE_OK) return r;
  SUPPORT(aligned16(ws), "the workspace must be 16-byte aligned");
  return hip_status(moe::launch_route_bwd(x, w_router, dtype == MOE_BF16, T, d, E, k, inv_tau, gate,
                                          topk_idx, topk_w, logits, d_topk_w, dz, dw_router,
                                          d_bias, dx, accumulate_dx, ws, stream),
                    "moe_route_bwd");
}

size_t moe_dispatch_workspace_size(int T, int k, int E_r) {
  if (T < 0 || k < 1 || E_r < 0) return 0;
  return moe::dispatch_ws_bytes(T, k, E_r);
}

int moe_dispatch(const void* x, int dtype, int T, int d, int k, int E_r,
                 const int32_t* topk_local, int32_t* counts, int32_t* offsets, int32_t* perm,
                 int32_t* inv_perm, void* xp, void* ws, size_t ws_bytes, hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0 && d >= 1 && k >= 1, "bad sizes T = %d, d = %d, k = %d", T, d, k);
  REQUIRE(E_r >= 0 && E_r <= 256, "E_r = %d must be in [0, 256]", E_r);
  REQUIRE(offsets && (E_r == 0 || counts), "counts and offsets must not be NULL");
  REQUIRE(T == 0 || (x && topk_local && inv_perm && (E_r == 0 || (perm && xp))),
          "x, topk_local, perm, inv_perm and xp must not be NULL");
  const size_t need = moe::dispatch_ws_bytes(T, k, E_r);
  REQUIRE(ws && ws_bytes >= need, "workspace of %zu bytes needed (got %zu)", need, ws_bytes);
  if ((r = check_rows16(d, "x", x)) != MOE_OK) return r;
  if ((r = check_rows16(d, "xp", xp)) != MOE_OK) return r;
  return hip_status(moe::launch_dispatch(x, dtype == MOE_BF16, T, d, k, E_r, topk_local, counts,
                                         offsets, perm, inv_perm, xp, ws, stream),
                    "moe_dispatch");
}

int moe_dispatch_noalloc(const void* x, int dtype, int T, int d, int k, int E_r,
                         const int32_t* topk_local, int32_t* counts, int32_t* offsets,
                         int32_t* perm, int32_t* inv_perm, void* xp, hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0 && d >= 1 && k >= 1, "bad sizes T = %d, d = %d, k = %d", T, d, k);
  REQUIRE(E_r >= 0 && E_r <= 256, "E_r = %d must be in [0, 256]", E_r);
  REQUIRE(offsets && (E_r == 0 || counts), "counts and offsets must not be NULL");
  REQUIRE(T == 0 || (x && topk_local && inv_perm && (E_r == 0 || (perm && xp))),
          "x, topk_local, perm, inv_perm and xp must not be NULL");
  const size_t need = moe::dispatch_ws_bytes(T, k, E_r);
  SUPPORT(need <= MOE_DISPATCH_NOALLOC_MAX_WS,
          "moe_dispatch_noalloc: T = %d, E_r = %d need a %zu-byte workspace, above the "
          "library's %zu-byte array (use moe_dispatch with a workspace)",
          T, E_r, need, (size_t)MOE_DISPATCH_NOALLOC_MAX_WS);
  if ((r = check_rows16(d, "x", x)) != MOE_OK) return r;
  if ((r = check_rows16(d, "xp", xp)) != MOE_OK) return r;
  return hip_status(moe::launch_dispatch_noalloc(x, dtype == MOE_BF16, T, d, k, E_r, topk_local,
                                                 counts, offsets, perm, inv_perm, xp, stream),
                    "moe_dispatch_noalloc");
}

int moe_dispatch_bwd(const void* dxp, int dtype, int T, int d, int k, int cap,
                     const int32_t* inv_perm, void* dx, int accumulate, hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0 && d >= 1 && k >= 1 && cap >= 0, "bad sizes T = %d, d = %d, k = %d, cap = %d",
          T, d, k, cap);
  REQUIRE(T == 0 || (inv_perm && dx && dxp), "dxp, inv_perm and dx must not be NULL");
  if ((r = check_rows16(d, "dxp", dxp)) != MOE_OK) return r;
  if ((r = check_rows16(d, "dx", dx)) != MOE_OK) return r;
  return hip_status(moe::launch_dispatch_bwd(dxp, dtype == MOE_BF16, T, d, k, cap, inv_perm, dx,
                                             accumulate, stream),
                    "moe_dispatch_bwd");
}

static int check_ffn(int dtype, int cap, int d, int H, int n_groups, const int32_t* offsets) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(cap >= 0 && d >= 1 && H >= 1, "bad sizes cap = %d, d = %d, H = %d", cap, d, H);
  REQUIRE(n_groups >= 0, "n_groups = %d must be >= 0", n_groups);
  SUPPORT(n_groups <= 256, "n_groups = %d: at most 256 groups per set", n_groups);
  REQUIRE(offsets, "offsets must not be NULL");
  SUPPORT(H % 64 == 0, "H = %d must be a multiple of 64", H);
  if (dtype == MOE_BF16) SUPPORT(d % 64 == 0, "d = %d must be a multiple of 64 for bf16", d);
  else SUPPORT(d % 8 == 0, "d = %d must be a multiple of 8", d);
  return MOE_OK;
}

namespace {

int check_set(const moe_ffn_set& f, int dtype, int d, bool fwd) {
  int r;
  if ((r = check_ffn(dtype, f.cap, d, f.H, f.n_groups, f.offsets)) != MOE_OK) return r;
  REQUIRE(f.n_groups == 0 || (f.w_gate_up && f.w_down), "expert weights must not be NULL");
  if (fwd) {
    REQUIRE(f.cap == 0 || (f.xp && f.gu && f.h && f.yp), "xp, gu, h and yp must not be NULL");
  } else {
    REQUIRE(f.n_groups == 0 || (f.dw_gate_up && f.dw_down),
            "the expert weight gradients must not be NULL");
    REQUIRE(f.cap == 0 || (f.dyp && f.xp && f.gu && f.h && f.dgu && f.dxp),
            "dyp, xp, gu, h, dgu and dxp must not be NULL");
  }
  if (dtype == MOE_BF16) {
    // the bf16 GEMMs address each operand with 32-bit byte offsets
    const long rows_bytes = 2L * f.cap * std::max<long>(d, 2L * f.H);
    const long w_bytes = 2L * f.n_groups * 2L * f.H * d;
    // and each expert's fp32 weight gradient (stored with 32-bit offsets)
    const long dw_bytes = 4L * 2L * f.H * d;
    SUPPORT(std::max(std::max(rows_bytes, w_bytes), dw_bytes) < 0xFFFFFFF0L,
            "bf16 expert operands must each stay below 4 GiB (cap = %d, H = %d, groups = %d)",
            f.cap, f.H, f.n_groups);
  }
  for (const void* p : {f.xp, f.w_gate_up, f.w_down, (const void*)f.gu, (const void*)f.h,
                        (const void*)f.yp, f.dyp, (const void*)f.dgu, (const void*)f.dxp,
                        (const void*)f.dw_gate_up, (const void*)f.dw_down})
    SUPPORT(p == nullptr || aligned16(p), "operands must be 16-byte aligned");
  return MOE_OK;
}

int check_sets(const moe_ffn_set* sets, int n_sets, int dtype, int d, bool fwd) {
  REQUIRE(sets != nullptr && n_sets >= 1 && n_sets <= 2, "n_sets = %d must be 1 or 2", n_sets);
  for (int i = 0; i < n_sets; ++i) {
    REQUIRE(sets[i].activation == MOE_ACT_SWIGLU || sets[i].activation == MOE_ACT_SILU,
            "sets[%d].activation = %d is not an expert form", i, sets[i].activation);
    REQUIRE(sets[i].activation == sets[0].activation, "all sets must have the same activation");
  }
  for (int i = 0; i < n_sets; ++i) {
    const int r = check_set(sets[i], dtype, d, fwd);
    if (r != MOE_OK) return r;
  }
  return MOE_OK;
}

}  // namespace

size_t moe_grouped_ffn_fwd_workspace_size(const moe_ffn_set* sets, int n_sets, int dtype, int d) {
  if (!sets || n_sets < 1 || n_sets > 2 || d < 1) return 0;
  return moe::ffn_fwd_ws_bytes(sets, n_sets, dtype == MOE_BF16, d);
}

int moe_grouped_ffn_fwd_sets(const moe_ffn_set* sets, int n_sets, int dtype, int d, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  int r;
  if ((r = check_sets(sets, n_sets, dtype, d, true)) != MOE_OK) return r;
  if (ws) {
    const size_t need = moe::ffn_fwd_ws_bytes(sets, n_sets, dtype == MOE_BF16, d);
    REQUIRE(ws_bytes >= need, "workspace of %zu bytes needed (got %zu)", need, ws_bytes);
    SUPPORT((reinterpret_cast<uintptr_t>(ws) & 255u) == 0, "the workspace must be 256-byte aligned");
    if (need == 0) ws = nullptr;
  }
  return hip_status(moe::launch_ffn_fwd_sets(sets, n_sets, dtype == MOE_BF16, d, ws, stream),
                    "moe_grouped_ffn_fwd_sets");
}

size_t moe_grouped_ffn_bwd_workspace_size(const moe_ffn_set* sets, int n_sets, int dtype, int d) {
  if (!sets || n_sets < 1 || n_sets > 2 || d < 1) return 0;
  return moe::ffn_bwd_ws_bytes(sets, n_sets, dtype == MOE_BF16, d);
}

int moe_grouped_ffn_bwd_sets(const moe_ffn_set* sets, int n_sets, int dtype, int d,
                             int accumulate_dw, void* ws, size_t ws_bytes, hipStream_t stream) {
  int r;
  if ((r = check_sets(sets, n_sets, dtype, d, false)) != MOE_OK) return r;
  if (ws) {
    const size_t need = moe::ffn_bwd_ws_bytes(sets, n_sets, dtype == MOE_BF16, d);
    REQUIRE(ws_bytes >= need, "workspace of %zu bytes needed (got %zu)", need, ws_bytes);
    SUPPORT((reinterpret_cast<uintptr_t>(ws) & 255u) == 0, "the workspace must be 256-byte aligned");
  }
  return hip_status(
      moe::launch_ffn_bwd_sets(sets, n_sets, dtype == MOE_BF16, d, accumulate_dw, ws, stream),
      "moe_grouped_ffn_bwd_sets");
}

int moe_grouped_ffn_fwd(const void* xp, const void* w_gate_up, const void* w_down, int dtype,
                        int cap, int d, int H, int n_groups, const int32_t* offsets, void* gu,
                        void* h, void* yp, hipStream_t stream) {
  moe_ffn_set f{};
  f.xp = xp; f.w_gate_up = w_gate_up; f.w_down = w_down; f.offsets = offsets;
  f.cap = cap; f.H = H; f.n_groups = n_groups;
  f.gu = gu; f.h = h; f.yp = yp;
  return moe_grouped_ffn_fwd_sets(&f, 1, dtype, d, nullptr, 0, stream);
}

int moe_grouped_ffn_bwd(const void* dyp, const void* xp, const void* gu, const void* h,
                        const void* w_gate_up, const void* w_down, int dtype, int cap, int d,
                        int H, int n_groups, const int32_t* offsets, void* dgu, void* dxp,
                        float* dw_gate_up, float* dw_down, int accumulate_dw,
                        hipStream_t stream) {
  moe_ffn_set f{};
  f.xp = xp; f.w_gate_up = w_gate_up; f.w_down = w_down; f.offsets = offsets;
  f.cap = cap; f.H = H; f.n_groups = n_groups;
  f.gu = const_cast<void*>(gu); f.h = const_cast<void*>(h);
  f.dyp = dyp; f.dgu = dgu; f.dxp = dxp; f.dw_gate_up = dw_gate_up; f.dw_down = dw_down;
  return moe_grouped_ffn_bwd_sets(&f, 1, dtype, d, accumulate_dw, nullptr, 0, stream);
}

int moe_combine_fwd(const void* yp, int dtype, int T, int d, int k, int cap, const float* topk_w,
                    const int32_t* inv_perm, const void* y_add, void* y, hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0 && d >= 1 && k >= 1 && cap >= 0, "bad sizes T = %d, d = %d, k = %d, cap = %d",
          T, d, k, cap);
  REQUIRE(T == 0 || (topk_w && inv_perm && y), "topk_w, inv_perm and y must not be NULL");
  if ((r = check_rows16(d, "yp", yp)) != MOE_OK) return r;
  if ((r = check_rows16(d, "y_add", y_add)) != MOE_OK) return r;
  if ((r = check_rows16(d, "y", y)) != MOE_OK) return r;
  return hip_status(moe::launch_combine_fwd(yp, dtype == MOE_BF16, T, d, k, cap, topk_w, inv_perm,
                                            y_add, y, stream),
                    "moe_combine_fwd");
}

int moe_combine_bwd(const void* dy, const void* yp, int dtype, int T, int d, int k, int cap,
                    const float* topk_w, const int32_t* inv_perm, void* dyp, float* d_topk_w,
                    hipStream_t stream) {
  int r;
  if ((r = check_dtype(dtype)) != MOE_OK) return r;
  REQUIRE(T >= 0 && d >= 1 && k >= 1 && cap >= 0, "bad sizes T = %d, d = %d, k = %d, cap = %d",
          T, d, k, cap);
  REQUIRE(T == 0 || (dy && topk_w && inv_perm && d_topk_w), "dy, topk_w, inv_perm and d_topk_w must not be NULL");
  if ((r = check_rows16(d, "dy", dy)) != MOE_OK) return r;
  if ((r = check_rows16(d, "yp", yp)) != MOE_OK) return r;
  if ((r = check_rows16(d, "dyp", dyp)) != MOE_OK) return r;
  return hip_status(moe::launch_combine_bwd(dy, yp, dtype == MOE_BF16, T, d, k, cap, topk_w,
                                            inv_perm, dyp, d_topk_w, stream),
                    "moe_combine_bwd");
}

int moe_expert_delta(const float* theta_start, const float* theta_now,
                     const float* const* peers, int n_peers, size_t n_params, float* delta_local,
                     float* delta_avg, hipStream_t stream) {
  REQUIRE(n_peers >= 0 && n_peers <= moe::kMaxPeers, "n_peers = %d must be in [0, %d]", n_peers,
          moe::kMaxPeers);
  REQUIRE(n_params == 0 || (theta_start && theta_now && delta_avg),
          "theta_start, theta_now and delta_avg must not be NULL");
  REQUIRE(n_peers == 0 || peers, "peers must not be NULL when n_peers > 0");
  for (int p = 0; p < n_peers; ++p) {
    REQUIRE(n_params == 0 || peers[p], "peers[%d] must not be NULL", p);
    SUPPORT(peers[p] == nullptr || aligned16(peers[p]), "peers[%d] must be 16-byte aligned", p);
  }
  for (const void* p : {(const void*)theta_start, (const void*)theta_now, (const void*)delta_local,
                        (const void*)delta_avg})
    SUPPORT(p == nullptr || aligned16(p), "arrays must be 16-byte aligned");
  return hip_status(moe::launch_expert_delta(theta_start, theta_now, peers, n_peers, n_params,
                                             delta_local, delta_avg, stream),
                    "moe_expert_delta");
}

int moe_adamw_step(float* theta, const float* grad, float* m, float* v, size_t n, int step,
                   float lr, float beta1, float beta2, float eps, float weight_decay,
                   void* theta_bf16, hipStream_t stream) {
  REQUIRE(n == 0 || (theta && grad && m && v), "theta, grad, m and v must not be NULL");
  REQUIRE(step >= 1, "step = %d must be >= 1", step);
  REQUIRE(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f && eps >= 0.f,
          "betas must lie in [0, 1) and eps must be >= 0");
  for (const void* p : {(const void*)theta, (const void*)grad, (const void*)m, (const void*)v,
                        (const void*)theta_bf16})
    SUPPORT(p == nullptr || aligned16(p), "arrays must be 16-byte aligned");
  const float c1 = (float)(1.0 - std::pow((double)beta1, (double)step));
  const float c2 = (float)(1.0 - std::pow((double)beta2, (double)step));
  REQUIRE(c1 > 0.f && c2 > 0.f, "bias corrections must be positive (betas > 0 at step %d)", step);
  return hip_status(moe::launch_adamw(theta, grad, m, v, n, lr, beta1, beta2, eps, weight_decay,
                                      c1, c2, theta_bf16, stream),
                    "moe_adamw_step");
}

int moe_outer_nesterov(float* theta_start, float* theta_now, const float* delta_avg,
                       float* momentum, size_t n, float lr, float mu, void* theta_bf16,
                       hipStream_t stream) {
  REQUIRE(n == 0 || (theta_start && theta_now && delta_avg && momentum),
          "theta_start, theta_now, delta_avg and momentum must not be NULL");
  for (const void* p : {(const void*)theta_start, (const void*)theta_now,
                        (const void*)delta_avg, (const void*)momentum, (const void*)theta_bf16})
    SUPPORT(p == nullptr || aligned16(p), "arrays must be 16-byte aligned");
  return hip_status(moe::launch_outer_nesterov(theta_start, theta_now, delta_avg, momentum, n, lr,
                                               mu, theta_bf16, stream),
                    "moe_outer_nesterov");
}

int moe_replica_mean(const float* local, const float* const* peers, int n_peers, size_t n,
                     float* out, hipStream_t stream) {
  REQUIRE(n_peers >= 0 && n_peers <= moe::kMaxPeers, "n_peers = %d must be in [0, %d]", n_peers,
          moe::kMaxPeers);
  REQUIRE(n == 0 || (local && out), "local and out must not be NULL");
  REQUIRE(n_peers == 0 || peers, "peers must not be NULL when n_peers > 0");
  for (int p = 0; p < n_peers; ++p) {
    REQUIRE(n == 0 || peers[p], "peers[%d] must not be NULL", p);
    SUPPORT(peers[p] == nullptr || aligned16(peers[p]), "peers[%d] must be 16-byte aligned", p);
  }
  SUPPORT((local == nullptr || aligned16(local)) && (out == nullptr || aligned16(out)),
          "arrays must be 16-byte aligned");
  return hip_status(moe::launch_replica_mean(local, peers, n_peers, n, out, stream),
                    "moe_replica_mean");
}

static bool is_permutation(const int32_t* p, int n) {
  if (!p) return true;
  std::vector<char> seen(n, 0);
  for (int i = 0; i < n; ++i) {
    if (p[i] < 0 || p[i] >= n || seen[p[i]]) return false;
    seen[p[i]] = 1;
  }
  return true;
}

int moe_gen_placement(int N_e, int O_e, int M, const int32_t* expert_perm,
                      const int32_t* worker_perm, int32_t* sets) {
  REQUIRE(sets, "sets must not be NULL");
  REQUIRE(N_e >= 1 && M >= 1 && O_e >= 1 && O_e <= M,
          "need N_e >= 1 and 1 <= O_e <= M (N_e = %d, O_e = %d, M = %d)", N_e, O_e, M);
  REQUIRE(((long)N_e * O_e) % M == 0, "M = %d must divide N_e O_e = %ld", M, (long)N_e * O_e);
  REQUIRE(is_permutation(expert_perm, N_e), "expert_perm is not a permutation of 0..N_e-1");
  REQUIRE(is_permutation(worker_perm, M), "worker_perm is not a permutation of 0..M-1");
  REQUIRE(moe::gen_placement(N_e, O_e, M, expert_perm, worker_perm, sets), "placement failed");
  return MOE_OK;
}

int moe_migration_map(const int32_t* prev_set, int n_prev, const int32_t* new_set, int n_new,
                      int32_t* map) {
  REQUIRE(n_prev >= 0 && n_new >= 0, "set sizes must be >= 0");
  REQUIRE((n_prev == 0 || prev_set) && (n_new == 0 || (new_set && map)),
          "sets and map must not be NULL");
  for (int i = 0; i < n_new; ++i) {
    REQUIRE(i == 0 || new_set[i] > new_set[i - 1], "new_set must be strictly ascending");
    map[i] = -1;
    for (int j = 0; j < n_prev; ++j)
      if (prev_set[j] == new_set[i]) map[i] = j;
  }
  return MOE_OK;
}

int moe_copy_expert_rows(const float* src, const int32_t* src_row, float* dst,
                         const int32_t* dst_row, int n_rows, size_t row_len, void* dst_bf16,
                         hipStream_t stream) {
  REQUIRE(n_rows >= 0 && n_rows <= 256, "n_rows = %d must be in [0, 256]", n_rows);
  REQUIRE(n_rows == 0 || row_len == 0 || (src_row && dst), "src_row and dst must not be NULL");
  bool any_src = false;
  for (int r = 0; r < n_rows; ++r) {
    any_src = any_src || src_row[r] >= 0;
    REQUIRE(src_row[r] >= -1, "src_row[%d] = %d must be >= -1", r, src_row[r]);
    if (dst_row) {
      REQUIRE(dst_row[r] >= 0, "dst_row[%d] = %d must be >= 0", r, dst_row[r]);
      for (int q = 0; q < r; ++q) REQUIRE(dst_row[q] != dst_row[r], "dst_row repeats %d", dst_row[r]);
    }
  }
  REQUIRE(!any_src || src, "src must not be NULL when a row is copied");
  SUPPORT((!src || aligned16(src)) && (!dst || aligned16(dst)) &&
              (!dst_bf16 || aligned16(dst_bf16)) && row_len % 4 == 0,
          "src, dst and dst_bf16 must be 16-byte aligned and row_len a multiple of 4");
  return hip_status(moe::launch_copy_expert_rows(src, src_row, dst, dst_row, n_rows, row_len,
                                                 dst_bf16, stream),
                    "moe_copy_expert_rows");
}

int moe_warmup_lr(const int* steps, int n_rows, double lr, int warmup_steps, float* lr_out) {
  REQUIRE(n_rows >= 0, "n_rows = %d must be >= 0", n_rows);
  REQUIRE(n_rows == 0 || (steps && lr_out), "steps and lr_out must not be NULL");
  REQUIRE(std::isfinite(lr), "lr must be finite");
  for (int r = 0; r < n_rows; ++r) REQUIRE(steps[r] >= 0, "steps[%d] = %d must be >= 0", r, steps[r]);
  for (int r = 0; r < n_rows; ++r) {
    const double f = warmup_steps > 0 ? std::min(1.0, (double)steps[r] / (double)warmup_steps) : 1.0;
    lr_out[r] = (float)(lr * f);
  }
  return MOE_OK;
}

int moe_adamw_step_rows(float* theta, const float* grad, float* m, float* v, int n_rows,
                        size_t row_len, const int* steps, const float* lr, float beta1,
                        float beta2, float eps, float weight_decay, void* theta_bf16,
                        hipStream_t stream) {
  REQUIRE(n_rows >= 0 && (n_rows == 0 || (steps && lr)), "steps and lr must not be NULL");
  REQUIRE(n_rows == 0 || row_len == 0 || (theta && grad && m && v),
          "theta, grad, m and v must not be NULL");
  REQUIRE(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f && eps >= 0.f,
          "betas must lie in [0, 1) and eps must be >= 0");
  SUPPORT(row_len % 4 == 0, "row_len must be a multiple of 4");
  for (const void* p : {(const void*)theta, (const void*)grad, (const void*)m, (const void*)v,
                        (const void*)theta_bf16})
    SUPPORT(p == nullptr || aligned16(p), "arrays must be 16-byte aligned");
  for (int r = 0; r < n_rows; ++r) REQUIRE(steps[r] >= 1, "steps[%d] = %d must be >= 1", r, steps[r]);
  // one launch per run of rows that share (step, lr)
  for (int r0 = 0; r0 < n_rows;) {
    int r1 = r0 + 1;
    while (r1 < n_rows && steps[r1] == steps[r0] && lr[r1] == lr[r0]) ++r1;
    const float c1 = (float)(1.0 - std::pow((double)beta1, (double)steps[r0]));
    const float c2 = (float)(1.0 - std::pow((double)beta2, (double)steps[r0]));
    REQUIRE(c1 > 0.f && c2 > 0.f, "bias corrections must be positive");
    const size_t o = (size_t)r0 * row_len, n = (size_t)(r1 - r0) * row_len;
    void* lp = theta_bf16 ? static_cast<uint16_t*>(theta_bf16) + o : nullptr;  // bf16 elements
    const int st = hip_status(moe::launch_adamw(theta + o, grad + o, m + o, v + o, n, lr[r0],
                                                beta1, beta2, eps, weight_decay, c1, c2, lp,
                                                stream),
                              "moe_adamw_step_rows");
    if (st != MOE_OK) return st;
    r0 = r1;
  }
  return MOE_OK;
}

}  // extern "C"
