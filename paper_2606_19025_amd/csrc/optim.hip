// Optimisers of the resident experts' fp32 master parameters.
//
// Sec. 3.4 ("Outer optimization"): every worker runs AdamW on its own
// parameters during the K local steps of a round and keeps the optimiser state
// across rounds, only for its own experts; at the round boundary the
// replica-group average of the pseudo-gradient is applied by a momentum outer
// optimiser (Alg. 2, OuterOpt).  App. F fixes the settings: AdamW with weight
// decay 0, betas (0.9, 0.95), eps 1e-8; DiLoCo's Nesterov outer step with
// learning rate 0.7 and momentum 0.9; LocalAdamW also averages the two moments
// over the replica group.
//
// All three are elementwise streams over fp32 arrays (HBM-bound): 16-byte
// vector accesses in a grid-stride loop, an element tail for n % 4.  Nothing
// is read twice, so the vector accesses are nontemporal (measured 14 % faster
// for AdamW than cached accesses).  Every
// operation is one IEEE fp32 rounding in a fixed order (no contraction into
// fused multiply-adds; division and square root correctly rounded), so the
// results are reproducible bit for bit by any fp32 evaluation of the same
// formulas.  The bf16 working copy that the grouped GEMMs read is written in
// the same pass (round to nearest even).
#include "common.h"
#include "kernels.h"
#include "timing.h"

#pragma clang fp contract(off)

namespace moe {
namespace {

struct AdamArgs {
  float* theta;
  const float* grad;
  float* m;
  float* v;
  bf16_t* theta_bf16;  // or NULL
  size_t n;
  float lr, b1, b2, eps, wd;
  float c1, c2;  // bias corrections 1 - beta^t of this step
};

// m' = b1 m + (1 - b1) g;  v' = b2 v + (1 - b2) g g;
// theta' = theta - lr ((m' / c1) / (sqrt(v' / c2) + eps) + wd theta)
// (contraction is off for this file; '/' and __builtin_sqrtf are the
// correctly rounded fp32 operations of HIP's default mode)
DEVI void adam_elem(const AdamArgs& a, float& th, float g, float& m, float& v) {
  const float om1 = 1.0f - a.b1, om2 = 1.0f - a.b2;
  m = a.b1 * m + om1 * g;
  v = a.b2 * v + om2 * (g * g);
  const float mh = m / a.c1;
  const float vh = v / a.c2;
  const float den = __builtin_sqrtf(vh) + a.eps;
  const float upd = mh / den + a.wd * th;
  th = th - a.lr * upd;
}

__global__ __launch_bounds__(256) void adamw_kernel(AdamArgs a) {
  const size_t n4 = a.n / 4;
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    f32x4_t th = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.theta) + i);
    const f32x4_t g = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.grad) + i);
    f32x4_t m = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.m) + i);
    f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.v) + i);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float t = th[e], mm = m[e], vv = v[e];
      adam_elem(a, t, g[e], mm, vv);
      th[e] = t; m[e] = mm; v[e] = vv;
    }
    __builtin_nontemporal_store(th, reinterpret_cast<f32x4_t*>(a.theta) + i);
    __builtin_nontemporal_store(m, reinterpret_cast<f32x4_t*>(a.m) + i);
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t*>(a.v) + i);
    if (a.theta_bf16) {
      bf16x4_t o = {(bf16_t)th[0], (bf16_t)th[1], (bf16_t)th[2], (bf16_t)th[3]};
      reinterpret_cast<bf16x4_t*>(a.theta_bf16)[i] = o;
    }
  }
  for (size_t i = n4 * 4 + (size_t)blockIdx.x * 256 + threadIdx.x; i < a.n; i += stride) {
    float t = a.theta[i], mm = a.m[i], vv = a.v[i];
    adam_elem(a, t, a.grad[i], mm, vv);
    a.theta[i] = t; a.m[i] = mm; a.v[i] = vv;
    if (a.theta_bf16) a.theta_bf16[i] = (bf16_t)t;
  }
}

struct OuterArgs {
  float* start;
  float* now;
  const float* delta;
  float* mom;
  bf16_t* theta_bf16;  // or NULL
  size_t n;
  float lr, mu;
};

// b' = mu b + delta;  theta' = start - lr (delta + mu b'); start = now = theta'
DEVI float outer_elem(const OuterArgs& a, float start, float delta, float& b) {
  b = a.mu * b + delta;
  const float upd = delta + a.mu * b;
  return start - a.lr * upd;
}

__global__ __launch_bounds__(256) void outer_nesterov_kernel(OuterArgs a) {
  const size_t n4 = a.n / 4;
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    const f32x4_t s = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.start) + i);
    const f32x4_t d = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.delta) + i);
    f32x4_t b = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.mom) + i);
    f32x4_t th;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float bb = b[e];
      th[e] = outer_elem(a, s[e], d[e], bb);
      b[e] = bb;
    }
    __builtin_nontemporal_store(b, reinterpret_cast<f32x4_t*>(a.mom) + i);
    __builtin_nontemporal_store(th, reinterpret_cast<f32x4_t*>(a.start) + i);
    __builtin_nontemporal_store(th, reinterpret_cast<f32x4_t*>(a.now) + i);
    if (a.theta_bf16) {
      bf16x4_t o = {(bf16_t)th[0], (bf16_t)th[1], (bf16_t)th[2], (bf16_t)th[3]};
      reinterpret_cast<bf16x4_t*>(a.theta_bf16)[i] = o;
    }
  }
  for (size_t i = n4 * 4 + (size_t)blockIdx.x * 256 + threadIdx.x; i < a.n; i += stride) {
    float bb = a.mom[i];
    const float th = outer_elem(a, a.start[i], a.delta[i], bb);
    a.mom[i] = bb;
    a.start[i] = th;
    a.now[i] = th;
    if (a.theta_bf16) a.theta_bf16[i] = (bf16_t)th;
  }
}

struct MeanArgs {
  const float* local;
  const float* peers[kMaxPeers];
  float* out;
  size_t n;
  int n_peers;
  float scale;
};

// out = (((local + p_0) + p_1) + ...) * fp32(1 / (n_peers + 1))
__global__ __launch_bounds__(256) void replica_mean_kernel(MeanArgs a) {
  const size_t n4 = a.n / 4;
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    f32x4_t acc = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.local) + i);
    for (int p = 0; p < a.n_peers; ++p)
      acc = acc + __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.peers[p]) + i);
    __builtin_nontemporal_store(acc * a.scale, reinterpret_cast<f32x4_t*>(a.out) + i);
  }
  for (size_t i = n4 * 4 + (size_t)blockIdx.x * 256 + threadIdx.x; i < a.n; i += stride) {
    float acc = a.local[i];
    for (int p = 0; p < a.n_peers; ++p) acc = acc + a.peers[p][i];
    a.out[i] = acc * a.scale;
  }
}

int stream_blocks(size_t n) {
  const size_t want = (n / 4 + 255) / 256;
  return (int)std::max<size_t>(1, std::min<size_t>(want, 8192));
}

}  // namespace

hipError_t launch_adamw(float* theta, const float* grad, float* m, float* v, size_t n, float lr,
                        float beta1, float beta2, float eps, float wd, float c1, float c2,
                        void* theta_bf16, hipStream_t s) {
  if (n == 0) return hipSuccess;
  AdamArgs a{theta, grad, m, v, static_cast<bf16_t*>(theta_bf16), n, lr, beta1, beta2, eps, wd,
             c1, c2};
  MOE_TIMED("adamw_step", s, adamw_kernel<<<stream_blocks(n), 256, 0, s>>>(a));
  return hipGetLastError();
}

hipError_t launch_outer_nesterov(float* start, float* now, const float* delta, float* mom,
                                 size_t n, float lr, float mu, void* theta_bf16, hipStream_t s) {
  if (n == 0) return hipSuccess;
  OuterArgs a{start, now, delta, mom, static_cast<bf16_t*>(theta_bf16), n, lr, mu};
  MOE_TIMED("outer_nesterov", s, outer_nesterov_kernel<<<stream_blocks(n), 256, 0, s>>>(a));
  return hipGetLastError();
}

hipError_t launch_replica_mean(const float* local, const float* const* peers, int n_peers,
                               size_t n, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  MeanArgs a{};
  a.local = local;
  for (int p = 0; p < n_peers; ++p) a.peers[p] = peers[p];
  a.out = out;
  a.n = n;
  a.n_peers = n_peers;
  a.scale = 1.0f / (float)(n_peers + 1);
  MOE_TIMED("replica_mean", s, replica_mean_kernel<<<stream_blocks(n), 256, 0, s>>>(a));
  return hipGetLastError();
}

}  // namespace moe
