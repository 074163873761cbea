// Dispatch of the resident routes, its backward, the weighted combine and its
// backward.
//
// Routing is strictly local (Sec. 3.3.2 "System context and routing logic"):
// a route is either executed by one of the worker's resident experts or, for a
// ghost expert, skipped (Sec. 3.3 "Ghost Experts and Skip-Token").  The
// dispatch is a stable counting sort of the routes by local expert id:
//   1. per 256-token block, an LDS histogram of local ids;
//   2. one block scans the histograms (expert-major, then block) into the
//      global offsets and per-block bases;
//   3. per block, an LDS bitmap [expert][token] gives every route its rank
//      among earlier tokens of the same expert (popcount), hence its slot;
//   4. the rows are gathered token-major: each wave reads a token row once and
//      writes it to every slot of that token (16-byte vector accesses).
// Combine, combine backward and un-permute are token-major too: one wave per
// token, 16-byte loads of the routed rows, fp32 accumulation.
#include <mutex>

#include "common.h"
#include "kernels.h"
#include "timing.h"

// Workspace of the allocation-free dispatch (moe_dispatch_noalloc): a
// file-scope device array, one copy per device, whose device address is
// resolved once per device with that device current (dispatch_scratch).  In
// host code the array's name is a host-side stand-in, so only the resolved
// address is ever passed to a kernel.  The counting sort overwrites every word
// it reads (per-block histograms, then bases), so the array needs no clearing
// between calls; calls that overlap on one device share it and race.
// External linkage on purpose: a static array is a LOCAL symbol of the device
// code object, which the runtime's lookup by name (hipGetSymbolAddress) does
// not find.
__device__ __attribute__((aligned(256))) char moe_dispatch_scratch[MOE_DISPATCH_NOALLOC_MAX_WS];

namespace moe {
namespace {

constexpr int DB = 256;  // tokens per block of the counting sort

__global__ __launch_bounds__(DB) void dispatch_count_kernel(const int32_t* local, int T, int k,
                                                            int E_r, int32_t* blk_counts) {
  __shared__ int hist[256];
  for (int r = threadIdx.x; r < E_r; r += DB) hist[r] = 0;
  __syncthreads();
  const int t = blockIdx.x * DB + threadIdx.x;
  if (t < T) {
    for (int j = 0; j < k; ++j) {
      const int r = local[(size_t)t * k + j];
      if (r >= 0 && r < E_r) atomicAdd(&hist[r], 1);
    }
  }
  __syncthreads();
  for (int r = threadIdx.x; r < E_r; r += DB) blk_counts[(size_t)blockIdx.x * E_r + r] = hist[r];
}

// Inclusive prefix sum over the 64 lanes of a wave.
DEVI int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

// One block of 16 waves: wave w scans experts w, w + 16, ... over the
// counting blocks (blk_base[b][r] = offsets[r] + sum_{b'<b} cnt[b'][r]); then
// wave 0 scans the expert totals into counts and offsets.
constexpr int SCAN_WAVES = 16;
__global__ __launch_bounds__(64 * SCAN_WAVES) void dispatch_scan_kernel(const int32_t* blk_counts,
                                                                       int nblk, int E_r,
                                                                       int32_t* blk_base,
                                                                       int32_t* counts,
                                                                       int32_t* offsets) {
  __shared__ int tot[256];
  __shared__ int base[256];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int r = wave; r < E_r; r += SCAN_WAVES) {
    int carry = 0;
    for (int b0 = 0; b0 < nblk; b0 += 64) {
      const int b = b0 + lane;
      const int c = b < nblk ? blk_counts[(size_t)b * E_r + r] : 0;
      const int inc = wave_inclusive_scan(c);
      if (b < nblk) blk_base[(size_t)b * E_r + r] = carry + inc - c;  // relative, fixed below
      carry += __shfl(inc, 63, 64);
    }
    if (lane == 0) tot[r] = carry;
  }
  __syncthreads();
  if (wave == 0) {
    int carry = 0;
    for (int r0 = 0; r0 < E_r; r0 += 64) {
      const int r = r0 + lane;
      const int c = r < E_r ? tot[r] : 0;
      const int inc = wave_inclusive_scan(c);
      if (r < E_r) {
        base[r] = carry + inc - c;
        counts[r] = c;
        offsets[r] = carry + inc - c;
      }
      carry += __shfl(inc, 63, 64);
    }
    if (lane == 0) offsets[E_r] = carry;
  }
  __syncthreads();
  for (int r = wave; r < E_r; r += SCAN_WAVES)
    for (int b = lane; b < nblk; b += 64) blk_base[(size_t)b * E_r + r] += base[r];
}

__global__ __launch_bounds__(DB) void dispatch_scatter_kernel(const int32_t* local, int T, int k,
                                                              int E_r, int cap,
                                                              const int32_t* blk_base,
                                                              int32_t* perm, int32_t* inv_perm) {
  __shared__ uint32_t bits[256][DB / 32];
  for (int i = threadIdx.x; i < E_r * (DB / 32); i += DB) bits[i / (DB / 32)][i % (DB / 32)] = 0;
  __syncthreads();
  const int t = blockIdx.x * DB + threadIdx.x;
  const int word = threadIdx.x >> 5, bit = threadIdx.x & 31;
  if (t < T) {
    for (int j = 0; j < k; ++j) {
      const int r = local[(size_t)t * k + j];
      if (r >= 0 && r < E_r) atomicOr(&bits[r][word], 1u << bit);
    }
  }
  __syncthreads();
  if (t < T) {
    for (int j = 0; j < k; ++j) {
      const int r = local[(size_t)t * k + j];
      const size_t o = (size_t)t * k + j;
      if (r >= 0 && r < E_r) {
        int rank = __popc(bits[r][word] & ((1u << bit) - 1u));
        for (int w = 0; w < word; ++w) rank += __popc(bits[r][w]);
        const int p = blk_base[(size_t)blockIdx.x * E_r + r] + rank;
        // p < cap whenever a token's routes name distinct experts; anything
        // else is malformed input and its extra routes are dropped
        if (p < cap) perm[p] = (int32_t)o;
        inv_perm[o] = p < cap ? p : -1;
      } else {
        inv_perm[o] = -1;
      }
    }
  }
}

// The resident routes of token t (o = t*k) in route order: up to KR of them
// as wave-uniform (slot, weight) pairs; slots outside [0, cap) count as ghost
// routes.  Routes past the KR-th resident one (k > KR) are handled by the
// callers' generic loop, using slot_of.
constexpr int KR = 8;

DEVI int slot_of(const int32_t* inv_perm, size_t o, int j, int cap) {
  const int p = inv_perm[o + j];
  return (p >= 0 && p < cap) ? p : -1;
}

// Returns the number of resident routes n (all k routes scanned when k <= 64);
// fills p[0..min(n, KR)) and w[...] (weights from tw, or 1 when tw is NULL).
// j_rest receives the route index after the KR-th resident route (k if none).
DEVI int token_routes(const int32_t* inv_perm, const float* tw, size_t o, int k, int cap, int* p,
                      float* w, int& j_rest) {
  const int lane = threadIdx.x & 63;
  int n = 0;
  j_rest = k;
  for (int j0 = 0; j0 < k; j0 += 64) {
    const int j = j0 + lane;
    int pj = -1;
    float wj = 1.f;
    if (j < k) {
      pj = slot_of(inv_perm, o, j, cap);
      if (tw) wj = tw[o + j];
    }
    uint64_t m = __ballot(pj >= 0);
    while (m) {
      const int src = __builtin_ctzll(m);
      m &= m - 1;
      if (n < KR) {
        p[n] = __shfl(pj, src, 64);
        w[n] = __shfl(wj, src, 64);
      } else if (n == KR) {
        j_rest = j0 + src;
      }
      ++n;
    }
    if (n > KR) break;
  }
  return n;
}

// Columns of a row handled per lane and pass: CPL chunks of 16 bytes, lanes
// interleaved (chunk cc of lane l is element (cc * 64 + l) * V).
constexpr int CPL = 4;

template <class T>
__global__ __launch_bounds__(256) void gather_rows_kernel(const T* x, int T_, int d, int k, int cap,
                                                          const int32_t* inv_perm, T* xp) {
  constexpr int V = Vec16<T>::N;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;
  const size_t o = (size_t)t * k;
  int p[KR];
  float w[KR];
  int j_rest;
  const int n = token_routes(inv_perm, nullptr, o, k, cap, p, w, j_rest);
  if (n == 0) return;
  const int nr = min(n, KR);
  for (int c0 = 0; c0 < d; c0 += CPL * 64 * V) {
    u32x4_t v[CPL];
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int c = c0 + (cc * 64 + lane) * V;
      if (c < d) v[cc] = *reinterpret_cast<const u32x4_t*>(x + (size_t)t * d + c);
    }
#pragma unroll
    for (int s = 0; s < KR; ++s) {
      if (s >= nr) break;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int c = c0 + (cc * 64 + lane) * V;
        if (c < d) *reinterpret_cast<u32x4_t*>(xp + (size_t)p[s] * d + c) = v[cc];
      }
    }
    for (int j = j_rest; j < k; ++j) {  // resident routes beyond the first KR
      const int q = slot_of(inv_perm, o, j, cap);
      if (q < 0) continue;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int c = c0 + (cc * 64 + lane) * V;
        if (c < d) *reinterpret_cast<u32x4_t*>(xp + (size_t)q * d + c) = v[cc];
      }
    }
  }
}

// Scan, slot assignment and gather in one kernel (k <= PK): block = PB
// tokens.  Its slots follow from the per-DB-token-block histograms: for local
// expert r, base = offsets[r] (exclusive scan of the totals) + the routes to r
// of the DB-blocks before its own + those of the tokens before it in its own
// DB-block (counted here) + the rank among the block's tokens (bitmap
// popcount).  The x rows are requested before any of that, so their latency
// overlaps the scan; each wave then writes its tokens' rows to their slots.
// Block 0 writes counts and offsets.
constexpr int PB = 32;  // tokens per block (one bitmap word per expert)
constexpr int PK = 8;   // routes per token handled here
template <class T>
__global__ __launch_bounds__(256) void dispatch_place_kernel(const T* x, const int32_t* local, int Tn,
                                                             int d, int k, int E_r, int cap,
                                                             int nblk, const int32_t* blk_counts,
                                                             int32_t* counts, int32_t* offsets,
                                                             int32_t* perm, int32_t* inv_perm,
                                                             T* xp) {
  constexpr int V = Vec16<T>::N;
  __shared__ int base[256];
  __shared__ int wsum[4];
  __shared__ uint32_t bits[256];
  __shared__ int slot[PB][PK];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * PB;
  const int B = t0 / DB;  // counting block of these tokens
  // this wave's tokens' rows (4 tokens per wave, CPL chunks of 16 bytes per
  // lane per pass; rows longer than one pass are handled by the loop below)
  constexpr int TPW = PB / 4;  // tokens per wave
  static_assert(TPW * 4 == PB, "tokens per wave");
  const int pass = CPL * 64 * V;  // elements per pass
  u32x4_t row[TPW][CPL];
  auto load_rows = [&](int c0) {
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const int t = t0 + wave * TPW + i;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int c = c0 + (cc * 64 + lane) * V;
        if (t < Tn && c < d) row[i][cc] = *reinterpret_cast<const u32x4_t*>(x + (size_t)t * d + c);
      }
    }
  };
  if (E_r > 0) load_rows(0);
  // per-expert totals and the routes of the DB-blocks before B
  int tot = 0, pre = 0;
  if (tid < E_r) {
    int b = 0;
    for (; b + 8 <= nblk; b += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = blk_counts[(size_t)(b + u) * E_r + tid];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        tot += v[u];
        if (b + u < B) pre += v[u];
      }
    }
    for (; b < nblk; ++b) {
      const int v = blk_counts[(size_t)b * E_r + tid];
      tot += v;
      if (b < B) pre += v;
    }
    bits[tid] = 0u;
  }
  // exclusive scan of the totals over the experts (4 waves of 64)
  int inc = tot;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(inc, o, 64);
    if (lane >= o) inc += u;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int carry = 0;
  for (int w = 0; w < wave; ++w) carry += wsum[w];
  const int off = carry + inc - tot;
  if (tid < E_r) {
    base[tid] = off + pre;
    if (blockIdx.x == 0) {
      counts[tid] = tot;
      offsets[tid] = off;
    }
  }
  if (blockIdx.x == 0 && tid == 0) offsets[E_r] = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  // routes of the tokens of B before this block
  for (int q = B * DB * k + tid; q < t0 * k; q += 256) {
    const int r = local[q];
    if (r >= 0 && r < E_r) atomicAdd(&base[r], 1);
  }
  // bitmaps of this block's tokens
  const int i = tid >> 3, jl = tid & 7;  // token, route
  const int t = t0 + i;
  int r = -1;
  if (t < Tn && jl < k) {
    r = local[(size_t)t * k + jl];
    if (r >= 0 && r < E_r) atomicOr(&bits[r], 1u << i);
  }
  __syncthreads();
  if (t < Tn && jl < k) {
    const size_t o = (size_t)t * k + jl;
    int p = -1;
    if (r >= 0 && r < E_r) {
      p = base[r] + __popc(bits[r] & ((1u << i) - 1u));
      // p < cap whenever a token's routes name distinct experts; anything
      // else is malformed input and its extra routes are dropped
      if (p < cap) perm[p] = (int32_t)o; else p = -1;
    }
    inv_perm[o] = p;
    slot[i][jl] = p;
  }
  __syncthreads();
  if (E_r == 0) return;
  // each wave writes its tokens' rows to their slots
  for (int c0 = 0; c0 < d; c0 += pass) {
    if (c0 > 0) load_rows(c0);
#pragma unroll
    for (int ii = 0; ii < TPW; ++ii) {
      const int ti = wave * TPW + ii;
      if (t0 + ti >= Tn) break;
      for (int j = 0; j < k; ++j) {
        const int pj = slot[ti][j];
        if (pj < 0) continue;
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          const int c = c0 + (cc * 64 + lane) * V;
          if (c < d) *reinterpret_cast<u32x4_t*>(xp + (size_t)pj * d + c) = row[ii][cc];
        }
      }
    }
  }
}

// 16 bytes of T held as raw words, widened to fp32 (exact).
DEVI void unpack16_f32(const u32x4_t& r, float* out, const float*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(r[i]);
}
DEVI void unpack16_f32(const u32x4_t& r, float* out, const bf16_t*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(r[i] << 16);
    out[2 * i + 1] = __uint_as_float(r[i] & 0xffff0000u);
  }
}

// Routes whose rows are requested together, before any of them is summed,
// and 16-byte chunks per lane and column pass of the weighted row sums: a
// d = 2048 bf16 row in one pass, two routes at a time (measured against 2
// chunks x 4 routes: combine_fwd 3 % faster warm, 6 % cold; 1 chunk or 4
// routes were slower).
constexpr int RB = 2;
constexpr int WCPL = 4;

// y[t] = sum over resident routes (in route order) of w * rows[slot] (+ add[t]);
// combine forward (weights tw, add = shared output) and un-permute (tw NULL,
// add = dx when accumulating, out = dx).  Per column pass, the add chunks and
// the rows of up to RB routes are loaded before the first is used, so a token
// costs one memory round trip per pass rather than one per route; the sums
// keep the route order.  A separate add row is requested before the route
// lookup; in place (add == out), a token without resident routes is left as
// it is.
template <class T, bool STREAM_ROWS>
DEVI void weighted_row_sum(const T* rows, int T_, int d, int k, int cap, const float* tw,
                           const int32_t* inv_perm, const T* add, T* out) {
  constexpr int V = Vec16<T>::N;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;
  const size_t o = (size_t)t * k;
  const bool in_place = add == out;
  const T* add_row = add ? add + (size_t)t * d : nullptr;
  u32x4_t a_raw[WCPL];
  auto load_add = [&](int c0) {
#pragma unroll
    for (int cc = 0; cc < WCPL; ++cc) {
      const int c = c0 + (cc * 64 + lane) * V;
      if (c < d) a_raw[cc] = *reinterpret_cast<const u32x4_t*>(add_row + c);
    }
  };
  const bool early_add = add && !in_place;
  if (early_add) load_add(0);
  int p[KR];
  float w[KR];
  int j_rest;
  const int n = token_routes(inv_perm, tw, o, k, cap, p, w, j_rest);
  if (n == 0 && in_place) return;
  const int nr = min(n, KR);
  for (int c0 = 0; c0 < d; c0 += WCPL * 64 * V) {
    if (add && (c0 > 0 || !early_add)) load_add(c0);
    float acc[WCPL][V];
#pragma unroll
    for (int cc = 0; cc < WCPL; ++cc)
#pragma unroll
      for (int u = 0; u < V; ++u) acc[cc][u] = 0.f;
#pragma unroll
    for (int s0 = 0; s0 < KR; s0 += RB) {
      if (s0 >= nr) break;
      u32x4_t raw[RB][WCPL];
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        if (s0 + b >= nr) continue;
#pragma unroll
        for (int cc = 0; cc < WCPL; ++cc) {
          const int c = c0 + (cc * 64 + lane) * V;
          if (c < d) {
            const u32x4_t* src = reinterpret_cast<const u32x4_t*>(rows + (size_t)p[s0 + b] * d + c);
            raw[b][cc] = STREAM_ROWS ? __builtin_nontemporal_load(src) : *src;
          }
        }
      }
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        if (s0 + b >= nr) continue;
#pragma unroll
        for (int cc = 0; cc < WCPL; ++cc) {
          float v[V];
          unpack16_f32(raw[b][cc], v, rows);
#pragma unroll
          for (int u = 0; u < V; ++u) acc[cc][u] = fmaf(w[s0 + b], v[u], acc[cc][u]);
        }
      }
    }
    for (int j = j_rest; j < k; ++j) {
      const int q = slot_of(inv_perm, o, j, cap);
      if (q < 0) continue;
      const float wq = tw ? tw[o + j] : 1.f;
#pragma unroll
      for (int cc = 0; cc < WCPL; ++cc) {
        const int c = c0 + (cc * 64 + lane) * V;
        if (c >= d) continue;
        float v[V];
        load16_f32(rows + (size_t)q * d + c, v);
#pragma unroll
        for (int u = 0; u < V; ++u) acc[cc][u] = fmaf(wq, v[u], acc[cc][u]);
      }
    }
#pragma unroll
    for (int cc = 0; cc < WCPL; ++cc) {
      const int c = c0 + (cc * 64 + lane) * V;
      if (c >= d) continue;
      if (add) {
        float v[V];
        unpack16_f32(a_raw[cc], v, rows);
#pragma unroll
        for (int u = 0; u < V; ++u) acc[cc][u] += v[u];
      }
      store16_f32(out + (size_t)t * d + c, acc[cc]);
    }
  }
}

template <class T>
__global__ __launch_bounds__(256) void unpermute_kernel(const T* dxp, int T_, int d, int k, int cap,
                                                        const int32_t* inv_perm, T* dx,
                                                        int accumulate) {
  // dxp is read only here: streamed past the caches
  weighted_row_sum<T, true>(dxp, T_, d, k, cap, nullptr, inv_perm, accumulate ? dx : nullptr, dx);
}

template <class T>
__global__ __launch_bounds__(256) void combine_fwd_kernel(const T* yp, int T_, int d, int k, int cap,
                                                          const float* tw,
                                                          const int32_t* inv_perm,
                                                          const T* y_add, T* y) {
  // yp stays cached: the backward's combine reads it again
  weighted_row_sum<T, false>(yp, T_, d, k, cap, tw, inv_perm, y_add, y);
}

// dyp[slot] = w * dy[t] and dtw[t, j] = <dy[t], yp[slot]> for every resident
// route, one route after the other (0 for ghost routes).  Kept lean on
// registers: this kernel runs best at full occupancy.
template <class T>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const T* dy, const T* yp, int T_, int d,
                                                          int k, int cap, const float* tw,
                                                          const int32_t* inv_perm, T* dyp,
                                                          float* dtw) {
  constexpr int V = Vec16<T>::N;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;
  const size_t o = (size_t)t * k;
  // lanes j < 64 hold route j's slot and weight
  const int my_p = lane < k ? slot_of(inv_perm, o, lane, cap) : -1;
  const float my_w = lane < k ? tw[o + lane] : 0.f;
  for (int j = 0; j < k; ++j) {
    const int p = j < 64 ? __shfl(my_p, j, 64) : slot_of(inv_perm, o, j, cap);
    if (p < 0) {  // ghost route: no gradient
      if (lane == 0) dtw[o + j] = 0.f;
      continue;
    }
    const float wj = j < 64 ? __shfl(my_w, j, 64) : tw[o + j];
    float dot = 0.f;
    for (int c = lane * V; c < d; c += 64 * V) {
      float g[V], v[V], out[V];
      load16_f32(dy + (size_t)t * d + c, g);
      load16_f32(yp + (size_t)p * d + c, v);
#pragma unroll
      for (int u = 0; u < V; ++u) {
        dot = fmaf(g[u], v[u], dot);
        out[u] = wj * g[u];
      }
      store16_f32(dyp + (size_t)p * d + c, out);
    }
    dot = wave_sum(dot);
    if (lane == 0) dtw[o + j] = dot;
  }
}

// combine_bwd for k <= 8: per token (one wave) the dy row is loaded once and
// the Yp rows of up to CB_RB resident routes are requested together with it,
// before any is used; routes beyond the batch (k > CB_RB) reuse the loaded
// dy.  dtw of route j (0 for ghost routes) is written by lane j.
constexpr int CB_RB = 4;
template <class T>
__global__ __launch_bounds__(256) void combine_bwd_rows_kernel(const T* dy, const T* yp, int T_,
                                                               int d, int k, int cap,
                                                               const float* tw,
                                                               const int32_t* inv_perm, T* dyp,
                                                               float* dtw) {
  constexpr int V = Vec16<T>::N;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;
  const size_t o = (size_t)t * k;
  const int my_p = lane < k ? slot_of(inv_perm, o, lane, cap) : -1;
  const float my_w = lane < k ? tw[o + lane] : 0.f;
  const uint64_t m = __ballot(my_p >= 0);
  const int nr = __popcll(m);
  // resident routes in route order: slot, weight
  int p[8];
  float w[8];
  {
    uint64_t mm = m;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int src = mm ? __builtin_ctzll(mm) : 0;
      p[s] = __shfl(my_p, src, 64);
      w[s] = __shfl(my_w, src, 64);
      mm &= mm - 1;
    }
  }
  float dot[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (nr > 0) {
    for (int c0 = 0; c0 < d; c0 += WCPL * 64 * V) {
      u32x4_t g_raw[WCPL];
#pragma unroll
      for (int cc = 0; cc < WCPL; ++cc) {
        const int c = c0 + (cc * 64 + lane) * V;
        if (c < d) g_raw[cc] = *reinterpret_cast<const u32x4_t*>(dy + (size_t)t * d + c);
      }
#pragma unroll
      for (int s0 = 0; s0 < 8; s0 += CB_RB) {
        if (s0 >= nr) break;
        u32x4_t v_raw[CB_RB][WCPL];
#pragma unroll
        for (int b = 0; b < CB_RB; ++b) {
          if (s0 + b >= nr) continue;
#pragma unroll
          for (int cc = 0; cc < WCPL; ++cc) {
            const int c = c0 + (cc * 64 + lane) * V;
            if (c < d) v_raw[b][cc] = *reinterpret_cast<const u32x4_t*>(yp + (size_t)p[s0 + b] * d + c);
          }
        }
#pragma unroll
        for (int b = 0; b < CB_RB; ++b) {
          if (s0 + b >= nr) continue;
#pragma unroll
          for (int cc = 0; cc < WCPL; ++cc) {
            const int c = c0 + (cc * 64 + lane) * V;
            if (c >= d) continue;
            float g[V], v[V], out[V];
            unpack16_f32(g_raw[cc], g, dy);
            unpack16_f32(v_raw[b][cc], v, yp);
#pragma unroll
            for (int u = 0; u < V; ++u) {
              dot[s0 + b] = fmaf(g[u], v[u], dot[s0 + b]);
              out[u] = w[s0 + b] * g[u];
            }
            store16_f32(dyp + (size_t)p[s0 + b] * d + c, out);
          }
        }
      }
    }
  }
  // the resident routes' dot products, reduced together (fixed xor order),
  // over as many as the token has (rounded up to 2, 4 or 8)
  auto reduce = [&](auto n_tag) {
    constexpr int N = decltype(n_tag)::value;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
#pragma unroll
      for (int s = 0; s < N; ++s) dot[s] += __shfl_xor(dot[s], off, 64);
  };
  if (nr > 4) reduce(std::integral_constant<int, 8>{});
  else if (nr > 2) reduce(std::integral_constant<int, 4>{});
  else if (nr > 0) reduce(std::integral_constant<int, 2>{});
  if (lane < k) {
    float r = 0.f;
    if (my_p >= 0) {
      const int pos = __popcll(m & ((1ull << lane) - 1ull));
#pragma unroll
      for (int s = 0; s < 8; ++s)
        if (s == pos) r = dot[s];
    }
    dtw[o + lane] = r;
  }
}

struct DeltaArgs {
  const float* start;
  const float* now;
  const float* peers[kMaxPeers];
  float* dl;
  float* avg;
  size_t n;
  int n_peers;
  float scale;
};

__global__ __launch_bounds__(256) void expert_delta_kernel(DeltaArgs a) {
  const size_t n4 = a.n / 4;
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    // a stream: nothing is read twice, so the accesses are nontemporal
    const f32x4_t s = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.start) + i);
    const f32x4_t w = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.now) + i);
    const f32x4_t dl = s - w;
    f32x4_t acc = dl;
    for (int p = 0; p < a.n_peers; ++p)
      acc = acc + __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(a.peers[p]) + i);
    if (a.dl) __builtin_nontemporal_store(dl, reinterpret_cast<f32x4_t*>(a.dl) + i);
    __builtin_nontemporal_store(acc * a.scale, reinterpret_cast<f32x4_t*>(a.avg) + i);
  }
  // scalar tail
  for (size_t i = n4 * 4 + (size_t)blockIdx.x * 256 + threadIdx.x; i < a.n; i += stride) {
    const float dl = a.start[i] - a.now[i];
    float acc = dl;
    for (int p = 0; p < a.n_peers; ++p) acc = acc + a.peers[p][i];
    if (a.dl) a.dl[i] = dl;
    a.avg[i] = acc * a.scale;
  }
}

}  // namespace

size_t dispatch_ws_bytes(int T, int k, int E_r) {
  (void)k;
  const size_t nblk = (size_t)(T + DB - 1) / DB;
  return 2 * nblk * (size_t)std::max(E_r, 1) * sizeof(int32_t) + 256;
}

hipError_t launch_dispatch(const void* x, int bf16, int T, int d, int k, int E_r,
                           const int32_t* local, int32_t* counts, int32_t* offsets,
                           int32_t* perm, int32_t* inv_perm, void* xp, void* ws, hipStream_t s) {
  const int nblk = ceil_div(T, DB);
  const int cap = T * std::min(k, E_r);
  int32_t* blk_counts = static_cast<int32_t*>(ws);
  int32_t* blk_base = blk_counts + (size_t)nblk * std::max(E_r, 1);
  if (nblk > 0 && E_r > 0)
    MOE_TIMED("dispatch_count", s, dispatch_count_kernel<<<nblk, DB, 0, s>>>(local, T, k, E_r, blk_counts));
  if (nblk > 0 && k <= PK && E_r <= 256) {
    // scan, slots and gather in one launch
    const int pblk = ceil_div(T, PB);
    if (bf16)
      MOE_TIMED("dispatch_place", s, dispatch_place_kernel<bf16_t><<<pblk, 256, 0, s>>>(
          static_cast<const bf16_t*>(x), local, T, d, k, E_r, cap, E_r > 0 ? nblk : 0, blk_counts,
          counts, offsets, perm, inv_perm, static_cast<bf16_t*>(xp)));
    else
      MOE_TIMED("dispatch_place", s, dispatch_place_kernel<float><<<pblk, 256, 0, s>>>(
          static_cast<const float*>(x), local, T, d, k, E_r, cap, E_r > 0 ? nblk : 0, blk_counts,
          counts, offsets, perm, inv_perm, static_cast<float*>(xp)));
    return hipGetLastError();
  }
  MOE_TIMED("dispatch_scan", s,
            dispatch_scan_kernel<<<1, 64 * SCAN_WAVES, 0, s>>>(blk_counts, E_r > 0 ? nblk : 0, E_r,
                                                               blk_base, counts, offsets));
  if (nblk > 0) {
    MOE_TIMED("dispatch_scatter", s,
              dispatch_scatter_kernel<<<nblk, DB, 0, s>>>(local, T, k, E_r, cap, blk_base, perm,
                                                          inv_perm));
    if (bf16)
      MOE_TIMED("dispatch_gather", s, gather_rows_kernel<bf16_t><<<ceil_div(T, 4), 256, 0, s>>>(
          static_cast<const bf16_t*>(x), T, d, k, cap, inv_perm, static_cast<bf16_t*>(xp)));
    else
      MOE_TIMED("dispatch_gather", s, gather_rows_kernel<float><<<ceil_div(T, 4), 256, 0, s>>>(
          static_cast<const float*>(x), T, d, k, cap, inv_perm, static_cast<float*>(xp)));
  }
  return hipGetLastError();
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t dispatch_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(moe_dispatch_scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_dispatch_noalloc(const void* x, int bf16, int T, int d, int k, int E_r,
                                   const int32_t* local, int32_t* counts, int32_t* offsets,
                                   int32_t* perm, int32_t* inv_perm, void* xp, hipStream_t s) {
  void* ws = nullptr;
  const hipError_t e = dispatch_scratch(&ws);
  if (e != hipSuccess) return e;
  return launch_dispatch(x, bf16, T, d, k, E_r, local, counts, offsets, perm, inv_perm, xp, ws, s);
}

hipError_t launch_dispatch_bwd(const void* dxp, int bf16, int T, int d, int k, int cap,
                               const int32_t* inv_perm, void* dx, int accumulate, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (bf16)
    MOE_TIMED("unpermute", s, unpermute_kernel<bf16_t><<<ceil_div(T, 4), 256, 0, s>>>(
        static_cast<const bf16_t*>(dxp), T, d, k, cap, inv_perm, static_cast<bf16_t*>(dx), accumulate));
  else
    MOE_TIMED("unpermute", s, unpermute_kernel<float><<<ceil_div(T, 4), 256, 0, s>>>(
        static_cast<const float*>(dxp), T, d, k, cap, inv_perm, static_cast<float*>(dx), accumulate));
  return hipGetLastError();
}

hipError_t launch_combine_fwd(const void* yp, int bf16, int T, int d, int k, int cap,
                              const float* tw, const int32_t* inv_perm, const void* y_add, void* y,
                              hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (bf16)
    MOE_TIMED("combine_fwd", s, combine_fwd_kernel<bf16_t><<<ceil_div(T, 4), 256, 0, s>>>(
        static_cast<const bf16_t*>(yp), T, d, k, cap, tw, inv_perm, static_cast<const bf16_t*>(y_add),
        static_cast<bf16_t*>(y)));
  else
    MOE_TIMED("combine_fwd", s, combine_fwd_kernel<float><<<ceil_div(T, 4), 256, 0, s>>>(
        static_cast<const float*>(yp), T, d, k, cap, tw, inv_perm, static_cast<const float*>(y_add),
        static_cast<float*>(y)));
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const void* dy, const void* yp, int bf16, int T, int d, int k,
                              int cap, const float* tw, const int32_t* inv_perm, void* dyp,
                              float* dtw, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (k <= 8) {
    if (bf16)
      MOE_TIMED("combine_bwd", s, combine_bwd_rows_kernel<bf16_t><<<ceil_div(T, 4), 256, 0, s>>>(
          static_cast<const bf16_t*>(dy), static_cast<const bf16_t*>(yp), T, d, k, cap, tw, inv_perm,
          static_cast<bf16_t*>(dyp), dtw));
    else
      MOE_TIMED("combine_bwd", s, combine_bwd_rows_kernel<float><<<ceil_div(T, 4), 256, 0, s>>>(
          static_cast<const float*>(dy), static_cast<const float*>(yp), T, d, k, cap, tw, inv_perm,
          static_cast<float*>(dyp), dtw));
    return hipGetLastError();
  }
  if (bf16)
    MOE_TIMED("combine_bwd", s, combine_bwd_kernel<bf16_t><<<ceil_div(T, 4), 256, 0, s>>>(
        static_cast<const bf16_t*>(dy), static_cast<const bf16_t*>(yp), T, d, k, cap, tw, inv_perm,
        static_cast<bf16_t*>(dyp), dtw));
  else
    MOE_TIMED("combine_bwd", s, combine_bwd_kernel<float><<<ceil_div(T, 4), 256, 0, s>>>(
        static_cast<const float*>(dy), static_cast<const float*>(yp), T, d, k, cap, tw, inv_perm,
        static_cast<float*>(dyp), dtw));
  return hipGetLastError();
}

hipError_t launch_expert_delta(const float* start, const float* now, const float* const* peers,
                               int n_peers, size_t n, float* dl, float* avg, hipStream_t s) {
  DeltaArgs a{};
  a.start = start;
  a.now = now;
  for (int p = 0; p < n_peers; ++p) a.peers[p] = peers[p];
  a.dl = dl;
  a.avg = avg;
  a.n = n;
  a.n_peers = n_peers;
  a.scale = 1.0f / (float)(n_peers + 1);
  if (n == 0) return hipSuccess;
  const size_t want = (n / 4 + 255) / 256;
  const int blocks = (int)std::max<size_t>(1, std::min<size_t>(want, 8192));
  MOE_TIMED("expert_delta", s, expert_delta_kernel<<<blocks, 256, 0, s>>>(a));
  return hipGetLastError();
}

}  // namespace moe
