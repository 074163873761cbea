// Router: logits over all E experts, top-k, gate weights, ghost-expert mask,
// and the router backward.
//
// Forward (App. A: TopK of the router scores; Sec. 3.3: the router stays
// unpartitioned under skip-token, routes to non-resident experts are masked):
//   one block = 32 tokens, 8 waves.  bf16 logits use v_mfma_f32_32x32x16_bf16
//   (tokens x experts tiles, the d reduction split over the 8 waves and summed
//   in a fixed order through LDS; x and, for up to 64 experts, W_r rows are
//   read whole and staged in LDS); fp32 logits use plain FMA loops.  For
//   k <= 8 every wave then selects for 4 tokens, 16 lanes per token
//   (select_groups, row maxima by DPP); for larger k each wave takes tokens
//   one at a time, lane = expert, with k wave-wide (max logit, min id)
//   reductions.
#include "common.h"
#include "kernels.h"
#include "timing.h"

namespace moe {
namespace {

constexpr int RT_TOK = 32;   // tokens per block
constexpr int RT_WAVES = 8;
constexpr int RT_THREADS = 64 * RT_WAVES;

struct RouteFwdArgs {
  const void* x;
  const void* w;
  const float* bias;
  const uint8_t* resident;
  float* logits;
  int32_t* idx;
  float* tw;
  int32_t* local;
  int T, d, E, k, gate;
  float inv_tau;
};

// Wave-wide (value desc, id asc) argmax.
DEVI void wave_argmax(float& v, int& e) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float ov = __shfl_xor(v, o, 64);
    int oe = __shfl_xor(e, o, 64);
    if (ov > v || (ov == v && oe < e)) { v = ov; e = oe; }
  }
}

// Local id (rank among resident experts, -1 for ghosts) of every expert, via
// ballots over chunks of 64 experts.  Executed by wave 0.
DEVI void build_local_map(const uint8_t* resident, int E, int* lmap) {
  const int lane = threadIdx.x & 63;
  int base = 0;
  for (int e0 = 0; e0 < E; e0 += 64) {
    const int e = e0 + lane;
    const bool r = (e < E) && resident[e] != 0;
    const uint64_t m = __ballot(r);
    const int below = __popcll(m & ((1ull << lane) - 1ull));
    if (e < E) lmap[e] = r ? base + below : -1;
    base += __popcll(m);
  }
}

// bf16 logits of RT_TOK tokens into zl[RT_TOK][ldz] (raw dot products).
// Wave w reduces the 64-wide slices w, w + RT_WAVES, ... of d, up to two
// slices per round with all their loads issued before the MFMAs; the per-wave partial
// sums are then added in wave order through LDS.
template <int NEB>
DEVI void logits_mfma(const RouteFwdArgs& a, int t0, float* zl, int ldz) {
  const bf16_t* x = static_cast<const bf16_t*>(a.x);
  const bf16_t* w = static_cast<const bf16_t*>(a.w);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int row = lane & 31;
  const int half = lane >> 5;
  f32x16_t acc[NEB];
#pragma unroll
  for (int eb = 0; eb < NEB; ++eb) acc[eb] = f32x16_t{};
  const bf16x8_t zero8 = {};
  const u32x4_t zero4 = {0u, 0u, 0u, 0u};
  const int n_slices = (a.d + 63) / 64;
  // x slices go through a wave-private LDS buffer: loaded as whole 128-byte
  // row pieces (8 lanes per token row; 32 rows per read in fragment order
  // would touch 32 cache lines per instruction), stored with the 16-byte
  // chunk c of row r at chunk position c ^ ((r >> 1) & 7) so that the
  // fragment reads (16 consecutive rows, same chunk) are free of bank
  // conflicts.  The W slices stay direct fragment loads (L2-resident).
  constexpr int UNR = NEB <= 2 ? 2 : 1;
  __shared__ __attribute__((aligned(16))) char xst[RT_WAVES][UNR][RT_TOK * 128];
  auto xswz = [](int r, int c) { return r * 128 + ((c ^ ((r >> 1) & 7)) << 4); };
  auto load_x = [&](int kb, u32x4_t* v) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tr = t0 + j * 8 + (lane >> 3);
      const int c = kb * 64 + (lane & 7) * 8;
      v[j] = (kb < n_slices && tr < a.T && c + 8 <= a.d)
                 ? *reinterpret_cast<const u32x4_t*>(x + (size_t)tr * a.d + c)
                 : zero4;
    }
  };
  auto store_x = [&](int u, const u32x4_t* v) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<u32x4_t*>(&xst[wave][u][xswz(j * 8 + (lane >> 3), lane & 7)]) = v[j];
  };
  // the lane's 32 consecutive elements of a slice feed the 4 k16 MFMA steps
  // in the same order for the token and the expert operand
  auto read_x = [&](bf16x8_t* av, int u) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      av[q] = *reinterpret_cast<const bf16x8_t*>(&xst[wave][u][xswz(row, half * 4 + q)]);
  };
  auto load_w = [&](int kb, bf16x8_t (*bv)[4]) {
    const int c0 = kb * 64 + half * 32;
#pragma unroll
    for (int eb = 0; eb < NEB; ++eb) {
      const int e = eb * 32 + row;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = c0 + q * 8;
        bv[eb][q] = (kb < n_slices && e < a.E && c + 8 <= a.d)
                        ? *reinterpret_cast<const bf16x8_t*>(w + (size_t)e * a.d + c) : zero8;
      }
    }
  };
  // UNR slices per round (fewer for wide expert sets, to stay in registers)
  for (int kb = wave; kb < n_slices; kb += UNR * RT_WAVES) {
    bf16x8_t av[UNR][4], bv[UNR][NEB][4];
    u32x4_t xv[UNR][4];
    // the W_r fragments (L2) are requested with the x rows (HBM), not after
    // the x rows have been staged
#pragma unroll
    for (int u = 0; u < UNR; ++u) load_w(kb + u * RT_WAVES, bv[u]);
#pragma unroll
    for (int u = 0; u < UNR; ++u) load_x(kb + u * RT_WAVES, xv[u]);  // zeros past the end
#pragma unroll
    for (int u = 0; u < UNR; ++u) store_x(u, xv[u]);
#pragma unroll
    for (int u = 0; u < UNR; ++u) read_x(av[u], u);
#pragma unroll
    for (int u = 0; u < UNR; ++u)
#pragma unroll
      for (int eb = 0; eb < NEB; ++eb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          acc[eb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[u][q], bv[u][eb][q], acc[eb], 0, 0, 0);
  }
  // deterministic cross-wave sum (wave order).  Up to 64 experts: every wave
  // stores its partial tile, then each thread adds its entries' RT_WAVES
  // partials and finishes z (bias, temperature, logits store); wider expert
  // sets add wave by wave into zl and the caller finishes z.
  if constexpr (NEB <= 2) {
    __shared__ float part[RT_WAVES][RT_TOK * NEB * 32];
#pragma unroll
    for (int eb = 0; eb < NEB; ++eb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = (r >> 2) * 8 + half * 4 + (r & 3);
        part[wave][i * NEB * 32 + eb * 32 + row] = acc[eb][r];
      }
    }
    __syncthreads();
    for (int p = threadIdx.x; p < RT_TOK * NEB * 32; p += RT_THREADS) {
      const int i = p / (NEB * 32), e = p % (NEB * 32);
      float v = part[0][p];
#pragma unroll
      for (int wv = 1; wv < RT_WAVES; ++wv) v += part[wv][p];
      if (e < a.E) {
        // z = (dot + bias) * inv_tau, stored as it is summed
        if (a.bias) v += a.bias[e];
        v *= a.inv_tau;
        zl[i * ldz + e] = v;
        const int t = t0 + i;
        if (a.logits && t < a.T) a.logits[(size_t)t * a.E + e] = v;
      }
    }
    __syncthreads();
  } else {
    for (int wv = 0; wv < RT_WAVES; ++wv) {
      if (wave == wv) {
#pragma unroll
        for (int eb = 0; eb < NEB; ++eb) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int i = (r >> 2) * 8 + half * 4 + (r & 3);
            const int e = eb * 32 + row;
            if (e < a.E) {
              float* p = zl + i * ldz + e;
              *p = (wv == 0) ? acc[eb][r] : *p + acc[eb][r];
            }
          }
        }
      }
      __syncthreads();
    }
  }
}

// bf16 logits for up to 64 experts and d <= 64 XS RT_WAVES.  Wave w reduces
// the slices w + RT_WAVES u (u < XS) of d.  The x rows and W_r rows of a
// slice are read whole (8 lanes per 128-byte row piece, two slices ahead of
// their use, into registers) and staged in the wave's own LDS region, from
// which the MFMA fragments are read.  (Read in fragment order instead, 32
// rows per load, W_r took twice as long to arrive.)  The per-wave partial
// sums are then added in wave order through LDS and z is finished as in
// logits_mfma.
template <int NEB, int XS>
DEVI void logits_mfma_staged(const RouteFwdArgs& a, int t0, float* zl, int ldz) {
  static_assert(NEB <= 2 && XS >= 2, "up to 64 experts, at least two slices per wave");
  const bf16_t* x = static_cast<const bf16_t*>(a.x);
  const bf16_t* w = static_cast<const bf16_t*>(a.w);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int row = lane & 31;
  const int half = lane >> 5;
  constexpr int XR = RT_TOK, WR = NEB * 32;  // x and W_r rows of a slice
  constexpr int SLOT = (XR + WR) * 128;
  constexpr int STG = RT_WAVES * SLOT;
  constexpr int PART = RT_WAVES * RT_TOK * NEB * 32 * 4;
  __shared__ __attribute__((aligned(16))) char lbuf[STG > PART ? STG : PART];
  char* slot = lbuf + wave * SLOT;
  // 16-byte chunk c of staged row r at chunk position c ^ ((r >> 1) & 7): the
  // fragment reads (16 consecutive rows, one chunk) are free of bank conflicts
  auto swz = [](int r, int c) { return r * 128 + ((c ^ ((r >> 1) & 7)) << 4); };
  const int n_slices = (a.d + 63) / 64;
  const u32x4_t zero4 = {0u, 0u, 0u, 0u};
  struct Piece {
    u32x4_t x[XR / 8], w[WR / 8];
  };
  auto load = [&](int kb, Piece& p) {
    const int c = kb * 64 + (lane & 7) * 8;
    const bool ok = kb < n_slices && c + 8 <= a.d;
#pragma unroll
    for (int j = 0; j < XR / 8; ++j) {
      const int t = t0 + j * 8 + (lane >> 3);
      p.x[j] = ok && t < a.T ? *reinterpret_cast<const u32x4_t*>(x + (size_t)t * a.d + c) : zero4;
    }
#pragma unroll
    for (int j = 0; j < WR / 8; ++j) {
      const int e = j * 8 + (lane >> 3);
      p.w[j] = ok && e < a.E ? *reinterpret_cast<const u32x4_t*>(w + (size_t)e * a.d + c) : zero4;
    }
  };
  f32x16_t acc[NEB];
#pragma unroll
  for (int eb = 0; eb < NEB; ++eb) acc[eb] = f32x16_t{};
  Piece pc[XS];
  load(wave, pc[0]);
  load(wave + RT_WAVES, pc[1]);
#pragma unroll
  for (int u = 0; u < XS; ++u) {
    const int kb = wave + u * RT_WAVES;
    if (kb >= n_slices) break;
    // a wave's LDS accesses run in order: the previous slice's fragment
    // reads are done before these stores overwrite them
#pragma unroll
    for (int j = 0; j < XR / 8; ++j)
      *reinterpret_cast<u32x4_t*>(slot + swz(j * 8 + (lane >> 3), lane & 7)) = pc[u].x[j];
#pragma unroll
    for (int j = 0; j < WR / 8; ++j)
      *reinterpret_cast<u32x4_t*>(slot + XR * 128 + swz(j * 8 + (lane >> 3), lane & 7)) = pc[u].w[j];
    if (u + 2 < XS) load(kb + 2 * RT_WAVES, pc[u + 2]);
    bf16x8_t av[4], bv[NEB][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      av[q] = *reinterpret_cast<const bf16x8_t*>(slot + swz(row, half * 4 + q));
#pragma unroll
    for (int eb = 0; eb < NEB; ++eb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        bv[eb][q] = *reinterpret_cast<const bf16x8_t*>(slot + XR * 128 + swz(eb * 32 + row, half * 4 + q));
#pragma unroll
    for (int eb = 0; eb < NEB; ++eb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        acc[eb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[q], bv[eb][q], acc[eb], 0, 0, 0);
  }
  __syncthreads();  // every wave is done with its staging region: the partial sums reuse it
  float* part = reinterpret_cast<float*>(lbuf);
#pragma unroll
  for (int eb = 0; eb < NEB; ++eb) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = (r >> 2) * 8 + half * 4 + (r & 3);
      part[wave * (RT_TOK * NEB * 32) + i * NEB * 32 + eb * 32 + row] = acc[eb][r];
    }
  }
  __syncthreads();
  for (int p = threadIdx.x; p < RT_TOK * NEB * 32; p += RT_THREADS) {
    const int i = p / (NEB * 32), e = p % (NEB * 32);
    float v = part[p];
#pragma unroll
    for (int wv = 1; wv < RT_WAVES; ++wv) v += part[wv * (RT_TOK * NEB * 32) + p];
    if (e < a.E) {
      // z = (dot + bias) * inv_tau, stored as it is summed
      if (a.bias) v += a.bias[e];
      v *= a.inv_tau;
      zl[i * ldz + e] = v;
      const int t = t0 + i;
      if (a.logits && t < a.T) a.logits[(size_t)t * a.E + e] = v;
    }
  }
  __syncthreads();
}

DEVI void logits_f32(const RouteFwdArgs& a, int t0, float* zl, int ldz) {
  const float* x = static_cast<const float*>(a.x);
  const float* w = static_cast<const float*>(a.w);
  for (int p = threadIdx.x; p < RT_TOK * a.E; p += RT_THREADS) {
    const int i = p / a.E, e = p % a.E;
    const int t = t0 + i;
    float s = 0.f;
    if (t < a.T) {
      const float* xr = x + (size_t)t * a.d;
      const float* wr = w + (size_t)e * a.d;
      for (int c = 0; c < a.d; ++c) s = fmaf(xr[c], wr[c], s);
    }
    zl[i * ldz + e] = s;
  }
  __syncthreads();
}

// Logit as read for selection: NaN ranks as -inf (some expert is always
// picked) and -0 as +0 (they tie, as equal values do).
DEVI float sel_value(float v) { return (v != v) ? -INFINITY : v + 0.0f; }

// Order-preserving map of a float to uint32 (larger float -> larger key);
// every float maps above 0, the key of an empty slot.
DEVI uint32_t sel_key(float v) {
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int RT_KSEL = 8;

// Lane permutations within a row of 16 lanes (DPP), applied to a 64-bit value
// (its two halves moved alike): xor 1 and xor 2 inside each quad, then lane
// i <- 7 - i inside each half-row and lane i <- 15 - i inside the row.  After
// taking the maximum with each in turn, every lane of the row holds the row's
// maximum.
template <int CTRL>
DEVI uint64_t row_perm64(uint64_t v) {
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, 0xF, 0xF, false);
  return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}
DEVI uint64_t max64(uint64_t a, uint64_t b) { return a > b ? a : b; }
DEVI uint64_t row16_max64(uint64_t m) {
  m = max64(m, row_perm64<0xB1>(m));   // quad_perm [1, 0, 3, 2]
  m = max64(m, row_perm64<0x4E>(m));   // quad_perm [2, 3, 0, 1]
  m = max64(m, row_perm64<0x141>(m));  // row_half_mirror
  m = max64(m, row_perm64<0x140>(m));  // row_mirror
  return m;
}

// Top-k (k <= RT_KSEL), gate weights and local ids of the block's tokens, 16
// lanes per token (all RT_WAVES waves: wave w takes tokens 4w .. 4w+3): lane
// s of a group holds experts s, s + 16, ... as 64-bit keys (order-preserving
// logit key, then the inverted expert id, so that equal logits rank the lower
// id first; 0 = taken or absent).  Round j takes the group's largest key (a
// row of 16 lanes, by DPP moves) and lane j keeps it, so the selections come
// out in rank order.
template <int LDZ, int NE>
DEVI void select_groups(const RouteFwdArgs& a, const float* zl, int t0, const int* lmap) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int s = lane & 15;
  const int i = wave * 4 + (lane >> 4);
  const int t = t0 + i;
  const float* z = zl + i * LDZ;
  uint64_t cand[NE];
#pragma unroll
  for (int q = 0; q < NE; ++q) {
    const int e = q * 16 + s;
    cand[q] = e < a.E ? ((uint64_t)sel_key(sel_value(z[e])) << 32) | (uint32_t)~e : 0ull;
  }
  int my_id = 0;
  for (int j = 0; j < a.k; ++j) {
    uint64_t m = 0ull;
#pragma unroll
    for (int q = 0; q < NE; ++q) m = cand[q] > m ? cand[q] : m;
    m = row16_max64(m);
#pragma unroll
    for (int q = 0; q < NE; ++q)
      if (cand[q] == m) cand[q] = 0ull;
    if (s == j) my_id = (int)~(uint32_t)m;
  }
  const float my_z = sel_value(z[my_id]);
  const float zmax = __shfl(my_z, lane & 48, 64);  // the group's first selection
  float denom = 1.f;
  if (a.gate == 0 || a.gate == 1) {  // softmax over the k selected / all E logits
    float acc = 0.f;
    if (a.gate == 0) {
      if (s < a.k) acc = expf(my_z - zmax);
    } else {
#pragma unroll
      for (int q = 0; q < NE; ++q) {
        const int e = q * 16 + s;
        if (e < a.E) acc += expf(sel_value(z[e]) - zmax);
      }
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) acc += __shfl_xor(acc, o, 64);
    denom = acc;
  }
  if (s < a.k && t < a.T) {
    const float wj = (a.gate == 2) ? sigmoid_f(my_z) : expf(my_z - zmax) / denom;
    const size_t o = (size_t)t * a.k + s;
    a.idx[o] = my_id;
    a.tw[o] = wj;
    a.local[o] = lmap[my_id];
  }
}

// XS > 0: bf16 with up to 64 experts and d <= 64 XS RT_WAVES (logits_mfma_staged)
template <int NEB, bool BF16, int XS>
__global__ __launch_bounds__(RT_THREADS) void route_fwd_kernel(RouteFwdArgs a) {
  constexpr int LDZ = NEB * 32 + 1;
  constexpr int NQ = (NEB * 32 + 63) / 64;  // logits (and selections) per lane
  __shared__ float zl[RT_TOK * LDZ];
  __shared__ int lmap[256];
  const int t0 = blockIdx.x * RT_TOK;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  if (wave == 0) build_local_map(a.resident, a.E, lmap);
  if constexpr (XS > 0) logits_mfma_staged<NEB, XS>(a, t0, zl, LDZ);
  else if constexpr (BF16) logits_mfma<NEB>(a, t0, zl, LDZ);
  else logits_f32(a, t0, zl, LDZ);
  // z = (dot + bias) * inv_tau (the bf16 logits paths finish it for up to 64 experts)
  constexpr bool z_done = BF16 && NEB <= 2;
  for (int p = threadIdx.x; !z_done && p < RT_TOK * a.E; p += RT_THREADS) {
    const int i = p / a.E, e = p % a.E;
    float v = zl[i * LDZ + e];
    if (a.bias) v += a.bias[e];
    v *= a.inv_tau;
    zl[i * LDZ + e] = v;
    const int t = t0 + i;
    if (a.logits && t < a.T) a.logits[(size_t)t * a.E + e] = v;
  }
  if constexpr (!z_done) __syncthreads();  // (those paths end with one)

  if (a.k <= RT_KSEL) {
    static_assert(RT_TOK == 4 * RT_WAVES, "16 lanes per token in every wave");
    select_groups<LDZ, 2 * NEB>(a, zl, t0, lmap);
    return;
  }
  for (int i = wave; i < RT_TOK; i += RT_WAVES) {
    const int t = t0 + i;
    if (t >= a.T) break;
    float v[NQ];
    bool taken[NQ];
    int my_e[NQ];
    float my_z[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e = q * 64 + lane;
      taken[q] = !(e < a.E);
      v[q] = (e < a.E) ? zl[i * LDZ + e] : 0.f;
      if (v[q] != v[q]) v[q] = -INFINITY;  // NaN ranks last; some expert is always picked
      my_e[q] = 0;
      my_z[q] = 0.f;
    }
    float zmax = 0.f;
    for (int j = 0; j < a.k; ++j) {
      float bv = -INFINITY;
      int be = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int e = q * 64 + lane;
        if (!taken[q] && (v[q] > bv || (v[q] == bv && e < be))) { bv = v[q]; be = e; }
      }
      wave_argmax(bv, be);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        if (q * 64 + lane == be) taken[q] = true;
        if (q * 64 + lane == j) { my_e[q] = be; my_z[q] = bv; }
      }
      if (j == 0) zmax = bv;
    }
    // gate weights of the selected experts (selection j lives in lane j % 64)
    float denom = 1.f;
    if (a.gate == 0) {  // softmax over the k selected logits
      float s = 0.f;
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        if (q * 64 + lane < a.k) s += expf(my_z[q] - zmax);
      denom = wave_sum(s);
    } else if (a.gate == 1) {  // softmax over all E logits
      float s = 0.f;
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        if (q * 64 + lane < a.E) s += expf(v[q] - zmax);
      denom = wave_sum(s);
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int j = q * 64 + lane;
      if (j < a.k) {
        float wj;
        if (a.gate == 2) wj = sigmoid_f(my_z[q]);
        else wj = expf(my_z[q] - zmax) / denom;
        const size_t o = (size_t)t * a.k + j;
        a.idx[o] = my_e[q];
        a.tw[o] = wj;
        a.local[o] = lmap[my_e[q]];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward.  dz per token (wave per token, lane per expert), then
// dW_r = inv_tau * dz^T x as per-chunk partial sums reduced in a fixed order,
// and dx (+)= inv_tau * dz W_r.

struct RouteBwdArgs {
  const void* x;
  const void* w;
  const int32_t* idx;
  const float* tw;
  const float* logits;
  const float* dtw;
  float* dz;
  float* dw;
  float* db;
  void* dx;
  float* part_w;  // [n_chunks][E][d]
  float* part_b;  // [n_chunks][n_bparts][E]
  int T, d, E, k, gate, accumulate_dx, n_chunks;
  int n_bparts;   // d_bias partial sums per chunk
  float inv_tau;
};

constexpr int RB_CHUNK = 256;  // tokens per partial sum of dW_r

__global__ __launch_bounds__(256) void route_dz_kernel(RouteBwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= a.T) return;
  const size_t o = (size_t)t * a.k;
  // s = <w, dw> over the k routes (lane-parallel, fixed tree order)
  float s = 0.f;
  for (int j = lane; j < a.k; j += 64) s += a.tw[o + j] * a.dtw[o + j];
  s = wave_sum(s);
  float zmax = 0.f, denom = 1.f;
  if (a.gate == 1) {
    float m = -INFINITY;
    for (int e = lane; e < a.E; e += 64) m = fmaxf(m, a.logits[(size_t)t * a.E + e]);
    zmax = wave_max(m);
    float acc = 0.f;
    for (int e = lane; e < a.E; e += 64) acc += expf(a.logits[(size_t)t * a.E + e] - zmax);
    denom = wave_sum(acc);
  }
  for (int e = lane; e < a.E; e += 64) {
    int jj = -1;
    for (int j = 0; j < a.k; ++j)
      if (a.idx[o + j] == e) { jj = j; break; }
    float g = 0.f;
    if (a.gate == 0) {
      if (jj >= 0) g = a.tw[o + jj] * (a.dtw[o + jj] - s);
    } else if (a.gate == 2) {
      if (jj >= 0) { const float wv = a.tw[o + jj]; g = a.dtw[o + jj] * wv * (1.f - wv); }
    } else {
      const float p = expf(a.logits[(size_t)t * a.E + e] - zmax) / denom;
      g = p * ((jj >= 0 ? a.dtw[o + jj] : 0.f) - s);
    }
    a.dz[(size_t)t * a.E + e] = g;
  }
}

// partial[c][e][col] = sum_{t in chunk c} dz[t,e] x[t,col]; block = 64 cols x
// 64 experts of one chunk, thread = 4 experts x 4 cols.
template <class T>
__global__ __launch_bounds__(256) void route_dw_partial_kernel(RouteBwdArgs a) {
  __shared__ float sdz[32][65];
  __shared__ float sx[32][65];
  const T* x = static_cast<const T*>(a.x);
  const int c0 = blockIdx.x * 64;
  const int e0 = blockIdx.y * 64;
  const int chunk = blockIdx.z;
  const int tb = chunk * RB_CHUNK;
  const int te = min(a.T, tb + RB_CHUNK);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  float bacc = 0.f;
  for (int t1 = tb; t1 < te; t1 += 32) {
    for (int p = threadIdx.x; p < 32 * 64; p += 256) {
      const int i = p >> 6, c = p & 63;
      const int t = t1 + i;
      sdz[i][c] = (t < te && e0 + c < a.E) ? a.dz[(size_t)t * a.E + e0 + c] : 0.f;
      sx[i][c] = (t < te && c0 + c < a.d) ? to_f32(x[(size_t)t * a.d + c0 + c]) : 0.f;
    }
    __syncthreads();
    for (int i = 0; i < 32; ++i) {
      float zv[4], xv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { zv[u] = sdz[i][ty * 4 + u]; xv[u] = sx[i][tx * 4 + u]; }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(zv[u], xv[v], acc[u][v]);
    }
    if (blockIdx.x == 0 && threadIdx.x < 64)
      for (int i = 0; i < 32; ++i) bacc += sdz[i][threadIdx.x];
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = e0 + ty * 4 + u;
    if (e >= a.E) continue;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int c = c0 + tx * 4 + v;
      if (c < a.d) a.part_w[((size_t)chunk * a.E + e) * a.d + c] = acc[u][v];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < 64 && e0 + (int)threadIdx.x < a.E)
    a.part_b[(size_t)chunk * a.n_bparts * a.E + e0 + threadIdx.x] = bacc;
}

__global__ __launch_bounds__(256) void route_dw_reduce_kernel(RouteBwdArgs a) {
  // dW_r[i] = inv_tau * (((p_0[i] + p_1[i]) + p_2[i]) + ...); the chunk
  // loads of a thread are issued 8 at a time
  const size_t n = (size_t)a.E * a.d;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    float s = 0.f;
    int c = 0;
    for (; c + 8 <= a.n_chunks; c += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = a.part_w[(size_t)(c + u) * n + i];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; c < a.n_chunks; ++c) s += a.part_w[(size_t)c * n + i];
    a.dw[i] = s * a.inv_tau;
  }
  if (a.db && blockIdx.x == 0) {
    // d_bias[e] = inv_tau * sum of the (chunk, part) partials: four
    // consecutive ranges summed by four threads, then added in range order
    __shared__ float q4[4][64];
    const int np = a.n_chunks * a.n_bparts;
    for (int e0 = 0; e0 < a.E; e0 += 64) {
      const int e = e0 + (threadIdx.x & 63), q = threadIdx.x >> 6;
      const int pb = (int)((long)np * q / 4), pe = (int)((long)np * (q + 1) / 4);
      float s = 0.f;
      if (e < a.E) {
        int c = pb;
        for (; c + 8 <= pe; c += 8) {
          float v[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) v[u] = a.part_b[(size_t)(c + u) * a.E + e];
#pragma unroll
          for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; c < pe; ++c) s += a.part_b[(size_t)c * a.E + e];
      }
      q4[q][threadIdx.x & 63] = s;
      __syncthreads();
      if (q == 0 && e < a.E)
        a.db[e] = (((q4[0][threadIdx.x] + q4[1][threadIdx.x]) + q4[2][threadIdx.x]) +
                   q4[3][threadIdx.x]) * a.inv_tau;
      __syncthreads();
    }
  }
}

// dx[t, c..c+V) (+)= inv_tau * sum_e dz[t,e] W_r[e, c..c+V); block = 8 tokens,
// thread = 8 tokens x one 16-byte column vector.
template <class T>
__global__ __launch_bounds__(256) void route_dx_kernel(RouteBwdArgs a) {
  constexpr int V = Vec16<T>::N;
  constexpr int TT = 8;
  __shared__ float sdz[TT][257];
  const T* w = static_cast<const T*>(a.w);
  T* dx = static_cast<T*>(a.dx);
  const int t0 = blockIdx.x * TT;
  for (int p = threadIdx.x; p < TT * a.E; p += 256) {
    const int i = p / a.E, e = p % a.E;
    sdz[i][e] = (t0 + i < a.T) ? a.dz[(size_t)(t0 + i) * a.E + e] : 0.f;
  }
  __syncthreads();
  for (int c = threadIdx.x * V; c < a.d; c += 256 * V) {
    float acc[TT][V];
#pragma unroll
    for (int i = 0; i < TT; ++i)
#pragma unroll
      for (int u = 0; u < V; ++u) acc[i][u] = 0.f;
    for (int e = 0; e < a.E; ++e) {
      float wv[V];
      load16_f32(w + (size_t)e * a.d + c, wv);
#pragma unroll
      for (int i = 0; i < TT; ++i) {
        const float z = sdz[i][e];
#pragma unroll
        for (int u = 0; u < V; ++u) acc[i][u] = fmaf(z, wv[u], acc[i][u]);
      }
    }
#pragma unroll
    for (int i = 0; i < TT; ++i) {
      const int t = t0 + i;
      if (t >= a.T) break;
      T* p = dx + (size_t)t * a.d + c;
      float o[V];
      if (a.accumulate_dx) load16_f32(p, o);
#pragma unroll
      for (int u = 0; u < V; ++u) o[u] = (a.accumulate_dx ? o[u] : 0.f) + a.inv_tau * acc[i][u];
      store16_f32(p, o);
    }
  }
}

// bf16 router backward on MFMA (E <= 64, d % 128 == 0): one block = 128
// columns x RB_CHUNK tokens, in sub-chunks of 64 tokens.  Per sub-chunk the
// block stages x[tokens, cols] and dz[tokens, 0..63] in LDS, the fp32 dz split
// into a bf16 pair hi + lo (|dz - hi - lo| <= 2^-17 |dz|), and computes
//   dW partial[e, c] += sum_t (hi + lo)[t, e] x[t, c]            (k = tokens)
//   dx[t, c] (+)= inv_tau * sum_e (hi + lo)[t, e] W_r[e, c]       (k = experts)
// with v_mfma_f32_32x32x16_bf16; wave w owns columns 32w..32w+31 of both.
// The next sub-chunk's x and dz are loaded into registers while the current
// one is computed; the dx result is staged through LDS so that the update of
// dx reads and writes whole row segments.  The per-chunk dW partials, and
// one d_bias partial per block (its column block's share of the chunk's
// tokens, so that no block carries the whole chunk's bias sum: that made the
// blocks of column 0 the critical path, 15 us of about 50), are summed in a
// fixed order by route_dw_reduce_kernel.
constexpr int RBM_COLS = 128;
constexpr int RBM_SUB = 64;                   // tokens per sub-chunk
constexpr int RBM_XS = RBM_COLS * 2 + 64;     // x row stride (bytes): the 4 rows of
                                              // a transposed read on distinct banks
constexpr int RBM_ZS = 64 * 2 + 16;           // dz row stride: 16 rows of a 16-byte
                                              // read on distinct banks
constexpr int RBM_WS = RBM_COLS * 2 + 64;     // W_r row stride
constexpr int RBM_LDS = RBM_SUB * RBM_XS + 2 * RBM_SUB * RBM_ZS + 64 * RBM_WS;
constexpr int RBM_STG = RBM_COLS + 4;  // fp32 row stride of the staged dx update
static_assert(RBM_SUB * RBM_STG * 4 <= RBM_SUB * RBM_XS + 2 * RBM_SUB * RBM_ZS,
              "the staged dx update must fit over the x and dz tiles");
constexpr int RBM_XV = RBM_SUB * RBM_COLS / 8 / 256;  // 16-byte x vectors per thread
constexpr int RBM_ZV = RBM_SUB * 64 / 8 / 256;        // 8-expert dz groups per thread
static_assert(RBM_XV * 256 * 8 == RBM_SUB * RBM_COLS && RBM_ZV * 256 * 8 == RBM_SUB * 64,
              "staging split");

__global__ __launch_bounds__(256, 2) void route_bwd_mfma_kernel(RouteBwdArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[RBM_LDS];
  char* xs = lds;
  char* zh = xs + RBM_SUB * RBM_XS;
  char* zl = zh + RBM_SUB * RBM_ZS;
  char* wl = zl + RBM_SUB * RBM_ZS;
  const bf16_t* x = static_cast<const bf16_t*>(a.x);
  const bf16_t* w = static_cast<const bf16_t*>(a.w);
  bf16_t* dx = static_cast<bf16_t*>(a.dx);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int c0 = blockIdx.x * RBM_COLS;
  const int chunk = blockIdx.y;
  const int n_sub = min(RB_CHUNK, a.T - chunk * RB_CHUNK + RBM_SUB - 1) / RBM_SUB;
  const bool vec_dz = (a.E & 3) == 0 && ((uintptr_t)a.dz & 15) == 0;
  const u32x4_t zero4 = {0u, 0u, 0u, 0u};

  // W_r[0..63, c0..c0+127] (rows >= E are zero)
  for (int p = tid; p < 64 * (RBM_COLS / 8); p += 256) {
    const int e = p / (RBM_COLS / 8), c = (p % (RBM_COLS / 8)) * 8;
    *reinterpret_cast<u32x4_t*>(wl + e * RBM_WS + c * 2) =
        e < a.E ? *reinterpret_cast<const u32x4_t*>(w + (size_t)e * a.d + c0 + c) : zero4;
  }

  // register staging of one sub-chunk: thread owns x vectors p = tid + 256 v
  // (row p / 16, columns 8 (p % 16)..) and dz groups p = tid + 256 v (row p / 8,
  // experts 8 (p % 8)..)
  u32x4_t xr[RBM_XV];
  float zr[RBM_ZV][8];
  auto load_sub = [&](int t0) {
#pragma unroll
    for (int v = 0; v < RBM_XV; ++v) {
      const int p = tid + 256 * v;
      const int t = t0 + (p >> 4);
      xr[v] = t < a.T ? *reinterpret_cast<const u32x4_t*>(x + (size_t)t * a.d + c0 + (p & 15) * 8)
                      : zero4;
    }
#pragma unroll
    for (int v = 0; v < RBM_ZV; ++v) {
      const int p = tid + 256 * v;
      const int t = t0 + (p >> 3), e0 = (p & 7) * 8;
      const float* src = a.dz + (size_t)t * a.E + e0;
      if (t < a.T && vec_dz && e0 + 8 <= a.E) {
        const f32x4_t u0 = *reinterpret_cast<const f32x4_t*>(src);
        const f32x4_t u1 = *reinterpret_cast<const f32x4_t*>(src + 4);
#pragma unroll
        for (int u = 0; u < 4; ++u) { zr[v][u] = u0[u]; zr[v][4 + u] = u1[u]; }
      } else {
#pragma unroll
        for (int u = 0; u < 8; ++u) zr[v][u] = (t < a.T && e0 + u < a.E) ? src[u] : 0.f;
      }
    }
  };
  auto store_sub = [&]() {
#pragma unroll
    for (int v = 0; v < RBM_XV; ++v) {
      const int p = tid + 256 * v;
      *reinterpret_cast<u32x4_t*>(xs + (p >> 4) * RBM_XS + (p & 15) * 16) = xr[v];
    }
#pragma unroll
    for (int v = 0; v < RBM_ZV; ++v) {
      const int p = tid + 256 * v;
      bf16x8_t hi, lo;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bf16_t h = (bf16_t)zr[v][u];
        hi[u] = h;
        lo[u] = (bf16_t)(zr[v][u] - (float)h);
      }
      *reinterpret_cast<bf16x8_t*>(zh + (p >> 3) * RBM_ZS + (p & 7) * 16) = hi;
      *reinterpret_cast<bf16x8_t*>(zl + (p >> 3) * RBM_ZS + (p & 7) * 16) = lo;
    }
  };

  f32x16_t accw[2] = {f32x16_t{}, f32x16_t{}};
  if (n_sub > 0) load_sub(chunk * RB_CHUNK);
  // d_bias partial: column block b < n_bparts sums the exact fp32 dz of the
  // sub-chunks s with s % n_bparts == b, from the registers that stage them:
  // per thread its two rows, then across the 8 lanes of an expert group
  // (xor shuffles), then (at the end) across the 4 waves in wave order
  const bool do_bias = (int)blockIdx.x < a.n_bparts;
  float bacc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int sc = 0; sc < n_sub; ++sc) {
    const int t0 = chunk * RB_CHUNK + sc * RBM_SUB;
    __syncthreads();  // previous sub-chunk's LDS reads are done
    store_sub();
    if (do_bias && sc % a.n_bparts == (int)blockIdx.x) {
      static_assert(RBM_ZV == 2, "two dz rows per thread");
      float b8[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) b8[u] = zr[0][u] + zr[1][u];
#pragma unroll
      for (int m = 8; m < 64; m <<= 1)
#pragma unroll
        for (int u = 0; u < 8; ++u) b8[u] += __shfl_xor(b8[u], m, 64);
#pragma unroll
      for (int u = 0; u < 8; ++u) bacc[u] += b8[u];
    }
    __syncthreads();
    if (sc + 1 < n_sub) load_sub(t0 + RBM_SUB);
    // old dx of this thread's 16-byte chunks of the sub-chunk (requested
    // before the MFMAs; used by the coalesced update below)
    u32x4_t old[RBM_XV];
    if (a.accumulate_dx) {
#pragma unroll
      for (int v = 0; v < RBM_XV; ++v) {
        const int p = tid + 256 * v;
        const int t = min(t0 + (p >> 4), a.T - 1);
        old[v] = *reinterpret_cast<const u32x4_t*>(dx + (size_t)t * a.d + c0 + (p & 15) * 8);
      }
    }

    // dW partial: k = tokens, m = experts (2 blocks), n = columns
#pragma unroll
    for (int ks = 0; ks < RBM_SUB / 16; ++ks) {
      const bf16x8_t bx = frag_tr(xs, RBM_XS, ks * 16, wave * 32);
#pragma unroll
      for (int eb = 0; eb < 2; ++eb) {
        const bf16x8_t ah = frag_tr(zh, RBM_ZS, ks * 16, eb * 32);
        const bf16x8_t al = frag_tr(zl, RBM_ZS, ks * 16, eb * 32);
        accw[eb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bx, ah, accw[eb], 0, 0, 0);
        accw[eb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bx, al, accw[eb], 0, 0, 0);
      }
    }

    // dx: k = experts (4 k16-steps), m = tokens (2 blocks), n = columns
    f32x16_t accx[2] = {f32x16_t{}, f32x16_t{}};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8_t bw = frag_tr(wl, RBM_WS, ks * 16, wave * 32);
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const int r = tb * 32 + (lane & 31);
        const int e = ks * 16 + 8 * (lane >> 5);
        const bf16x8_t ah = *reinterpret_cast<const bf16x8_t*>(zh + r * RBM_ZS + e * 2);
        const bf16x8_t al = *reinterpret_cast<const bf16x8_t*>(zl + r * RBM_ZS + e * 2);
        accx[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bw, ah, accx[tb], 0, 0, 0);
        accx[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bw, al, accx[tb], 0, 0, 0);
      }
    }
    // lane holds dx[t0 + 32 tb + lane%32][c0 + 32 wave + 8q + 4(lane/32) + 0..3];
    // staged as fp32 through LDS (over the x and dz tiles, now consumed) so
    // that the update of dx reads and writes whole 256-byte row segments
    __syncthreads();
    float* stg = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4_t v = {accx[tb][4 * q], accx[tb][4 * q + 1], accx[tb][4 * q + 2],
                           accx[tb][4 * q + 3]};
        *reinterpret_cast<f32x4_t*>(stg + (tb * 32 + (lane & 31)) * RBM_STG +
                                    wave * 32 + 8 * q + 4 * (lane >> 5)) = v;
      }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < RBM_XV; ++v) {
      const int p = tid + 256 * v;
      const int r = p >> 4, c = (p & 15) * 8;
      const int t = t0 + r;
      if (t >= a.T) continue;
      const f32x4_t lo = *reinterpret_cast<const f32x4_t*>(stg + r * RBM_STG + c);
      const f32x4_t hi = *reinterpret_cast<const f32x4_t*>(stg + r * RBM_STG + c + 4);
      const bf16x8_t ob = __builtin_bit_cast(bf16x8_t, old[v]);
      bf16x8_t o;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float add = a.inv_tau * (u < 4 ? lo[u] : hi[u - 4]);
        o[u] = (bf16_t)(a.accumulate_dx ? (float)ob[u] + add : add);
      }
      *reinterpret_cast<bf16x8_t*>(dx + (size_t)t * a.d + c0 + c) = o;
    }
  }

  // lane holds partial[e = 32 eb + lane%32][c0 + 32 wave + 8q + 4(lane/32) + 0..3]
#pragma unroll
  for (int eb = 0; eb < 2; ++eb) {
    const int e = eb * 32 + (lane & 31);
    if (e >= a.E) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float* p = a.part_w + ((size_t)chunk * a.E + e) * a.d + c0 + wave * 32 + 8 * q +
                 4 * (lane >> 5);
      const f32x4_t o = {accw[eb][4 * q], accw[eb][4 * q + 1], accw[eb][4 * q + 2],
                         accw[eb][4 * q + 3]};
      *reinterpret_cast<f32x4_t*>(p) = o;
    }
  }
  if (do_bias) {
    // lanes 0..7 hold experts 8 lane .. 8 lane + 7 of this wave's rows
    __shared__ float bpart[4][64];
    if (lane < 8)
#pragma unroll
      for (int u = 0; u < 8; ++u) bpart[wave][lane * 8 + u] = bacc[u];
    __syncthreads();
    if (tid < a.E)
      a.part_b[((size_t)chunk * a.n_bparts + blockIdx.x) * a.E + tid] =
          ((bpart[0][tid] + bpart[1][tid]) + bpart[2][tid]) + bpart[3][tid];
  }
}

}  // namespace

hipError_t launch_route_fwd(const void* x, const void* w, const float* bias, int bf16, int T,
                            int d, int E, int k, float inv_tau, int gate, const uint8_t* resident,
                            float* logits, int32_t* idx, float* tw, int32_t* local,
                            hipStream_t s) {
  RouteFwdArgs a{x, w, bias, resident, logits, idx, tw, local, T, d, E, k, gate, inv_tau};
  if (T == 0) return hipSuccess;
  const dim3 grid(ceil_div(T, RT_TOK));
  const int neb = E <= 32 ? 1 : E <= 64 ? 2 : E <= 128 ? 4 : 8;
  // slices of d per wave for the staged bf16 path (0: not taken)
  const int xs = (!bf16 || neb > 2) ? 0 : d <= 64 * 4 * RT_WAVES ? 4 : d <= 64 * 8 * RT_WAVES ? 8 : 0;
#define ROUTE_LAUNCH(N, B, X) \
  MOE_TIMED("route_fwd", s, route_fwd_kernel<N, B, X><<<grid, RT_THREADS, 0, s>>>(a))
  switch (neb) {
    case 1:
      if (xs == 4) ROUTE_LAUNCH(1, true, 4);
      else if (xs == 8) ROUTE_LAUNCH(1, true, 8);
      else if (bf16) ROUTE_LAUNCH(1, true, 0);
      else ROUTE_LAUNCH(1, false, 0);
      break;
    case 2:
      if (xs == 4) ROUTE_LAUNCH(2, true, 4);
      else if (xs == 8) ROUTE_LAUNCH(2, true, 8);
      else if (bf16) ROUTE_LAUNCH(2, true, 0);
      else ROUTE_LAUNCH(2, false, 0);
      break;
    case 4:
      if (bf16) ROUTE_LAUNCH(4, true, 0);
      else ROUTE_LAUNCH(4, false, 0);
      break;
    default:
      if (bf16) ROUTE_LAUNCH(8, true, 0);
      else ROUTE_LAUNCH(8, false, 0);
      break;
  }
#undef ROUTE_LAUNCH
  return hipGetLastError();
}

// d_bias partial sums per chunk: one per 64-token sub-chunk in the MFMA
// kernel (at most one per column block), one in the VALU kernels
int route_bwd_bparts(int d) { return std::max(1, std::min(d / RBM_COLS, RB_CHUNK / RBM_SUB)); }

size_t route_bwd_ws_bytes(int T, int d, int E) {
  const size_t chunks = (size_t)(T + RB_CHUNK - 1) / RB_CHUNK;
  return chunks * (size_t)E * ((size_t)d + route_bwd_bparts(d)) * sizeof(float) + 256;
}

hipError_t launch_route_bwd(const void* x, const void* w, int bf16, int T, int d, int E, int k,
                            float inv_tau, int gate, const int32_t* idx, const float* tw,
                            const float* logits, const float* dtw, float* dz, float* dw_router,
                            float* d_bias, void* dx, int accumulate_dx, void* ws,
                            hipStream_t s) {
  const int n_chunks = (T + RB_CHUNK - 1) / RB_CHUNK;
  float* part_w = static_cast<float*>(ws);
  float* part_b = part_w + (size_t)n_chunks * E * d;
  const bool mfma = bf16 && E <= 64 && d % RBM_COLS == 0;
  RouteBwdArgs a{x, w, idx, tw, logits, dtw, dz, dw_router, d_bias, dx, part_w, part_b,
                 T, d, E, k, gate, accumulate_dx, n_chunks,
                 mfma ? std::min(d / RBM_COLS, RB_CHUNK / RBM_SUB) : 1, inv_tau};
  if (T > 0) MOE_TIMED("route_dz", s, route_dz_kernel<<<ceil_div(T, 4), 256, 0, s>>>(a));
  if (n_chunks > 0) {
    if (mfma) {
      const dim3 g(d / RBM_COLS, n_chunks);
      MOE_TIMED("route_bwd_mfma", s, route_bwd_mfma_kernel<<<g, 256, 0, s>>>(a));
    } else {
      const dim3 g(ceil_div(d, 64), ceil_div(E, 64), n_chunks);
      if (bf16) MOE_TIMED("route_dw_partial", s, route_dw_partial_kernel<bf16_t><<<g, 256, 0, s>>>(a));
      else MOE_TIMED("route_dw_partial", s, route_dw_partial_kernel<float><<<g, 256, 0, s>>>(a));
    }
  }
  {
    // n_chunks == 0 (T == 0) sums nothing and writes zeros
    const int blocks = (int)std::min<size_t>(4096, ((size_t)E * d + 255) / 256);
    MOE_TIMED("route_dw_reduce", s, route_dw_reduce_kernel<<<blocks, 256, 0, s>>>(a));
  }
  if (T > 0 && !mfma) {
    if (bf16) MOE_TIMED("route_dx", s, route_dx_kernel<bf16_t><<<ceil_div(T, 8), 256, 0, s>>>(a));
    else MOE_TIMED("route_dx", s, route_dx_kernel<float><<<ceil_div(T, 8), 256, 0, s>>>(a));
  }
  return hipGetLastError();
}

}  // namespace moe
