// Grouped SwiGLU expert FFN (forward and backward) as grouped GEMMs.
//
// Per resident expert g (rows [offsets[g], offsets[g+1]) of the dispatched
// activations), the SwiGLU expert computes G = X Wg^T, U = X Wu^T,
// Hh = silu(G)*U, Y = Hh Wd^T, and its backward (the workloads' expert form;
// the paper's own expert is a projection followed by SiLU, App. B.3.1).  Six
// GEMM shapes cover it:
//
//   kind      C                 A (row = group token)   B                 layout
//   GU_FWD    [G|U]  M=n, N=2H  xp   [cap,d]  k-contig  w_gate_up[g]      NT, SwiGLU epilogue
//   DOWN_FWD  Y      M=n, N=d   h    [cap,H]  k-contig  w_down[g]         NT
//   DHH_BWD   dHh    M=n, N=H   dyp  [cap,d]  k-contig  w_down[g] [d,H]   NN, dSwiGLU epilogue
//   DX_BWD    dX     M=n, N=d   dgu  [cap,2H] k-contig  w_gate_up[g]      NN
//   DWD       dWd    M=d, N=H   dyp^T  (K = group rows)   h               TN, fp32 out
//   DWGU      dWgu   M=2H,N=d   dgu^T  (K = group rows)   xp              TN, fp32 out
//
// The first four are ragged in M (tiles are laid over the groups from the
// device-side offsets; no host read-back), the last two ragged in K.
//
// bf16: v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  Block tile 128x128,
// k-step 64, 4 waves of 64x64 (2x2 MFMA tiles each).  Both operands are kept
// in LDS k-contiguous (row = M or N index, 64 bf16 = 128 B per row) with the
// 16-byte chunks XOR-swizzled by (row & 7); the two stages are double
// buffered so the global loads of step k+1 overlap the MFMAs of step k.
// Operands that are contiguous along M/N in memory (the TN weight-gradient
// GEMMs and the NN weight operand) are loaded as 4 k-rows x 8 elements per
// thread (16-byte coalesced loads) and transposed in registers before the
// LDS store.
// fp32: a plain 64x64 SIMT tile (4x4 outputs per thread) with the same
// epilogues; used for fp32 layers.
#include "common.h"
#include "kernels.h"
#include "timing.h"

namespace moe {
namespace {

enum GemmKind { GU_FWD = 0, DOWN_FWD = 1, DHH_BWD = 2, DX_BWD = 3, DWD = 4, DWGU = 5 };

template <int KIND>
struct Kind {
  static constexpr bool MRAG = KIND <= DX_BWD;  // ragged in M (else in K)
  static constexpr bool A_KC = KIND <= DX_BWD;  // A contiguous along k
  static constexpr bool B_KC = KIND <= DOWN_FWD;  // B contiguous along k
};

struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  const void* aux;  // gu, read by the DHH_BWD epilogue
  void* out2;       // h, written by the GU_FWD epilogue
  const int32_t* offsets;
  long lda, ldb, ldc;
  long b_gs, c_gs;  // per-group strides (elements) of B and C
  int n_groups, cap, M, N, K, H, accumulate;
};

struct Tile {
  int g, row0, rows, m0, n0;
};

DEVI int clamp_row(int v, int cap) { return v < 0 ? 0 : (v > cap ? cap : v); }

// Decode the block's tile.  M-ragged: blockIdx.y enumerates the m-tiles of all
// groups in order; blocks past the last tile return false.  K-ragged:
// blockIdx.z is the group, rows = its token count (the K extent).
template <int BM, int BN, int KIND>
DEVI bool decode_tile(const GemmArgs& a, Tile& t) {
  t.n0 = blockIdx.x * BN;
  if constexpr (Kind<KIND>::MRAG) {
    int mt = blockIdx.y;
    int b = clamp_row(a.offsets[0], a.cap);
    for (int g = 0; g < a.n_groups; ++g) {
      int e = clamp_row(a.offsets[g + 1], a.cap);
      if (e < b) e = b;
      const int tiles = (e - b + BM - 1) / BM;
      if (mt < tiles) {
        t.g = g;
        t.row0 = b + mt * BM;
        t.rows = min(BM, e - t.row0);
        t.m0 = 0;
        return true;
      }
      mt -= tiles;
      b = e;
    }
    return false;
  } else {
    t.g = blockIdx.z;
    t.m0 = blockIdx.y * BM;
    const int b = clamp_row(a.offsets[t.g], a.cap);
    const int e = clamp_row(a.offsets[t.g + 1], a.cap);
    t.row0 = b;
    t.rows = e > b ? e - b : 0;
    return true;
  }
}

// GU_FWD: tile column c (within a tile of width BN) -> row of w_gate_up[g].
// Columns come in blocks of 32: gate h-block, up h-block, gate, up, ... so a
// lane holds G and U of the same hidden unit in two accumulators.
template <int BN>
DEVI int gu_brow(int tile_n, int c, int H, bool& ok) {
  const int q = c >> 5;
  const int h = tile_n * (BN / 2) + (q >> 1) * 32 + (c & 31);
  ok = h < H;
  return (q & 1) * H + h;
}

DEVI float dsilu_f(float g) {
  const float s = 1.0f / (1.0f + expf(-g));
  return s * (1.0f + g * (1.0f - s));
}

// Epilogue for one accumulator element at (tile row i, tile col j).
template <int KIND, class T>
DEVI void epi_store(const GemmArgs& a, const Tile& t, int i, int j, float v) {
  if constexpr (KIND == DOWN_FWD || KIND == DX_BWD) {
    const int n = t.n0 + j;
    if (i < t.rows && n < a.N) static_cast<T*>(a.C)[(size_t)(t.row0 + i) * a.ldc + n] = from_f32<T>(v);
  } else if constexpr (KIND == DHH_BWD) {
    const int h = t.n0 + j;
    if (i < t.rows && h < a.N) {
      const size_t m = (size_t)(t.row0 + i);
      const T* gu = static_cast<const T*>(a.aux);
      const float G = to_f32(gu[m * 2 * a.H + h]);
      const float U = to_f32(gu[m * 2 * a.H + a.H + h]);
      T* dgu = static_cast<T*>(a.C);
      dgu[m * 2 * a.H + h] = from_f32<T>(v * U * dsilu_f(G));
      dgu[m * 2 * a.H + a.H + h] = from_f32<T>(v * silu_f(G));
    }
  } else if constexpr (KIND == DWD || KIND == DWGU) {
    const int m = t.m0 + i, n = t.n0 + j;
    if (m < a.M && n < a.N) {
      float* c = static_cast<float*>(a.C) + (size_t)t.g * a.c_gs + (size_t)m * a.ldc + n;
      *c = a.accumulate ? *c + v : v;
    }
  }
}

// GU_FWD epilogue for the pair (G, U) of hidden unit h at tile row i.
template <class T>
DEVI void epi_swiglu(const GemmArgs& a, const Tile& t, int i, int h, float G, float U) {
  if (i < t.rows && h < a.H) {
    const size_t m = (size_t)(t.row0 + i);
    T* gu = static_cast<T*>(a.C);
    gu[m * 2 * a.H + h] = from_f32<T>(G);
    gu[m * 2 * a.H + a.H + h] = from_f32<T>(U);
    static_cast<T*>(a.out2)[m * a.H + h] = from_f32<T>(silu_f(G) * U);
  }
}

// ---------------------------------------------------------------------------
// fp32 SIMT kernel

template <int KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  Tile tl;
  if (!decode_tile<BM, BN, KIND>(a, tl)) return;
  const float* A = static_cast<const float*>(a.A);
  const float* B = static_cast<const float*>(a.B) + (Kind<KIND>::MRAG ? (size_t)tl.g * a.b_gs : 0);
  const int Kd = Kind<KIND>::MRAG ? a.K : tl.rows;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < Kd; k0 += BK) {
    for (int p = tid; p < BM * BK; p += 256) {
      int i, kk;
      if constexpr (Kind<KIND>::A_KC) { i = p / BK; kk = p % BK; } else { kk = p / BM; i = p % BM; }
      const int k = k0 + kk;
      float v = 0.f;
      if (k < Kd) {
        if constexpr (Kind<KIND>::MRAG) {
          if (i < tl.rows) v = A[(size_t)(tl.row0 + i) * a.lda + k];
        } else {
          if (tl.m0 + i < a.M) v = A[(size_t)(tl.row0 + k) * a.lda + tl.m0 + i];
        }
      }
      As[kk][i] = v;
    }
    for (int p = tid; p < BN * BK; p += 256) {
      int j, kk;
      if constexpr (Kind<KIND>::B_KC) { j = p / BK; kk = p % BK; } else { kk = p / BN; j = p % BN; }
      const int k = k0 + kk;
      float v = 0.f;
      if (k < Kd) {
        if constexpr (KIND == GU_FWD) {
          bool ok;
          const int br = gu_brow<BN>(blockIdx.x, j, a.H, ok);
          if (ok) v = B[(size_t)br * a.ldb + k];
        } else if constexpr (KIND == DOWN_FWD) {
          if (tl.n0 + j < a.N) v = B[(size_t)(tl.n0 + j) * a.ldb + k];
        } else if constexpr (Kind<KIND>::MRAG) {  // NN
          if (tl.n0 + j < a.N) v = B[(size_t)k * a.ldb + tl.n0 + j];
        } else {  // TN
          if (tl.n0 + j < a.N) v = B[(size_t)(tl.row0 + k) * a.ldb + tl.n0 + j];
        }
      }
      Bs[kk][j] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { av[u] = As[kk][ty + 16 * u]; bv[u] = Bs[kk][tx + 16 * u]; }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(av[u], bv[v], acc[u][v]);
    }
    __syncthreads();
  }
  if constexpr (KIND == GU_FWD) {
    // cols tx, tx+16 are gate units h = blockIdx.x*32 + col; cols +32 their up units
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 2; ++v)
        epi_swiglu<float>(a, tl, ty + 16 * u, blockIdx.x * (BN / 2) + tx + 16 * v, acc[u][v],
                          acc[u][v + 2]);
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) epi_store<KIND, float>(a, tl, ty + 16 * u, tx + 16 * v, acc[u][v]);
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
//
// Block tile 256 x 256, k-step 64, 256 threads = 4 waves in a 2 x 2 grid;
// each wave owns a 128 x 128 sub-tile = 4 x 4 v_mfma_f32_32x32x16_bf16 tiles
// (256 fp32 accumulators per lane), which keeps the LDS read traffic at
// 8 KB per 16 MFMAs.  Operand tiles go global -> LDS with 16-byte
// global_load_lds (no VGPR staging), two stages double-buffered (128 KB).
//
// LDS layouts (per operand and stage, 32 KB):
//  k-contiguous operand (rows = M or N index): row r holds 64 k = 128 B; its
//    16-byte chunk kc sits at chunk position kc ^ (r & 7).  A fragment row
//    is one ds_read_b128.
//  m/n-contiguous operand (rows = k): row k holds 256 m = 512 B; its 32-byte
//    chunk c sits at position c ^ (2 * (k & 3)).  A fragment is two
//    ds_read_b64_tr_b16: in each 16-lane group, lane j points at (k0 + j/4,
//    m0 + 4*(j%4)) and lane i receives m0 + i for k0..k0+3.
// Rows outside the valid range are clamped to a valid row (finite data) and
// the corresponding outputs are not stored; in the ragged-K tail the B
// fragment elements past the group's last row are zeroed in registers.

constexpr int GT = 256;                     // block tile (M and N)
constexpr int GK = 64;                      // k-step
constexpr int OP_BYTES = GT * GK * 2;       // one operand stage: 32 KB
constexpr int LDS_BYTES = 4 * OP_BYTES;     // 2 stages x (A, B)

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4_t;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8_t;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

DEVI void load_to_lds(const bf16_t* g, char* lds_base) {
  __builtin_amdgcn_global_load_lds((glb_void_t*)g, (lds_void_t*)lds_base, 16, 0, 0);
}

// k-contiguous fill: wave w issues loads i = 0..7, load q = 4i + w covers rows
// 8q .. 8q+7; lane l writes chunk position l%8 of row 8q + l/8.
template <class RowPtr>
DEVI void fill_kc(char* lds_op, const RowPtr& row_ptr, int k0) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int kc = (lane & 7) ^ ((lane >> 3) & 7);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int q = i * 4 + w;
    const int row = q * 8 + (lane >> 3);
    load_to_lds(row_ptr(row) + k0 + kc * 8, lds_op + q * 1024);
  }
}

// m/n-contiguous fill: load q covers k-rows 2q, 2q+1 (512 B each); lane l
// writes the 16-byte slot l%32 of row 2q + l/32.
template <class ElemPtr>
DEVI void fill_mn(char* lds_op, const ElemPtr& elem_ptr, int k0) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ps = lane & 31;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int q = i * 4 + w;
    const int row = q * 2 + (lane >> 5);
    const int c = (ps >> 1) ^ (2 * (row & 3));
    load_to_lds(elem_ptr(k0 + row, c * 16 + (ps & 1) * 8), lds_op + q * 1024);
  }
}

// fragment of rows/cols [mb, mb+32) at k16-step s, k-contiguous layout
DEVI bf16x8_t frag_kc(const char* lds_op, int mb, int s) {
  const int lane = threadIdx.x & 63;
  const int row = mb + (lane & 31);
  const int kc = s * 2 + (lane >> 5);
  return *reinterpret_cast<const bf16x8_t*>(lds_op + row * 128 + ((kc ^ (row & 7)) << 4));
}

// same fragment from the m/n-contiguous layout with two transposing reads
DEVI bf16x8_t frag_mn(const char* lds_op, int mb, int s) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, i = lane & 15;
  const int mn = mb + 16 * (g & 1) + 4 * (i & 3);
  s16x4_t v[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = s * 16 + 8 * (g >> 1) + 4 * h + (i >> 2);
    const int pc = (mn >> 4) ^ (2 * (k & 3));
    const char* p = lds_op + k * 512 + pc * 32 + (mn & 15) * 2;
    v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p));
  }
  // whole-vector concatenation (element-wise inserts of bit-cast lanes were
  // mis-generated into a splat of element 0)
  const s16x8_t both = __builtin_shufflevector(v[0], v[1], 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8_t, both);
}

template <int KIND>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a) {
  using K_ = Kind<KIND>;
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];
  Tile tl;
  if (!decode_tile<GT, GT, KIND>(a, tl)) return;
  const bf16_t* A = static_cast<const bf16_t*>(a.A);
  const bf16_t* B = static_cast<const bf16_t*>(a.B) + (K_::MRAG ? (size_t)tl.g * a.b_gs : 0);
  const int Kd = K_::MRAG ? a.K : tl.rows;
  const int nk = (Kd + GK - 1) / GK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tile_n = blockIdx.x;
  const int last_row = tl.row0 + (tl.rows > 0 ? tl.rows - 1 : 0);

  // operand pointers; out-of-range indices are clamped to valid memory
  auto a_row = [&](int r) -> const bf16_t* {  // M-ragged A, k-contiguous
    return A + (size_t)min(tl.row0 + r, last_row) * a.lda;
  };
  auto a_elem = [&](int k, int c) -> const bf16_t* {  // TN A(i = m0 + c, k)
    const int m = (tl.m0 + c + 8 <= a.M) ? tl.m0 + c : 0;
    return A + (size_t)min(tl.row0 + k, last_row) * a.lda + m;
  };
  auto b_row = [&](int r) -> const bf16_t* {  // NT B rows
    if constexpr (KIND == GU_FWD) {
      bool ok;
      int br = gu_brow<GT>(tile_n, r, a.H, ok);
      if (!ok) br = 0;
      return B + (size_t)br * a.ldb;
    } else {
      return B + (size_t)min(tl.n0 + r, a.N - 1) * a.ldb;
    }
  };
  auto b_elem = [&](int k, int c) -> const bf16_t* {  // NN / TN B(k, n = n0 + c)
    const int n = (tl.n0 + c + 8 <= a.N) ? tl.n0 + c : 0;
    if constexpr (K_::MRAG) return B + (size_t)k * a.ldb + n;
    else return B + (size_t)min(tl.row0 + k, last_row) * a.ldb + n;
  };

  auto fill = [&](int kt, int buf) {
    char* la = lds + buf * 2 * OP_BYTES;
    char* lb = la + OP_BYTES;
    const int k0 = kt * GK;
    if constexpr (K_::A_KC) fill_kc(la, a_row, k0); else fill_mn(la, a_elem, k0);
    if constexpr (K_::B_KC) fill_kc(lb, b_row, k0); else fill_mn(lb, b_elem, k0);
  };

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};

  if (nk > 0) {
    fill(0, 0);
    __builtin_amdgcn_s_waitcnt(0x0);  // vmcnt(0) expcnt(0) lgkmcnt(0)
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) fill(kt + 1, cur ^ 1);
    const char* la = lds + cur * 2 * OP_BYTES;
    const char* lb = la + OP_BYTES;
    const bool tail = !K_::MRAG && (kt + 1) * GK > Kd;
#pragma unroll
    for (int s = 0; s < GK / 16; ++s) {
      bf16x8_t af[4], bfr[4];
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        af[f] = K_::A_KC ? frag_kc(la, wm * 128 + f * 32, s) : frag_mn(la, wm * 128 + f * 32, s);
        bfr[f] = K_::B_KC ? frag_kc(lb, wn * 128 + f * 32, s) : frag_mn(lb, wn * 128 + f * 32, s);
      }
      if (tail) {  // zero B past the group's last row (A there is finite)
        const int kbase = kt * GK + s * 16 + 8 * (lane >> 5);
#pragma unroll
        for (int f = 0; f < 4; ++f)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (kbase + e >= Kd) bfr[f][e] = (bf16_t)0.0f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0x0);
    __syncthreads();
  }

  // accumulator (i, j) register r holds C[row, col] with
  //   row = (r/4)*8 + (lane/32)*4 + r%4,  col = lane%32  inside its 32x32 tile
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = wm * 128 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
      if constexpr (KIND == GU_FWD) {
        // tiles (i, 2p) = gate and (i, 2p+1) = up of hidden units h
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int h = tile_n * (GT / 2) + (2 * wn + p) * 32 + (lane & 31);
          epi_swiglu<bf16_t>(a, tl, row, h, acc[i][2 * p][r], acc[i][2 * p + 1][r]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = wn * 128 + j * 32 + (lane & 31);
          epi_store<KIND, bf16_t>(a, tl, row, col, acc[i][j][r]);
        }
      }
    }
  }
}

template <int KIND>
hipError_t run_gemm(const GemmArgs& a, int bf16, hipStream_t s) {
  const int BMt = bf16 ? GT : 64, BNt = bf16 ? GT : 64;
  dim3 grid;
  const int ncols = (KIND == GU_FWD) ? 2 * a.H : a.N;
  grid.x = ceil_div(ncols, BNt);
  if (Kind<KIND>::MRAG) {
    grid.y = ceil_div(a.cap, BMt) + a.n_groups;
    grid.z = 1;
  } else {
    grid.y = ceil_div(a.M, BMt);
    grid.z = a.n_groups;
  }
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return hipSuccess;
  static constexpr const char* names[] = {"gemm_gu_fwd", "gemm_down_fwd", "gemm_dhh_bwd",
                                          "gemm_dx_bwd", "gemm_dwd", "gemm_dwgu"};
  if (bf16) MOE_TIMED(names[KIND], s, gemm_bf16_kernel<KIND><<<grid, 256, 0, s>>>(a));
  else MOE_TIMED(names[KIND], s, gemm_f32_kernel<KIND><<<grid, 256, 0, s>>>(a));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ffn_fwd(const void* xp, const void* wgu, const void* wd, int bf16, int cap,
                          int d, int H, int n_groups, const int32_t* offsets, void* gu, void* h,
                          void* yp, hipStream_t s) {
  GemmArgs g{};
  g.offsets = offsets;
  g.n_groups = n_groups;
  g.cap = cap;
  g.H = H;
  // [G|U] = X [Wg;Wu]^T with the SwiGLU epilogue
  g.A = xp; g.lda = d;
  g.B = wgu; g.ldb = d; g.b_gs = 2L * H * d;
  g.C = gu; g.ldc = 2L * H; g.out2 = h;
  g.N = 2 * H; g.K = d;
  hipError_t e = run_gemm<GU_FWD>(g, bf16, s);
  if (e != hipSuccess) return e;
  // Y = Hh Wd^T
  g.A = h; g.lda = H;
  g.B = wd; g.ldb = H; g.b_gs = (long)d * H;
  g.C = yp; g.ldc = d; g.out2 = nullptr;
  g.N = d; g.K = H;
  return run_gemm<DOWN_FWD>(g, bf16, s);
}

hipError_t launch_ffn_bwd(const void* dyp, const void* xp, const void* gu, const void* h,
                          const void* wgu, const void* wd, int bf16, int cap, int d, int H,
                          int n_groups, const int32_t* offsets, void* dgu, void* dxp,
                          float* dwgu, float* dwd, int accumulate_dw, hipStream_t s) {
  GemmArgs g{};
  g.offsets = offsets;
  g.n_groups = n_groups;
  g.cap = cap;
  g.H = H;
  g.accumulate = accumulate_dw;
  // dHh = dY Wd, epilogue -> [dG | dU]
  g.A = dyp; g.lda = d;
  g.B = wd; g.ldb = H; g.b_gs = (long)d * H;
  g.C = dgu; g.ldc = 2L * H; g.aux = gu;
  g.N = H; g.K = d;
  hipError_t e = run_gemm<DHH_BWD>(g, bf16, s);
  if (e != hipSuccess) return e;
  // dX = [dG|dU] [Wg;Wu]
  g.A = dgu; g.lda = 2L * H;
  g.B = wgu; g.ldb = d; g.b_gs = 2L * H * d;
  g.C = dxp; g.ldc = d; g.aux = nullptr;
  g.N = d; g.K = 2 * H;
  if ((e = run_gemm<DX_BWD>(g, bf16, s)) != hipSuccess) return e;
  // dWd[g] = dY^T Hh
  g.A = dyp; g.lda = d;
  g.B = h; g.ldb = H; g.b_gs = 0;
  g.C = dwd; g.ldc = H; g.c_gs = (long)d * H;
  g.M = d; g.N = H; g.K = 0;
  if ((e = run_gemm<DWD>(g, bf16, s)) != hipSuccess) return e;
  // dWgu[g] = [dG|dU]^T X
  g.A = dgu; g.lda = 2L * H;
  g.B = xp; g.ldb = d;
  g.C = dwgu; g.ldc = d; g.c_gs = 2L * H * d;
  g.M = 2 * H; g.N = d;
  return run_gemm<DWGU>(g, bf16, s);
}

}  // namespace moe
