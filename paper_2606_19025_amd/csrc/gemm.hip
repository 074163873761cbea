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
// bf16: v_mfma_f32_32x32x16_bf16 with fp32 accumulation in a persistent
// kernel with 256 x 256 block tiles of 8 waves fed from an LDS ring by
// global -> LDS DMA (details at gemm_bf16_kernel and Cfg).  One launch per
// GEMM kind
// covers up to two expert sets (routed and shared experts).
// fp32: a plain 64x64 SIMT tile (4x4 outputs per thread) with the same
// epilogues; used for fp32 layers.
#include "common.h"
#include "kernels.h"
#include "timing.h"

namespace moe {
namespace {

// UP_FWD and DH_BWD are GU_FWD and DHH_BWD for the SiLU expert (one first
// projection W1 [H, d] instead of [Wg; Wu]).
enum GemmKind {
  GU_FWD = 0, DOWN_FWD = 1, DHH_BWD = 2, DX_BWD = 3, DWD = 4, DWGU = 5, UP_FWD = 6, DH_BWD = 7
};

template <int KIND>
struct Kind {
  static constexpr bool MRAG = KIND <= DX_BWD || KIND >= UP_FWD;  // ragged in M (else in K)
  static constexpr bool A_KC = MRAG;                                // A contiguous along k
  static constexpr bool B_KC = KIND <= DOWN_FWD || KIND == UP_FWD;  // B contiguous along k
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
  long c_split;     // K-ragged kinds: stride between the split-K partial outputs
  int n_groups, cap, M, N, K, H, accumulate;
  int ksplit;       // K-ragged kinds: each group's rows split in ksplit parts (0 = 1)
};

struct Tile {
  int g, row0, rows, m0, n0, split;
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
        t.split = 0;
        return true;
      }
      mt -= tiles;
      b = e;
    }
    return false;
  } else {
    t.g = blockIdx.z;
    t.split = 0;
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
  } else if constexpr (KIND == UP_FWD) {
    const int h = t.n0 + j;
    if (i < t.rows && h < a.N) {
      const size_t m = (size_t)(t.row0 + i);
      const T A = from_f32<T>(v);
      static_cast<T*>(a.C)[m * a.ldc + h] = A;
      static_cast<T*>(a.out2)[m * a.H + h] = from_f32<T>(silu_f(to_f32(A)));
    }
  } else if constexpr (KIND == DH_BWD) {
    const int h = t.n0 + j;
    if (i < t.rows && h < a.N) {
      const size_t m = (size_t)(t.row0 + i);
      const float A = to_f32(static_cast<const T*>(a.aux)[m * a.H + h]);
      static_cast<T*>(a.C)[m * a.ldc + h] = from_f32<T>(v * dsilu_f(A));
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
        } else if constexpr (KIND == DOWN_FWD || KIND == UP_FWD) {
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
// Persistent: one 512-thread block per CU loops over output tiles.  Block tile
// 256 x 256; the 8 waves (two per SIMD) form a 4 x 2 grid and each owns a
// 64 x 128 sub-tile = 2 x 4 v_mfma_f32_32x32x16_bf16 tiles (128 fp32
// accumulators per lane), reading 6 fragments (6 KB per wave) per 8 MFMAs.
//
// Operands stream through a ring of NS LDS stages of one k-step (GK) each,
// filled with 16-byte global -> LDS DMA: M-ragged kinds NS = 2 stages of
// GK = 64 (64 KB each), weight-gradient kinds NS = 4 stages of GK = 32
// (32 KB each).  A k-step is GK / 16 k16-steps; per k-step and wave:
//   k16-steps 0 .. GK/16 - 2: 8 MFMAs each, interleaved with the LDS reads of
//   the next k16-step
//   wait for own DMA of k-step kt+1 (vmcnt leaves the later k-steps' loads in
//   flight) and for the LDS reads, barrier (stage kt+1 complete, stage kt
//   free)
//   last k16-step: its MFMAs, interleaved with the LDS reads of k-step kt+1's
//   k16-step 0 and the DMA of k-step kt+NS into stage kt
// So every load has NS - 1 k-steps less one k16-step to land.
// Every k-step issues the same number of DMA loads (past the last k-step the
// last one is loaded again into an unused stage) so vmcnt counting is uniform;
// the ring is drained (vmcnt(0)) before a block moves to its next tile.
//
// Tile order (see tile_decode): bands of GROUP_M m-tiles (2 to 8, per kind,
// see Cfg).  Workgroups are dealt to the 8 XCDs round-robin by id, so block b
// works on tiles of the ranges assigned to XCD b % 8 (an eighth of each set's
// tiles): the 32 tiles an XCD runs at a time form a band rectangle whose
// operand panels its L2 serves.  Output tiles
// end in an epilogue: bf16 results are staged through the drained ring so
// global accesses are whole 16-byte chunks; fp32 weight gradients are stored
// (or added) straight from the accumulators.
//
// LDS layouts (per operand and stage):
//  k-contiguous operand (rows = M or N index): row r holds GK k (2 GK bytes);
//    its 16-byte chunk kc sits at chunk position kc ^ swz(r), swz(r) =
//    (r >> 2) & 3 for GK = 32 and (r >> 1) & 7 for GK = 64, so the 16 lanes of
//    one ds_read_b128 pass (16 consecutive rows, same kc) hit 16 distinct
//    16-byte bank groups of the 64-bank LDS.
//  m/n-contiguous operand (rows = k, GK of them): row k holds 256 m = 512 B; its 32-byte
//    chunk c sits at position c ^ (2 * (k & 3)).  A fragment is two
//    ds_read_b64_tr_b16: in each 16-lane group, lane j points at (k0 + j/4,
//    m0 + 4*(j%4)) and lane i receives m0 + i for k0..k0+3.
// The MFMA is issued with the B fragment as its first operand, so lane l
// accumulates C[m0 + l%32][n0 + 8q + 4(l/32) + t] in register 4q + t: four
// consecutive output columns per lane, stored with 8- or 16-byte vectors.
// Out-of-range M/N rows are clamped to valid memory (their outputs are not
// stored); k-rows past a group's last row (ragged K) are loaded with an
// offset past the buffer resource's range, which reads zeros, so they
// contribute exactly 0.

constexpr int GT = 256;                     // block tile width (N), and height (M) of full tiles
constexpr int N_XCD = 8;

// Tile configuration per kind.  Every kind runs 256 x 256 block tiles with 8
// waves (two per SIMD), one block per CU; each wave owns 64 x 128 of the tile
// (2 x 4 MFMA tiles, 128 accumulators).  Measured on the fine-grained
// workload against 4 waves of 128 x 128 (one per SIMD): DOWN_FWD and DX_BWD
// 9 % faster, the weight-gradient kinds level; and against 128 x 256 tiles at
// two blocks per CU (which padded ragged groups less): GU_FWD 9 % and DHH_BWD
// 3 % faster.  The second wave of a SIMD issues MFMAs while the first waits
// on its operand loads; the 1.5x fragment reads per MFMA of the narrower wave
// tile cost less than that gains.
// M-ragged tiles take k-steps of 64 in a ring of two 64 KB stages: every DMA
// load then fetches whole 128-byte row pieces (half the L2 requests of 64-byte
// pieces; DOWN_FWD 6-10 % and DX_BWD 1-2 % faster than k-steps of 32).  The
// weight-gradient kinds keep k-steps of 32 in four 32 KB stages (equal on the
// fine-grained workload, 2-6 % faster on the mid-size one, and a ragged K
// pads at most 31 rows).
template <int KIND>
struct Cfg {
  static constexpr int NW = 8;                     // waves per block (two per SIMD)
  static constexpr int GK = Kind<KIND>::MRAG ? 64 : 32;  // k-step
  static constexpr int KS = GK / 16;               // k16-steps per k-step
  static constexpr int BM = GT;                    // block tile rows
  static constexpr int WM = BM / (NW / 2);         // wave sub-tile rows (64)
  static constexpr int MI = WM / 32;               // 32-row MFMA tiles per wave
  static constexpr int NS = GK == 64 ? 2 : 4;      // LDS ring stages
  static constexpr int A_BYTES = BM * GK * 2;      // A operand of one stage
  static constexpr int B_BYTES = GT * GK * 2;      // B operand of one stage
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS = NS * STAGE;
  static constexpr int DMA_A = A_BYTES / (1024 * NW);  // 16-byte DMA loads per wave and k-step
  static constexpr int DMA_B = B_BYTES / (1024 * NW);
  static constexpr int DMA_N = DMA_A + DMA_B;
  static constexpr int DMA_MAX = DMA_A > DMA_B ? DMA_A : DMA_B;
  static constexpr int EPI_WAVE = WM * 256;        // epilogue staging per wave
  // m-tiles per band of the tile order, measured per kind on the
  // fine-grained workload (bands of 2, 4, 8 and 16 tried)
  static constexpr int GROUP = (KIND == GU_FWD || KIND == UP_FWD || KIND == DOWN_FWD) ? 8
                               : (KIND == DHH_BWD || KIND == DH_BWD || KIND == DX_BWD) ? 4
                                                                                        : 2;
  static_assert(NW * EPI_WAVE <= LDS, "epilogue staging exceeds the ring");
};


// Sentinel the operand lambdas return for k-rows past the extent; the DMA
// set-up turns it into an out-of-range offset (it is never read).
__device__ const u32x4_t kZero16 = {0u, 0u, 0u, 0u};

// s_waitcnt immediate (gfx9 family): vmcnt in bits [3:0] and [15:14],
// expcnt in [6:4], lgkmcnt in [11:8]; a field at its maximum does not wait.
constexpr int waitcnt_imm(int vm, int lgkm) {
  return (vm & 15) | (((vm >> 4) & 3) << 14) | (7 << 4) | ((lgkm & 15) << 8);
}
#define WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(waitcnt_imm((n), 15))
#define WAIT_LGKMCNT(n) __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, (n)))

// Wait until at most PER * min(n, MAXN) vector memory operations are
// outstanding; n <= 0 waits for all of them (n wave-uniform: s_waitcnt takes
// only an immediate).
template <int PER, int MAXN>
DEVI void wait_vm_groups(int n) {
  if constexpr (MAXN > 0) {
    if (n >= MAXN) {
      WAIT_VMCNT(PER * MAXN);
      return;
    }
    wait_vm_groups<PER, MAXN - 1>(n);
  } else {
    WAIT_VMCNT(0);
  }
}

// 16-byte global -> LDS DMA through a buffer resource: lane l reads the 16
// bytes at byte offset off of the operand and writes them to lds_base + 16 l
// (lds_base must be wave-uniform).  An offset at or past the resource's
// record count (kOOB) reads zeros.  The per-lane offsets are 32-bit, half the
// address registers of 64-bit pointers; timed on the fine-grained workload
// the step was 0.8 % faster than with global_load_lds_dwordx4 on 64-bit
// addresses.  Issued as inline asm so the compiler does not treat every
// later LDS read as possibly aliasing the pending DMA (it would wait for all
// outstanding global loads before each transposing read); the kernel waits for
// the DMA explicitly (vmcnt) before the barrier that publishes a stage.  The
// asm sets m0 itself; the compiler keeps no value of its own in m0 across it
// (m0 is reserved, and nothing else in these kernels uses it), which the
// "m0" clobber records for the reader.
DEVI void load_to_lds(u32x4_t rsrc, unsigned off, char* lds_base) {
  const unsigned m0 = (unsigned)(uintptr_t)(lds_void_t*)lds_base;
  asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(off), "s"(rsrc), "s"(m0)
               : "m0", "memory");
}
// Raw buffer resource over [base, base + kOOB): stride 0, no swizzle, word 3
// the gfx9 default data format.  Every operand stays below kOOB bytes (the
// entry points reject larger ones).
constexpr unsigned kOOB = 0xFFFFFFF0u;
DEVI u32x4_t make_rsrc(const void* base) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  u32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((unsigned)b);
  r[1] = __builtin_amdgcn_readfirstlane((unsigned)(b >> 32) & 0xFFFFu);
  r[2] = kOOB;
  r[3] = 0x00020000u;
  return r;
}

// Per-lane byte offsets (from the operand's base) of the DMA loads a wave
// issues per operand and k-step.  k-contiguous operand with C = GK / 8 chunks per row: load q = 4i + w
// covers rows (64 / C) q .. (64 / C) (q + 1) - 1, lane l writes chunk position
// l % C of row (64 / C) q + l / C.  m/n-contiguous operand:
// load q covers k-rows 2q, 2q+1 (512 B each), lane l writes 16-byte slot l%32
// of row 2q + l/32.
template <int N>
struct DmaPtrs {
  unsigned p[N];
};

// k-contiguous rows hold GK k (GK / 8 chunks of 16 bytes); the chunk
// position is XOR-swizzled by the row so that 16 consecutive rows at one
// chunk fall on 16 distinct 16-byte bank groups.
template <int GK>
DEVI int kc_swz(int r) { return GK == 32 ? (r >> 2) & 3 : (r >> 1) & 7; }

template <int GK, int NW, int N, class RowPtr>
DEVI void dma_kc_init(DmaPtrs<N>& d, const RowPtr& row_ptr, int w, const bf16_t* base) {
  constexpr int CPR = GK / 8;  // chunks per row
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int row = (i * NW + w) * (64 / CPR) + lane / CPR;
    const bf16_t* q = row_ptr(row) + ((lane % CPR) ^ kc_swz<GK>(row)) * 8;
    d.p[i] = (unsigned)((const char*)q - (const char*)base);
  }
}

template <int NW>
DEVI int mn_row(int i, int w) { return (i * NW + w) * 2 + ((threadIdx.x & 63) >> 5); }
DEVI int mn_col(int row) {
  const int ps = threadIdx.x & 31;
  return (((ps >> 1) ^ (2 * (row & 3))) * 16) + (ps & 1) * 8;
}

template <int NW, int N, class ElemPtr>
DEVI void dma_mn_init(DmaPtrs<N>& d, const ElemPtr& elem_ptr, int w, int k0, const bf16_t* base) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int row = mn_row<NW>(i, w);
    // the zero block (k-rows past the extent) becomes an out-of-range offset
    const bf16_t* q = elem_ptr(k0 + row, mn_col(row));
    d.p[i] = q == reinterpret_cast<const bf16_t*>(&kZero16)
                 ? kOOB
                 : (unsigned)((const char*)q - (const char*)base);
  }
}

// fragment of rows/cols [mb, mb+32) at k16-step s, k-contiguous layout
template <int GK>
DEVI bf16x8_t frag_kc(const char* lds_op, int mb, int s) {
  const int lane = threadIdx.x & 63;
  const int row = mb + (lane & 31);
  const int kc = s * 2 + (lane >> 5);
  return *reinterpret_cast<const bf16x8_t*>(lds_op + row * (GK * 2) +
                                            ((kc ^ kc_swz<GK>(row)) << 4));
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

// Epilogue staging.  A wave's 64 x 128 bf16 sub-tile occupies 64 rows of
// 256 B.  The 8-byte unit u (4 columns) of row r sits at unit u ^ epi_key(r):
// the key is a bijection on r mod 32, so the accumulator writes (32 rows at
// one unit per half-wave) hit 32 distinct bank pairs, and rows 2m, 2m+1
// differ in key bit 3, so the SwiGLU reads (8 chunks of two rows per 16
// lanes) fall on disjoint chunks.  A 16-byte chunk c is read back from chunk
// c ^ (key >> 1), halves swapped when the key is odd.

DEVI int epi_key(int r) { return ((r & 1) << 3) | ((r >> 1) & 7) | (r & 16); }

DEVI void epi_put(char* reg, int row, int u, float v0, float v1, float v2, float v3) {
  bf16x4_t o = {(bf16_t)v0, (bf16_t)v1, (bf16_t)v2, (bf16_t)v3};
  *reinterpret_cast<bf16x4_t*>(reg + row * 256 + ((u ^ epi_key(row)) << 3)) = o;
}

DEVI bf16x8_t epi_get(const char* reg, int row, int c) {
  const int key = epi_key(row);
  u32x4_t v = *reinterpret_cast<const u32x4_t*>(reg + row * 256 + ((c ^ (key >> 1)) << 4));
  if (key & 1) v = __builtin_shufflevector(v, v, 2, 3, 0, 1);
  return __builtin_bit_cast(bf16x8_t, v);
}

// Hardware exp2 / reciprocal (about 1 ulp of fp32); their results are rounded
// to bf16.
DEVI float sigmoid_fast(float g) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.44269504088896341f * g));
}
DEVI float silu_fast(float g) { return g * sigmoid_fast(g); }

// Tile enumeration.  Output tiles form an m_tiles x n_tiles grid (M-ragged
// kinds: m-tiles of all groups in group order; K-ragged kinds: (group,
// m-tile) pairs).  Linear tile t walks bands of GROUP_M m-tiles: inside a band
// m varies fastest, then n, so any 32 consecutive tiles cover a GROUP_M x
// (32 / GROUP_M) rectangle and share GROUP_M A panels and 32 / GROUP_M B
// panels in L2.

template <int KIND>
DEVI int m_tile_count(const GemmArgs& a) {
  constexpr int BM = Cfg<KIND>::BM;
  if constexpr (Kind<KIND>::MRAG) {
    int tiles = 0;
    int b = clamp_row(a.offsets[0], a.cap);
    for (int g = 0; g < a.n_groups; ++g) {
      int e = clamp_row(a.offsets[g + 1], a.cap);
      if (e < b) e = b;
      tiles += (e - b + BM - 1) / BM;
      b = e;
    }
    return tiles;
  } else {
    return a.n_groups * max(1, a.ksplit) * ((a.M + BM - 1) / BM);
  }
}

template <int KIND>
DEVI void tile_decode(const GemmArgs& a, int t, int m_tiles, int n_tiles, Tile& tl,
                      int& tile_n) {
  constexpr int BM = Cfg<KIND>::BM, GROUP_M = Cfg<KIND>::GROUP;
  const int band = t / (GROUP_M * n_tiles);
  const int first_m = band * GROUP_M;
  const int band_m = min(GROUP_M, m_tiles - first_m);
  const int r = t - band * GROUP_M * n_tiles;
  const int q = first_m + r % band_m;  // m-tile
  tile_n = r / band_m;
  tl.n0 = tile_n * GT;
  if constexpr (Kind<KIND>::MRAG) {
    int mt = q;
    int b = clamp_row(a.offsets[0], a.cap);
    for (int g = 0; g < a.n_groups; ++g) {
      int e = clamp_row(a.offsets[g + 1], a.cap);
      if (e < b) e = b;
      const int tiles = (e - b + BM - 1) / BM;
      if (mt < tiles) {
        tl.g = g;
        tl.row0 = b + mt * BM;
        tl.rows = min(BM, e - tl.row0);
        tl.m0 = 0;
        tl.split = 0;
        return;
      }
      mt -= tiles;
      b = e;
    }
    tl.g = 0; tl.row0 = 0; tl.rows = 0; tl.m0 = 0; tl.split = 0;  // not reached for t < count
  } else {
    // (group, split part, m-tile); part p of a group of rows [b, e) is
    // [b + len p / S, b + len (p + 1) / S)
    const int S = max(1, a.ksplit);
    const int mt_per_g = (a.M + BM - 1) / BM;
    const int gs = q / mt_per_g;
    tl.g = gs / S;
    tl.split = gs % S;
    tl.m0 = (q % mt_per_g) * BM;
    const int b = clamp_row(a.offsets[tl.g], a.cap);
    int e = clamp_row(a.offsets[tl.g + 1], a.cap);
    if (e < b) e = b;
    const long len = e - b;
    tl.row0 = b + (int)(len * tl.split / S);
    tl.rows = b + (int)(len * (tl.split + 1) / S) - tl.row0;
  }
}

template <int KIND>
DEVI int col_tiles(const GemmArgs& a) {
  return ((KIND == GU_FWD ? 2 * a.H : a.N) + GT - 1) / GT;
}

// Kernel argument of the bf16 kernel: one or two sets of groups of the same
// GEMM kind (the routed experts and the merged shared experts) in one launch,
// so that the tiles of both fill the CUs together.
struct GemmLaunch {
  GemmArgs s0, s1;
  int n_sets;
  int* counters;  // non-null: per-XCD tile counters (zero at launch) for dynamic dealing
  int* zero;      // block 0 zeroes zero[0..n_zero) (the next launches' counters)
  int n_zero;
};

template <int KIND>
__global__ __launch_bounds__(64 * Cfg<KIND>::NW, Cfg<KIND>::NW / 4) void gemm_bf16_kernel(GemmLaunch L) {
  using K_ = Kind<KIND>;
  using C_ = Cfg<KIND>;
  constexpr int MI = C_::MI, WM = C_::WM, NS = C_::NS, GK = C_::GK, KS = C_::KS;
  __shared__ __attribute__((aligned(1024))) char lds[C_::LDS];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const bf16_t* zero16 = reinterpret_cast<const bf16_t*>(&kZero16);
  // XCD-aware assignment (the grid is a multiple of N_XCD blocks): XCD x takes
  // the x-th eighth of every set's tile range (so each XCD gets an equal share
  // of each set's work), set 0 first.  Its blocks deal these tiles
  // round-robin, or - with counters - each block takes the XCD's next tile
  // when it finishes one (tiles of unequal K then balance across blocks).
  const int per_xcd = gridDim.x / N_XCD;
  const int xcd = blockIdx.x % N_XCD;
  if (L.zero && blockIdx.x == 0 && (int)threadIdx.x < L.n_zero) L.zero[threadIdx.x] = 0;

  const int nt0 = col_tiles<KIND>(L.s0);
  const int mt0 = m_tile_count<KIND>(L.s0);
  const int tot0 = mt0 * nt0;
  const int nt1 = L.n_sets > 1 ? col_tiles<KIND>(L.s1) : 0;
  const int mt1 = L.n_sets > 1 ? m_tile_count<KIND>(L.s1) : 0;
  const int tot1 = mt1 * nt1;
  const int lo0 = (int)((long)tot0 * xcd / N_XCD);
  const int cnt0 = (int)((long)tot0 * (xcd + 1) / N_XCD) - lo0;
  const int lo1 = (int)((long)tot1 * xcd / N_XCD);
  const int cnt1 = (int)((long)tot1 * (xcd + 1) / N_XCD) - lo1;
  const bool dyn = L.counters != nullptr;
  __shared__ int next_tile[2];  // double-buffered broadcast of the dealt tile
  int it_parity = 0;
  int nxt = 0;                  // thread 0: tile prefetched for the next round
  int i;
  if (dyn) {
    if (threadIdx.x == 0) {
      next_tile[0] = atomicAdd(L.counters + xcd, 1);
      nxt = atomicAdd(L.counters + xcd, 1);
    }
    __syncthreads();
    i = next_tile[0];
  } else {
    i = (int)(blockIdx.x / N_XCD);
  }

  while (i < cnt0 + cnt1) {
    const bool second = i >= cnt0;
    GemmArgs a;
    if (second) a = L.s1; else a = L.s0;
    const int t = second ? lo1 + (i - cnt0) : lo0 + i;
    const int m_tiles = second ? mt1 : mt0;
    const int n_tiles = second ? nt1 : nt0;
    Tile tl;
    int tile_n;
    tile_decode<KIND>(a, t, m_tiles, n_tiles, tl, tile_n);
    const bf16_t* A = static_cast<const bf16_t*>(a.A);
    const bf16_t* B = static_cast<const bf16_t*>(a.B) + (K_::MRAG ? (size_t)tl.g * a.b_gs : 0);
    const int Kd = K_::MRAG ? a.K : tl.rows;
    const int nk = (Kd + GK - 1) / GK;
    const int n_full = Kd / GK;  // k-steps without a ragged tail
    const int last_row = tl.row0 + (tl.rows > 0 ? tl.rows - 1 : 0);

    // operand pointers; out-of-range M/N indices are clamped to valid memory
    // (outputs not stored), out-of-range k-rows read zeros
    auto a_row = [&](int r) -> const bf16_t* {  // M-ragged A, k-contiguous
      return A + (size_t)min(tl.row0 + r, last_row) * a.lda;
    };
    auto a_elem = [&](int k, int c) -> const bf16_t* {  // TN A(i = m0 + c, k)
      if (k >= Kd) return zero16;
      const int m = (tl.m0 + c + 8 <= a.M) ? tl.m0 + c : 0;
      return A + (size_t)(tl.row0 + k) * a.lda + m;
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
      if constexpr (K_::MRAG) {
        return B + (size_t)k * a.ldb + n;
      } else {
        if (k >= Kd) return zero16;
        return B + (size_t)(tl.row0 + k) * a.ldb + n;
      }
    };

    // DMA addresses at k-step 0 (k-contiguous operands advance by GK
    // elements, m/n-contiguous ones by GK rows per k-step) and of the ragged
    // tail k-step
    DmaPtrs<C_::DMA_A> da, ta;
    DmaPtrs<C_::DMA_B> db, tb;
    if constexpr (K_::A_KC) dma_kc_init<GK, C_::NW>(da, a_row, wave, A); else dma_mn_init<C_::NW>(da, a_elem, wave, 0, A);
    if constexpr (K_::B_KC) dma_kc_init<GK, C_::NW>(db, b_row, wave, B); else dma_mn_init<C_::NW>(db, b_elem, wave, 0, B);
    if constexpr (!K_::MRAG) {
      dma_mn_init<C_::NW>(ta, a_elem, wave, n_full * GK, A);
      dma_mn_init<C_::NW>(tb, b_elem, wave, n_full * GK, B);
    }
    const u32x4_t rs_a = make_rsrc(A), rs_b = make_rsrc(B);
    const unsigned a_step = 2u * (K_::A_KC ? GK : (unsigned)GK * a.lda);
    const unsigned b_step = 2u * (K_::B_KC ? GK : (unsigned)GK * a.ldb);

    // DMA load i of each operand (A: i < DMA_A, B: i < DMA_B) for k-step ks
    // into stage st
    auto dma = [&](int ks, int st, int i) {
      char* la = lds + st * C_::STAGE;
      const bool tail = !K_::MRAG && ks >= n_full;
      if (i < C_::DMA_A) {
        const int ia = i < C_::DMA_A ? i : 0;
        unsigned pa = da.p[ia] + ks * a_step;
        if constexpr (!K_::MRAG) pa = tail ? ta.p[ia] : pa;
        load_to_lds(rs_a, pa, la + (i * C_::NW + wave) * 1024);
      }
      if (i < C_::DMA_B) {
        const int ib = i < C_::DMA_B ? i : 0;
        unsigned pb = db.p[ib] + ks * b_step;
        if constexpr (!K_::MRAG) pb = tail ? tb.p[ib] : pb;
        load_to_lds(rs_b, pb, la + C_::A_BYTES + (i * C_::NW + wave) * 1024);
      }
    };

    auto read_frag = [&](const char* stage, int s, int idx, bf16x8_t* af, bf16x8_t* bfr) {
      // in the order the next k16-step's MFMAs consume them: idx 0 = A
      // fragment 0, 1..4 = B fragments 0..3, 5.. = A fragments 1..MI-1
      if (idx == 0 || idx > 4) {
        const int f = idx == 0 ? 0 : idx - 4;
        af[f] = K_::A_KC ? frag_kc<GK>(stage, wm * WM + f * 32, s)
                         : frag_mn(stage, wm * WM + f * 32, s);
      } else {
        const int f = idx - 1;
        const char* lb = stage + C_::A_BYTES;
        bfr[f] = K_::B_KC ? frag_kc<GK>(lb, wn * 128 + f * 32, s)
                          : frag_mn(lb, wn * 128 + f * 32, s);
      }
    };

    f32x16_t acc[MI][4];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};

    // One k16-step: 4 MI MFMAs on (A_c, B_c) in 2 MI chunks of two; chunk q
    // also reads fragments [q NF / NQ, (q + 1) NF / NQ) of the next k16-step
    // (NF = MI + 4 of them, from stage_n) into (A_n, B_n) and, for
    // q < DMA_MAX when dma_ks >= 0, issues DMA load q of k-step dma_ks into
    // stage dma_st.  sched_barrier(0) fences keep this order, so each fragment
    // read has a whole k16-step to land and the compiler's waits fall at the
    // first use in the next k16-step.
    constexpr int NQ = 2 * MI, NF = MI + 4;
    static_assert(C_::DMA_MAX <= NQ, "DMA loads per k-step exceed the chunks");
    auto kstep = [&](const bf16x8_t* A_c, const bf16x8_t* B_c, const char* stage_n, int s_n,
                     bf16x8_t* A_n, bf16x8_t* B_n, int dma_ks, int dma_st) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        if (dma_ks >= 0 && q < C_::DMA_MAX) dma(dma_ks, dma_st, q);
#pragma unroll
        for (int f = q * NF / NQ; f < (q + 1) * NF / NQ; ++f) read_frag(stage_n, s_n, f, A_n, B_n);
        const int i = q >> 1, j0 = 2 * (q & 1);
        acc[i][j0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(B_c[j0], A_c[i], acc[i][j0], 0, 0, 0);
        acc[i][j0 + 1] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(B_c[j0 + 1], A_c[i], acc[i][j0 + 1], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    bf16x8_t af0[MI], bf0[4], af1[MI], bf1[4];
    // Only k-steps below nk are loaded: every wait below lets the loads of
    // the real k-steps issued after the one it needs stay in flight, DMA_N
    // per k-step (vector memory loads complete in issue order).
    if (nk > 0) {
#pragma unroll
      for (int p = 0; p < NS; ++p)
        if (p < nk) {
#pragma unroll
          for (int i = 0; i < C_::DMA_MAX; ++i) dma(p, p, i);
        }
      // own DMA of k-step 0 done (k-steps 1 .. min(NS, nk) - 1 may stay in flight)
      wait_vm_groups<C_::DMA_N, NS - 1>(nk - 1);
      __syncthreads();
#pragma unroll
      for (int q = 0; q < NF; ++q) read_frag(lds, 0, q, af0, bf0);
    }
    for (int kt = 0; kt < nk; ++kt) {
      const int st = kt % NS;
      const char* stage = lds + st * C_::STAGE;
      const char* stage_next = lds + ((kt + 1) % NS) * C_::STAGE;
      // k16-steps 0 .. KS-2 read the next fragments from this stage
#pragma unroll
      for (int s = 0; s < KS - 1; ++s) {
        if (s % 2 == 0) kstep(af0, bf0, stage, s + 1, af1, bf1, -1, 0);
        else kstep(af1, bf1, stage, s + 1, af0, bf0, -1, 0);
      }
      WAIT_LGKMCNT(0);
      // k-step kt + 1 landed (kt + 2 .. min(kt + NS, nk) - 1 may stay in flight)
      wait_vm_groups<C_::DMA_N, NS - 2>(nk - 2 - kt);
      __syncthreads();
      // the last one reads k16-step 0 of the next stage and refills this one
      // (with k-step kt + NS if there is one)
      const int refill = kt + NS < nk ? kt + NS : -1;
      if constexpr ((KS - 1) % 2 == 0)
        kstep(af0, bf0, stage_next, 0, af1, bf1, refill, st);
      else
        kstep(af1, bf1, stage_next, 0, af0, bf0, refill, st);
    }
    WAIT_VMCNT(0);  // drain the ring before the next tile

    // epilogue: accumulator (i, j) register 4q + t holds
    //   C[wm*WM + 32i + lane%32][wn*128 + 32j + 8q + 4(lane/32) + t]
    if constexpr (KIND == DWD || KIND == DWGU) {
      // fp32 weight gradient of group g, 16 bytes per lane straight from the
      // accumulators
      const int r_in = lane & 31;
      const int c_in = 4 * (lane >> 5);
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int row = wm * WM + i * 32 + r_in;
        if (tl.m0 + row >= a.M) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int col = tl.n0 + wn * 128 + j * 32 + 8 * q + c_in;
            if (col >= a.N) continue;
            float* c = static_cast<float*>(a.C) + (size_t)tl.g * a.c_gs +
                       (size_t)tl.split * a.c_split + (size_t)(tl.m0 + row) * a.ldc + col;
            f32x4_t o = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                         acc[i][j][4 * q + 3]};
            if (a.accumulate) o += *reinterpret_cast<const f32x4_t*>(c);
            *reinterpret_cast<f32x4_t*>(c) = o;
          }
      }
    } else {
      // bf16 outputs go through LDS so that every global access is a whole
      // 16-byte chunk and a wave instruction covers 256 contiguous bytes of a
      // row (4 rows) instead of 16 bytes of 32 rows.  Each wave transposes its
      // 64 x 128 sub-tile in a private 16 KB region (the drained ring).  The
      // outputs (and the G/U that the dSwiGLU epilogue reads) are touched
      // once here, so they go past the caches (nontemporal: measured 2-4 %
      // faster for DHH_BWD, DX_BWD and DOWN_FWD; the fp32 weight gradients
      // below are not, they were 1.4-1.7x slower that way).
      __syncthreads();  // every wave is done with the ring
      char* reg = lds + wave * C_::EPI_WAVE;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = i * 32 + (lane & 31);
            const int u = 8 * j + 2 * q + (lane >> 5);
            epi_put(reg, row, u, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                    acc[i][j][4 * q + 3]);
          }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // region is wave-private
      const int row_lim = tl.rows - wm * WM;  // rows of this wave's sub-tile to store
      if constexpr (KIND == GU_FWD) {
        // region row: [G h0..31 | U h0..31 | G h32..63 | U h32..63] of the
        // wave's 64 hidden units; lane -> (row, 8 hidden units)
        const int h = tile_n * (GT / 2) + wn * 64 + 32 * ((lane & 7) >> 2) + 8 * (lane & 3);
        const int cg = 8 * ((lane & 7) >> 2) + (lane & 3);
        bf16_t* gu = static_cast<bf16_t*>(a.C);
        bf16_t* hh = static_cast<bf16_t*>(a.out2);
        if (h < a.H) {
#pragma unroll 4
          for (int it = 0; it < WM / 8; ++it) {
            const int row = it * 8 + (lane >> 3);
            if (row >= row_lim) break;
            const bf16x8_t G = epi_get(reg, row, cg);
            const bf16x8_t U = epi_get(reg, row, cg + 4);
            bf16x8_t Hv;
#pragma unroll
            for (int e = 0; e < 8; ++e) Hv[e] = (bf16_t)(silu_fast((float)G[e]) * (float)U[e]);
            const size_t m = (size_t)(tl.row0 + wm * WM + row);
            __builtin_nontemporal_store(G, reinterpret_cast<bf16x8_t*>(gu + m * 2 * a.H + h));
            __builtin_nontemporal_store(U, reinterpret_cast<bf16x8_t*>(gu + m * 2 * a.H + a.H + h));
            __builtin_nontemporal_store(Hv, reinterpret_cast<bf16x8_t*>(hh + m * a.H + h));
          }
        }
      } else {
        const int c = lane & 15;
        const int col = tl.n0 + wn * 128 + 8 * c;
        if (col < a.N) {
          if constexpr (KIND == DHH_BWD) {
            // dG = dHh * U * silu'(G), dU = dHh * silu(G); G and U of a batch of
            // rows are loaded before any store of it
            const bf16_t* gu = static_cast<const bf16_t*>(a.aux);
            bf16_t* dgu = static_cast<bf16_t*>(a.C);
            for (int it0 = 0; it0 < WM / 4; it0 += 8) {
              if (it0 * 4 >= row_lim) break;
              bf16x8_t G[8], U[8];
#pragma unroll
              for (int b = 0; b < 8; ++b) {
                const int row = min((it0 + b) * 4 + (lane >> 4), row_lim - 1);
                const size_t m = (size_t)(tl.row0 + wm * WM + row);
                G[b] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(gu + m * 2 * a.H + col));
                U[b] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(gu + m * 2 * a.H + a.H + col));
              }
#pragma unroll
              for (int b = 0; b < 8; ++b) {
                const int row = (it0 + b) * 4 + (lane >> 4);
                const bf16x8_t v = epi_get(reg, row, c);
                bf16x8_t dG, dU;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                  const float g = (float)G[b][e], dh = (float)v[e];
                  const float s = sigmoid_fast(g);
                  dG[e] = (bf16_t)(dh * (float)U[b][e] * (s * (1.0f + g * (1.0f - s))));
                  dU[e] = (bf16_t)(dh * g * s);
                }
                if (row < row_lim) {
                  const size_t m = (size_t)(tl.row0 + wm * WM + row);
                  __builtin_nontemporal_store(dG, reinterpret_cast<bf16x8_t*>(dgu + m * 2 * a.H + col));
                  __builtin_nontemporal_store(dU, reinterpret_cast<bf16x8_t*>(dgu + m * 2 * a.H + a.H + col));
                }
              }
            }
          } else if constexpr (KIND == DH_BWD) {
            // dA = dHh * silu'(A); A of a batch of rows is loaded before any
            // store of it
            const bf16_t* Ab = static_cast<const bf16_t*>(a.aux);
            bf16_t* C = static_cast<bf16_t*>(a.C);
            for (int it0 = 0; it0 < WM / 4; it0 += 8) {
              if (it0 * 4 >= row_lim) break;
              bf16x8_t Av[8];
#pragma unroll
              for (int b = 0; b < 8; ++b) {
                const int row = min((it0 + b) * 4 + (lane >> 4), row_lim - 1);
                Av[b] = *reinterpret_cast<const bf16x8_t*>(
                    Ab + (size_t)(tl.row0 + wm * WM + row) * a.H + col);
              }
#pragma unroll
              for (int b = 0; b < 8; ++b) {
                const int row = (it0 + b) * 4 + (lane >> 4);
                const bf16x8_t v = epi_get(reg, row, c);
                bf16x8_t dA;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                  const float g = (float)Av[b][e];
                  const float sg = sigmoid_fast(g);
                  dA[e] = (bf16_t)((float)v[e] * (sg * (1.0f + g * (1.0f - sg))));
                }
                if (row < row_lim)
                  __builtin_nontemporal_store(dA, reinterpret_cast<bf16x8_t*>(C + (size_t)(tl.row0 + wm * WM + row) * a.ldc + col));
              }
            }
          } else if constexpr (KIND == UP_FWD) {
            // A and h = silu(A) (of the bf16-rounded A)
            bf16_t* C = static_cast<bf16_t*>(a.C);
            bf16_t* hh = static_cast<bf16_t*>(a.out2);
#pragma unroll 8
            for (int it = 0; it < WM / 4; ++it) {
              const int row = it * 4 + (lane >> 4);
              if (row >= row_lim) break;
              const bf16x8_t A = epi_get(reg, row, c);
              bf16x8_t Hv;
#pragma unroll
              for (int e = 0; e < 8; ++e) Hv[e] = (bf16_t)silu_fast((float)A[e]);
              const size_t m = (size_t)(tl.row0 + wm * WM + row);
              __builtin_nontemporal_store(A, reinterpret_cast<bf16x8_t*>(C + m * a.ldc + col));
              __builtin_nontemporal_store(Hv, reinterpret_cast<bf16x8_t*>(hh + m * a.H + col));
            }
          } else {  // DOWN_FWD / DX_BWD
            bf16_t* C = static_cast<bf16_t*>(a.C);
#pragma unroll 8
            for (int it = 0; it < WM / 4; ++it) {
              const int row = it * 4 + (lane >> 4);
              if (row >= row_lim) break;
              __builtin_nontemporal_store(epi_get(reg, row, c), reinterpret_cast<bf16x8_t*>(C + (size_t)(tl.row0 + wm * WM + row) * a.ldc + col));
            }
          }
        }
      }
    }
    // next tile: the prefetched counter value (dynamic) or the next stride
    if (dyn) {
      it_parity ^= 1;
      if (threadIdx.x == 0) {
        next_tile[it_parity] = nxt;
        if (nxt < cnt0 + cnt1) nxt = atomicAdd(L.counters + xcd, 1);
      }
    }
    __syncthreads();  // LDS is reused by the next tile
    i = dyn ? next_tile[it_parity] : i + per_xcd;
  }
}

int num_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <int KIND>
long max_tiles(const GemmArgs& a) {
  constexpr int BM = Cfg<KIND>::BM;
  const long n_tiles = ceil_div((KIND == GU_FWD) ? 2 * a.H : a.N, GT);
  return Kind<KIND>::MRAG ? (ceil_div(a.cap, BM) + (long)a.n_groups) * n_tiles
                          : (long)a.n_groups * std::max(1, a.ksplit) * ceil_div(a.M, BM) * n_tiles;
}

constexpr const char* kGemmNames[] = {"gemm_gu_fwd", "gemm_down_fwd", "gemm_dhh_bwd",
                                      "gemm_dx_bwd", "gemm_dwd", "gemm_dwgu",
                                      "gemm_up_fwd", "gemm_dh_bwd"};

// One launch over the sets sets[0..n_sets) (at most 2) of one GEMM kind.
// counters (bf16 only): zeroed per-XCD tile counters for dynamic dealing;
// zero[0..n_zero): words the launch's block 0 clears for later launches (the
// launch then runs even without tiles).
template <int KIND>
hipError_t run_gemm(const GemmArgs* sets, int n_sets, int bf16, hipStream_t s,
                    int* counters = nullptr, int* zero = nullptr, int n_zero = 0) {
  if (bf16) {
    // persistent: at most one block per CU, a multiple of N_XCD blocks
    GemmLaunch L{};
    L.s0 = sets[0];
    L.n_sets = n_sets;
    // dynamic dealing: the set with the longer reduction per tile goes first,
    // so that its tiles do not start last
    auto k_per_tile = [](const GemmArgs& a) -> long {
      return Kind<KIND>::MRAG ? a.K
                              : a.cap / std::max(1, a.n_groups) / std::max(1, a.ksplit);
    };
    const bool swap = counters && n_sets > 1 && k_per_tile(sets[1]) > k_per_tile(sets[0]);
    L.counters = counters;
    L.zero = zero;
    L.n_zero = n_zero;
    long tiles = max_tiles<KIND>(sets[0]);
    if (n_sets > 1) {
      L.s1 = sets[1];
      tiles += max_tiles<KIND>(sets[1]);
      if (swap) std::swap(L.s0, L.s1);
    }
    if (tiles == 0 && n_zero == 0) return hipSuccess;
    long blocks = std::min<long>((long)num_cus(), std::max<long>(tiles, 1));
    blocks = std::max<long>(N_XCD, (blocks + N_XCD - 1) / N_XCD * N_XCD);
    MOE_TIMED(kGemmNames[KIND], s, gemm_bf16_kernel<KIND><<<(int)blocks, 64 * Cfg<KIND>::NW, 0, s>>>(L));
    return hipGetLastError();
  }
  for (int i = 0; i < n_sets; ++i) {
    const GemmArgs& a = sets[i];
    dim3 grid;
    grid.x = ceil_div((KIND == GU_FWD) ? 2 * a.H : a.N, 64);
    if (Kind<KIND>::MRAG) {
      grid.y = ceil_div(a.cap, 64) + a.n_groups;
      grid.z = 1;
    } else {
      grid.y = ceil_div(a.M, 64);
      grid.z = a.n_groups;
    }
    if (grid.x == 0 || grid.y == 0 || grid.z == 0) continue;
    MOE_TIMED(kGemmNames[KIND], s, gemm_f32_kernel<KIND><<<grid, 256, 0, s>>>(a));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// dst[i] = (accumulate ? dst[i] : 0) + p_0[i] + p_1[i] + ... (fixed order),
// n % 4 == 0, all 16-byte aligned; the partials are read once and dst is
// written once, both past the caches (nontemporal)
__global__ __launch_bounds__(256) void splitk_reduce_kernel(float* dst, const float* parts,
                                                            int n_parts, size_t n,
                                                            int accumulate) {
  const size_t n4 = n / 4;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    f32x4_t q[4];  // all loads first (n_parts <= 4)
#pragma unroll
    for (int p = 0; p < 4; ++p)
      if (p < n_parts) q[p] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(parts + p * n) + i);
    f32x4_t v = accumulate ? reinterpret_cast<const f32x4_t*>(dst)[i] : f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < 4; ++p)
      if (p < n_parts) v += q[p];
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t*>(dst) + i);
  }
}

// Split-K factor of a K-ragged (weight-gradient) GEMM of one set: a single
// large group whose M x N tiles cannot fill the CUs (the merged shared
// experts: one group over all T tokens) is cut into parts of its rows, each
// part writing its own fp32 partial, summed afterwards in a fixed order.
int ksplit_factor(int bf16, long M, long N, const moe_ffn_set& f) {
  if (!bf16 || f.n_groups != 1 || f.cap < 4096) return 1;
  const long tiles = ceil_div((int)M, GT) * (long)ceil_div((int)N, GT);
  const long sp = num_cus() / std::max<long>(tiles, 1);
  return (int)std::max<long>(1, std::min<long>(4, sp));
}

constexpr size_t kWsAlign = 256;
constexpr int kCounterWords = 2 * N_XCD;  // DWD then DWGU per-XCD counters
size_t align_up(size_t v) { return (v + kWsAlign - 1) / kWsAlign * kWsAlign; }

}  // namespace

// Rows of an expert's first weight per hidden unit: 2 (gate and up) for
// SwiGLU, 1 for the SiLU expert.
long first_rows(const moe_ffn_set& f) { return f.activation == MOE_ACT_SILU ? 1 : 2; }

size_t ffn_bwd_ws_bytes(const moe_ffn_set* sets, int n_sets, int bf16, int d) {
  size_t bytes = align_up(kCounterWords * sizeof(int));
  for (int i = 0; i < n_sets; ++i) {
    const moe_ffn_set& f = sets[i];
    const long H = f.H, R1 = first_rows(f);
    const int s_wd = ksplit_factor(bf16, d, H, f);
    const int s_wgu = ksplit_factor(bf16, R1 * H, d, f);
    if (s_wd > 1) bytes += align_up((size_t)s_wd * d * H * sizeof(float));
    if (s_wgu > 1) bytes += align_up((size_t)s_wgu * R1 * H * d * sizeof(float));
  }
  return bytes;
}

hipError_t launch_ffn_fwd_sets(const moe_ffn_set* sets, int n_sets, int bf16, int d,
                               hipStream_t s) {
  GemmArgs g[2]{}, o[2]{};
  const bool silu = sets[0].activation == MOE_ACT_SILU;  // the same for every set
  for (int i = 0; i < n_sets; ++i) {
    const moe_ffn_set& f = sets[i];
    const long R1 = first_rows(f);
    // [G|U] = X [Wg;Wu]^T with the SwiGLU epilogue, or A = X W1^T with SiLU
    GemmArgs& a = g[i];
    a.offsets = f.offsets; a.n_groups = f.n_groups; a.cap = f.cap; a.H = f.H;
    a.A = f.xp; a.lda = d;
    a.B = f.w_gate_up; a.ldb = d; a.b_gs = R1 * f.H * d;
    a.C = f.gu; a.ldc = R1 * f.H; a.out2 = f.h;
    a.N = (int)(R1 * f.H); a.K = d;
    // Y = Hh Wd^T
    GemmArgs& b = o[i];
    b.offsets = f.offsets; b.n_groups = f.n_groups; b.cap = f.cap; b.H = f.H;
    b.A = f.h; b.lda = f.H;
    b.B = f.w_down; b.ldb = f.H; b.b_gs = (long)d * f.H;
    b.C = f.yp; b.ldc = d;
    b.N = d; b.K = f.H;
  }
  hipError_t e = silu ? run_gemm<UP_FWD>(g, n_sets, bf16, s) : run_gemm<GU_FWD>(g, n_sets, bf16, s);
  if (e != hipSuccess) return e;
  return run_gemm<DOWN_FWD>(o, n_sets, bf16, s);
}

hipError_t launch_ffn_bwd_sets(const moe_ffn_set* sets, int n_sets, int bf16, int d,
                               int accumulate_dw, void* ws, hipStream_t s) {
  GemmArgs hh[2]{}, dx[2]{}, wd[2]{}, wgu[2]{};
  // workspace: per-XCD counters, then the split-K partials
  int* counters = static_cast<int*>(ws);
  char* part = static_cast<char*>(ws) + (ws ? align_up(kCounterWords * sizeof(int)) : 0);
  struct Reduce { float* dst; const float* parts; int n_parts; size_t n; };
  Reduce red[4];
  int n_red = 0;
  const bool silu = sets[0].activation == MOE_ACT_SILU;  // the same for every set
  for (int i = 0; i < n_sets; ++i) {
    const moe_ffn_set& f = sets[i];
    const long H = f.H, R1 = first_rows(f);
    GemmArgs base{};
    base.offsets = f.offsets; base.n_groups = f.n_groups; base.cap = f.cap; base.H = f.H;
    base.accumulate = accumulate_dw;
    // dHh = dY Wd, epilogue -> [dG | dU] (SwiGLU) or dA (SiLU)
    GemmArgs& a = hh[i] = base;
    a.A = f.dyp; a.lda = d;
    a.B = f.w_down; a.ldb = H; a.b_gs = (long)d * H;
    a.C = f.dgu; a.ldc = R1 * H; a.aux = f.gu;
    a.N = f.H; a.K = d;
    // dX = [dG|dU] [Wg;Wu]  (SiLU: dA W1)
    GemmArgs& b = dx[i] = base;
    b.A = f.dgu; b.lda = R1 * H;
    b.B = f.w_gate_up; b.ldb = d; b.b_gs = R1 * H * d;
    b.C = f.dxp; b.ldc = d;
    b.N = d; b.K = (int)(R1 * f.H);
    // dWd[g] = dY^T Hh
    GemmArgs& c = wd[i] = base;
    c.A = f.dyp; c.lda = d;
    c.B = f.h; c.ldb = H;
    c.C = f.dw_down; c.ldc = H; c.c_gs = (long)d * H;
    c.M = d; c.N = f.H;
    // dWgu[g] = [dG|dU]^T X  (SiLU: dW1 = dA^T X)
    GemmArgs& w = wgu[i] = base;
    w.A = f.dgu; w.lda = R1 * H;
    w.B = f.xp; w.ldb = d;
    w.C = f.dw_gate_up; w.ldc = d; w.c_gs = R1 * H * d;
    w.M = (int)(R1 * f.H); w.N = d;
    if (ws) {
      for (GemmArgs* g : {&c, &w}) {
        const int S = ksplit_factor(bf16, g->M, g->N, f);
        if (S <= 1) continue;
        const size_t n = (size_t)g->M * g->N;
        red[n_red++] = Reduce{static_cast<float*>(g->C), reinterpret_cast<const float*>(part), S, n};
        g->C = part;
        g->ksplit = S;
        g->c_split = (long)n;
        g->accumulate = 0;
        part += align_up((size_t)S * n * sizeof(float));
      }
    }
  }
  hipError_t e;
  // the first launch clears the counters of the two weight-gradient launches
  e = silu ? run_gemm<DH_BWD>(hh, n_sets, bf16, s, nullptr, ws ? counters : nullptr,
                              ws ? kCounterWords : 0)
           : run_gemm<DHH_BWD>(hh, n_sets, bf16, s, nullptr, ws ? counters : nullptr,
                               ws ? kCounterWords : 0);
  if (e != hipSuccess) return e;
  if ((e = run_gemm<DX_BWD>(dx, n_sets, bf16, s)) != hipSuccess) return e;
  if ((e = run_gemm<DWD>(wd, n_sets, bf16, s, ws ? counters : nullptr)) != hipSuccess) return e;
  if ((e = run_gemm<DWGU>(wgu, n_sets, bf16, s, ws ? counters + N_XCD : nullptr)) != hipSuccess)
    return e;
  for (int r = 0; r < n_red; ++r) {
    const int blocks = (int)std::min<size_t>(8192, (red[r].n / 4 + 255) / 256);
    MOE_TIMED("splitk_reduce", s,
              splitk_reduce_kernel<<<std::max(blocks, 1), 256, 0, s>>>(
                  red[r].dst, red[r].parts, red[r].n_parts, red[r].n, accumulate_dw));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace moe
