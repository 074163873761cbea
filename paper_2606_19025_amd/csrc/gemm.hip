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
// bf16: v_mfma_f32_16x16x32_bf16 with fp32 accumulation in a persistent
// kernel with 256 x 256 block tiles of 8 waves fed from an LDS ring by
// global -> LDS DMA (details at gemm_bf16_kernel and Cfg).  One launch
// covers up to two expert sets (routed and shared experts) of one kind, or
// in the backward two independent kinds (dHh with dW_d, dX with dW_gu).
// fp32: a plain 64x64 SIMT tile (4x4 outputs per thread) with the same
// epilogues; used for fp32 layers.
#include <type_traits>

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
  long c_split;     // stride (elements) between the split-K partial outputs
  int n_groups, cap, M, N, K, H, accumulate;
  int ksplit;       // K-ragged kinds: each group's rows split in ksplit parts (0 = 1)
  // DOWN_FWD and DX_BWD (bf16): the kernel may cut K into up to ksplit_max
  // parts (its choice from the device-side group sizes); part p's fp32
  // partial goes to part + p c_split ([cap, N] each) and the choice to
  // *ksplit_used, for splitk_rows_reduce_kernel.  ksplit_max <= 1: no split.
  int ksplit_max;
  float* part;
  int* ksplit_used;
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
// Persistent: one 512-thread block per CU loops over output tiles, of up to
// two GEMM kinds KA and KB (GemmLaunch).  Block tile 256 x 256; the 8 waves
// (two per SIMD) form a 4 x 2 grid and each owns a 64 x 128 sub-tile = 4 x 8
// v_mfma_f32_16x16x32_bf16 tiles (128 fp32 accumulators per lane).
//
// Operands stream through a ring of NS LDS stages of one k-step (GK) each,
// filled with 16-byte global -> LDS DMA: M-ragged kinds NS = 2 stages of
// GK = 64 (64 KB each), weight-gradient kinds NS = 4 stages of GK = 32
// (32 KB each).  A k-step is GK / 32 k32-steps; a k32-step is 8 chunks of 4
// MFMAs (k32step).  The last k32-step of k-step kt waits for the wave's DMA
// of k-step kt+1 (vmcnt leaves the later k-steps' loads in flight), takes the
// barrier after which stage kt is free, and refills it with k-step kt+NS (if
// the tile has one).
//
// Tile order (see tile_decode): bands of GROUP_M m-tiles (2 to 8, per kind,
// see Cfg).  Each XCD takes an equal share of every set's tile range (blocks
// are placed on the 8 XCDs round-robin by id): the 32 tiles an XCD runs at a
// time form a band rectangle whose operand panels its L2 serves.  With
// counters the blocks of an XCD take its tiles one at a time.  Output tiles
// end in an epilogue: bf16 results are staged through a wave-private region
// of the ring so global accesses are whole 16-byte chunks; fp32 weight
// gradients and K-part partials are stored (or added) straight from the
// accumulators.
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
// The MFMA is issued with the B fragment as its first operand, so for each
// 16 x 16 tile lane l accumulates C[m0 + l%16][n0 + 4(l/16) + t] in register
// t: four consecutive output columns per lane.
// Out-of-range M/N rows are clamped to valid memory (their outputs are not
// stored); k-rows past a group's last row (ragged K) are loaded with an
// offset past the buffer resource's range, which reads zeros, so they
// contribute exactly 0.

constexpr int GT = 256;                     // block tile width (N), and height (M) of full tiles
constexpr int N_XCD = 8;

// Tile configuration per kind.  Every kind runs 256 x 256 block tiles with 8
// waves (two per SIMD), one block per CU; each wave owns 64 x 128 of the tile
// (4 x 8 MFMA tiles of 16 x 16, 128 accumulators).  Measured on the fine-grained
// workload against 4 waves of 128 x 128 (one per SIMD, 256 accumulators in
// AGPRs): every launch 6-12 % faster; and against 128 x 256 tiles at
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
  static constexpr int K32 = GK / 32;              // k32-steps per k-step
  static constexpr int BM = GT;                    // block tile rows
  static constexpr int WM = BM / (NW / 2);         // wave sub-tile rows (64)
  static constexpr int MI = WM / 16;               // 16-row MFMA tiles per wave
  static constexpr int NJ = 128 / 16;              // 16-column MFMA tiles per wave
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
  // fine-grained workload (bands of 1, 2, 4, 8 and 16 tried)
  static constexpr int GROUP = KIND == DOWN_FWD || KIND == DX_BWD ? 8 : 2;
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
// 16-byte (b128) or 8-byte store through a buffer resource; an offset at or
// past the resource's record count is dropped, so every lane issues the
// store and the count of outstanding vector memory operations is known at
// compile time.  nt: past the caches (outputs touched once).
template <bool NT>
DEVI void store16(__amdgpu_buffer_rsrc_t r, unsigned off, u32x4_t v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, NT ? 2 : 0);
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
  // the resource is wave-uniform; readfirstlane keeps it in SGPRs after the
  // tile context has passed through registers the compiler treats as per-lane
#pragma unroll
  for (int w = 0; w < 4; ++w) rsrc[w] = __builtin_amdgcn_readfirstlane(rsrc[w]);
  asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(off), "s"(rsrc), "s"(m0)
               : "m0", "memory");
}
// Raw buffer resource over [base, base + kOOB): stride 0, no swizzle, word 3
// the gfx9 default data format.  Every operand stays below kOOB bytes (the
// entry points reject larger ones).
constexpr unsigned kOOB = 0xFFFFFFF0u;
// The same resource for the epilogue's buffer stores.
DEVI __amdgpu_buffer_rsrc_t store_rsrc(void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)kOOB, 0x00020000);
}
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

// m/n-contiguous layout: row k holds 256 m (512 B) in 32-byte chunks; chunk c
// sits at position c ^ mn_swz(k), so that the 8 rows (k0..k0+3 and
// k0+8..k0+11) a half-wave of transposing fragment reads touches fall on 8
// distinct 32-byte bank groups.
DEVI int mn_swz(int k) { return (2 * (k & 3)) ^ ((k >> 3) & 1); }

template <int NW>
DEVI int mn_row(int i, int w) { return (i * NW + w) * 2 + ((threadIdx.x & 63) >> 5); }
// source column of the 16-byte LDS slot this lane writes in row `row`
DEVI int mn_col(int row) {
  const int ps = threadIdx.x & 31;
  return (((ps >> 1) ^ mn_swz(row)) * 16) + (ps & 1) * 8;
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

// MFMA 16x16x32 operand fragment of rows/cols [mb, mb+16) at k32-step s:
// lane l holds index mb + l%16 and k = 32 s + 8 (l/16) + 0..7.
// k-contiguous layout: one 16-byte read (16-byte chunk 4 s + l/16 of the row)
template <int GK>
DEVI bf16x8_t frag_kc(const char* lds_op, int mb, int s) {
  const int lane = threadIdx.x & 63;
  const int row = mb + (lane & 15);
  const int kc = s * 4 + (lane >> 4);
  return *reinterpret_cast<const bf16x8_t*>(lds_op + row * (GK * 2) +
                                            ((kc ^ kc_swz<GK>(row)) << 4));
}

// the same fragment from the m/n-contiguous layout with two transposing
// reads: in each 16-lane group g, lane i points at row k0 + i/4 (k0 = 32 s +
// 8 g + 4 h) and columns mb + 4 (i%4) .. +3, and receives column mb + i of
// rows k0 .. k0+3
DEVI bf16x8_t frag_mn(const char* lds_op, int mb, int s) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, i = lane & 15;
  const int mn = mb + 4 * (i & 3);
  s16x4_t v[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = s * 32 + 8 * g + 4 * h + (i >> 2);
    const int pc = (mn >> 4) ^ mn_swz(k);
    const char* p = lds_op + k * 512 + pc * 32 + (mn & 15) * 2;
    v[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p));
  }
  // whole-vector concatenation (element-wise inserts of bit-cast lanes were
  // mis-generated into a splat of element 0)
  const s16x8_t both = __builtin_shufflevector(v[0], v[1], 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8_t, both);
}

// Epilogue staging.  A wave's 64 x 128 bf16 sub-tile occupies 64 rows of
// 256 B.  The 8-byte unit u (4 columns) of row r sits at unit u ^ epi_key(r),
// epi_key(r) = 2 f(r mod 16) with f a bijection of 0..15 (bits b3 b2 b1 b0 of
// r -> b3 b0 b2 b1).  The accumulator writes (16 rows x units 4j, 4j+1 per
// half-wave) hit 32 distinct bank pairs because the keys are 16 distinct even
// values; a 16-byte chunk c reads back whole from chunk c ^ (key >> 1); and
// rows 2m, 2m+1 differ in key bit 3, so the SwiGLU reads (chunks 0-3 and 8-11
// of two rows per 16 lanes) fall on disjoint chunks.
DEVI int epi_key(int r) { return 2 * ((r & 8) | ((r & 1) << 2) | ((r >> 1) & 3)); }

DEVI void epi_put(char* reg, int row, int u, float v0, float v1, float v2, float v3) {
  bf16x4_t o = {(bf16_t)v0, (bf16_t)v1, (bf16_t)v2, (bf16_t)v3};
  *reinterpret_cast<bf16x4_t*>(reg + row * 256 + ((u ^ epi_key(row)) << 3)) = o;
}

DEVI bf16x8_t epi_get(const char* reg, int row, int c) {
  const int key = epi_key(row);
  return *reinterpret_cast<const bf16x8_t*>(reg + row * 256 + ((c ^ (key >> 1)) << 4));
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

// Group table of one set, staged in LDS once per block: the group offsets
// clamped to [0, cap] (c), their running maximum (b: group g of an M-ragged
// kind is rows [b[g], b[g+1])) and the number of m-tiles before group g (p).
constexpr int kMaxGroups = 256;
struct GroupTable {
  int c[kMaxGroups + 1], b[kMaxGroups + 1], p[kMaxGroups + 1];
};

DEVI int wave_incl_max(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v = max(v, u);
  }
  return v;
}
DEVI int wave_incl_sum(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

// Fill t from set a (one wave; n_groups <= kMaxGroups).
DEVI void build_group_table(const GemmArgs& a, GroupTable& t) {
  const int lane = threadIdx.x & 63;
  const int ng = a.n_groups;
  int run = 0;
  for (int g0 = 0; g0 <= ng; g0 += 64) {
    const int g = g0 + lane;
    const int c = g <= ng ? clamp_row(a.offsets[g], a.cap) : 0;
    int m = wave_incl_max(g <= ng ? c : 0);
    if (g0 > 0) m = max(m, run);
    if (g <= ng) {
      t.c[g] = c;
      t.b[g] = m;
    }
    run = __shfl(m, 63, 64);
  }
  WAIT_LGKMCNT(0);  // the wave's own table writes (lanes read their neighbours')
  int acc = 0;
  for (int g0 = 0; g0 <= ng; g0 += 64) {
    const int g = g0 + lane;
    const int tiles = g < ng ? (t.b[g + 1] - t.b[g] + GT - 1) / GT : 0;
    const int inc = wave_incl_sum(tiles);
    if (g <= ng) t.p[g] = acc + inc - tiles;
    acc += __shfl(inc, 63, 64);
  }
}

// Output tiles form an m_tiles x n_tiles grid (M-ragged kinds: m-tiles of all
// groups in group order; K-ragged kinds: (group, split part, m-tile)
// triples).
template <int KIND>
DEVI int m_tile_count(const GemmArgs& a, const GroupTable& t) {
  constexpr int BM = Cfg<KIND>::BM;
  if constexpr (Kind<KIND>::MRAG) {
    return t.p[a.n_groups];
  } else {
    return a.n_groups * max(1, a.ksplit) * ((a.M + BM - 1) / BM);
  }
}

// Linear tile t walks bands of GROUP_M m-tiles: inside a band m varies
// fastest, then n, so any 32 consecutive tiles cover a GROUP_M x
// (32 / GROUP_M) rectangle and share GROUP_M A panels and 32 / GROUP_M B
// panels in L2.  The m-tile's group is found by all lanes of the wave at once
// (the number of groups whose m-tiles all lie before it).
// M-ragged kinds cut into `parts` K parts: m_tiles counts (m-tile, part)
// pairs, part fastest.
template <int KIND>
DEVI void tile_decode(const GemmArgs& a, const GroupTable& gt, int t, int m_tiles, int n_tiles,
                      int parts, Tile& tl, int& tile_n) {
  constexpr int BM = Cfg<KIND>::BM, GROUP_M = Cfg<KIND>::GROUP;
  const int band = t / (GROUP_M * n_tiles);
  const int first_m = band * GROUP_M;
  const int band_m = min(GROUP_M, m_tiles - first_m);
  const int r = t - band * GROUP_M * n_tiles;
  int q = first_m + r % band_m;  // m-tile (and part)
  tile_n = r / band_m;
  tl.n0 = tile_n * GT;
  if constexpr (Kind<KIND>::MRAG) {
    const int part = q % parts;
    q /= parts;
    const int lane = threadIdx.x & 63;
    int g = 0;
    for (int g0 = 0; g0 < a.n_groups; g0 += 64) {
      const int gg = g0 + lane;
      g += __builtin_popcountll(__ballot(gg < a.n_groups && gt.p[gg + 1] <= q));
    }
    g = __builtin_amdgcn_readfirstlane(g);
    tl.g = g;
    tl.row0 = gt.b[g] + (q - gt.p[g]) * BM;
    tl.rows = min(BM, gt.b[g + 1] - tl.row0);
    tl.m0 = 0;
    tl.split = part;
  } else {
    // (group, split part, m-tile); part p of a group of rows [b, e) is
    // [b + len p / S, b + len (p + 1) / S)
    const int S = max(1, a.ksplit);
    const int mt_per_g = (a.M + BM - 1) / BM;
    const int gs = q / mt_per_g;
    tl.g = gs / S;
    tl.split = gs % S;
    tl.m0 = (q % mt_per_g) * BM;
    const int b = gt.c[tl.g];
    int e = gt.c[tl.g + 1];
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

// Kernel argument of the bf16 kernel: up to kMaxSets sets of groups, each of
// GEMM kind KA or KB (kind_b[s] != 0), whose tiles share one persistent
// launch - the routed and the merged shared experts of one kind, and in the
// backward two independent kinds (dHh with dW_d, dX with dW_gu), so that
// tiles of different lengths fill the CUs together, keep the CUs out of step
// (their epilogue stores do not all fall at once) and fill each other's last
// round.
constexpr int kMaxSets = 4;
struct GemmLaunch {
  GemmArgs s[kMaxSets];
  int kind_b[kMaxSets];
  int n_sets;
  int* counters;  // non-null: per-XCD tile counters (zero at launch) for dynamic dealing
};

template <int K>
using KindTag = std::integral_constant<int, K>;

// One output tile: its decode and the operands' DMA addressing (the first
// DMA_A / DMA_B entries are used; the tail entries by the K-ragged kinds).
struct TileCtx {
  int set;
  bool kb;  // of kind KB
  Tile tl;
  int tile_n, nk, n_full;
  int parts;  // K parts of an M-ragged tile (1: whole K, bf16 output)
  unsigned a_step, b_step;
  u32x4_t rs_a, rs_b;
  DmaPtrs<4> da, db;
  DmaPtrs<2> ta, tb;
};

template <int KA, int KB>
__global__ __launch_bounds__(512, 2) void gemm_bf16_kernel(GemmLaunch L) {
  static_assert(Cfg<KA>::NW == 8 && Cfg<KB>::NW == 8, "8 waves per block");
  static_assert(Cfg<KA>::LDS == Cfg<KB>::LDS, "one LDS ring size per launch");
  constexpr int NW = 8, MI = Cfg<KA>::MI, NJ = Cfg<KA>::NJ, WM = Cfg<KA>::WM;
  __shared__ __attribute__((aligned(1024))) char lds[Cfg<KA>::LDS];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const bf16_t* zero16 = reinterpret_cast<const bf16_t*>(&kZero16);

  // runs f(KindTag<K>) for the kind of a set
  auto for_kind = [&](bool kb, auto&& f) {
    if constexpr (KA == KB) {
      f(KindTag<KA>{});
    } else {
      if (kb) f(KindTag<KB>{});
      else f(KindTag<KA>{});
    }
  };

  // XCD-aware assignment (the grid is a multiple of N_XCD blocks): XCD x takes
  // the x-th eighth of every set's tile range (so each XCD gets an equal share
  // of each set's work), in set order.  Its blocks deal these tiles
  // round-robin, or - with counters - each block takes the XCD's next tile
  // when it finishes one (tiles of unequal K then balance across blocks).
  const int per_xcd = gridDim.x / N_XCD;
  const int xcd = blockIdx.x % N_XCD;
  __shared__ GroupTable gtab[kMaxSets];
  if (wave < L.n_sets) build_group_table(L.s[wave], gtab[wave]);
  __syncthreads();
  // per set: m-tiles, n-tiles, this XCD's first tile and its reduction
  // length per tile (rows per group for the K-ragged kinds, from the table)
  int mt[kMaxSets], ntl[kMaxSets], lo[kMaxSets], cnt[kMaxSets], kpt[kMaxSets], prt[kMaxSets];
  long work = 0;  // sum over tiles of their reduction lengths
#pragma unroll
  for (int q = 0; q < kMaxSets; ++q) {
    mt[q] = ntl[q] = kpt[q] = 0;
    prt[q] = 1;
    if (q < L.n_sets) {
      for_kind(L.kind_b[q] != 0, [&](auto kc) {
        constexpr int KIND = decltype(kc)::value;
        const GemmArgs& a = L.s[q];
        ntl[q] = col_tiles<KIND>(a);
        mt[q] = __builtin_amdgcn_readfirstlane(m_tile_count<KIND>(a, gtab[q]));
        kpt[q] = Kind<KIND>::MRAG
                     ? a.K
                     : __builtin_amdgcn_readfirstlane(gtab[q].b[a.n_groups] - gtab[q].b[0]) /
                           max(1, a.n_groups) / max(1, a.ksplit);
      });
      work += (long)mt[q] * ntl[q] * kpt[q];
    }
  }
  // K parts of the linear M-ragged kinds: a tile whose reduction is longer
  // than 4/3 of the launch's average load per block (work / blocks) would
  // finish last with most CUs idle (few tiles: small groups, narrow N), so it
  // is cut into parts of about that length (at most ksplit_max, at least two
  // k-steps each): the parts then fill about three quarters of the blocks.
  // (Filling all of them was slower: each part writes a whole fp32 partial
  // tile, and more parts moved more bytes than they saved in time.)  Every
  // block derives the same choice from the group table.
#pragma unroll
  for (int q = 0; q < kMaxSets; ++q) {
    if (q < L.n_sets && L.s[q].ksplit_max > 1) {
      for_kind(L.kind_b[q] != 0, [&](auto kc) {
        constexpr int KIND = decltype(kc)::value;
        if constexpr (KIND == DOWN_FWD || KIND == DX_BWD) {
          const GemmArgs& a = L.s[q];
          const long want = work > 0 ? ((long)a.K * gridDim.x * 3 / 4 + work - 1) / work : 1;
          const int most = max(1, a.K / (2 * Cfg<KIND>::GK));
          prt[q] = (int)max(1L, min(want, (long)min(a.ksplit_max, most)));
          prt[q] = __builtin_amdgcn_readfirstlane(prt[q]);
          kpt[q] = a.K / prt[q];
          if (blockIdx.x == 0 && threadIdx.x == 0) *a.ksplit_used = prt[q];
        }
      });
    }
  }
#pragma unroll
  for (int q = 0; q < kMaxSets; ++q) {
    const int tot = q < L.n_sets ? mt[q] * prt[q] * ntl[q] : 0;
    lo[q] = (int)((long)tot * xcd / N_XCD);
    cnt[q] = (int)((long)tot * (xcd + 1) / N_XCD) - lo[q];
  }
  // dealing order of the sets: with dynamic dealing the longest reduction per
  // tile first (so that long tiles do not start last and short ones fill the
  // last round), otherwise as given.  rank[q] = position of set q (stable);
  // pre[p] = first tile of position p.  (Indices stay compile-time constants:
  // runtime indexing of these arrays would move them to scratch memory.)
  int rank[kMaxSets], pre[kMaxSets + 1];
#pragma unroll
  for (int q = 0; q < kMaxSets; ++q) {
    rank[q] = q;
    if constexpr (KA != KB) {  // the single-kind launches keep the given order
      if (L.counters) {
        rank[q] = 0;
#pragma unroll
        for (int r = 0; r < kMaxSets; ++r)
          if (r != q && (kpt[r] > kpt[q] || (kpt[r] == kpt[q] && r < q))) ++rank[q];
      }
    }
  }
  pre[0] = 0;
#pragma unroll
  for (int p = 0; p < kMaxSets; ++p) {
    int c = 0;
#pragma unroll
    for (int q = 0; q < kMaxSets; ++q)
      if (rank[q] == p) c = cnt[q];
    pre[p + 1] = pre[p] + c;
  }
  const int total = pre[kMaxSets];
  const bool dyn = L.counters != nullptr;
  __shared__ int next_tile[2];  // double-buffered broadcast of the dealt tile
  int it_parity = 0;
  int nxt = 0;                  // thread 0: the block's next tile
  int i;
  if (dyn) {
    if (threadIdx.x == 0) {
      next_tile[0] = atomicAdd(L.counters + xcd, 1);
    }
    __syncthreads();
    // wave-uniform: every value derived from the tile index stays scalar
    i = __builtin_amdgcn_readfirstlane(next_tile[0]);
  } else {
    i = (int)(blockIdx.x / N_XCD);
  }

  auto make_ctx = [&](int it, TileCtx& c) {
    int pos = 0, first = 0;
#pragma unroll
    for (int r = 1; r < kMaxSets; ++r)
      if (it >= pre[r]) {
        pos = r;
        first = pre[r];
      }
    int q = 0, t = 0, m_t = 0, n_t = 0, p_t = 1;
#pragma unroll
    for (int x = 0; x < kMaxSets; ++x)
      if (rank[x] == pos) {
        q = x;
        t = lo[x] + (it - first);
        m_t = mt[x];
        n_t = ntl[x];
        p_t = prt[x];
      }
    c.set = q;
    c.kb = L.kind_b[q] != 0;
    for_kind(c.kb, [&](auto kc) {
      constexpr int KIND = decltype(kc)::value;
      using K_ = Kind<KIND>;
      constexpr int GK = Cfg<KIND>::GK;
      const GemmArgs& a = L.s[q];
      tile_decode<KIND>(a, gtab[q], t, m_t * p_t, n_t, p_t, c.tl, c.tile_n);
      c.parts = p_t;
      const Tile tl = c.tl;
      const int tile_n = c.tile_n;
      const bf16_t* A = static_cast<const bf16_t*>(a.A);
      const bf16_t* B = static_cast<const bf16_t*>(a.B) + (K_::MRAG ? (size_t)tl.g * a.b_gs : 0);
      const int Kd = K_::MRAG ? a.K : tl.rows;
      c.nk = (Kd + GK - 1) / GK;
      c.n_full = Kd / GK;  // k-steps without a ragged tail
      // K part tl.split of p_t: k-steps [ks0, ks1) (M-ragged kinds only)
      const int ks0 = c.nk * tl.split / p_t;
      if constexpr (K_::MRAG) c.nk = c.nk * (tl.split + 1) / p_t - ks0;
      const int last_row = tl.row0 + (tl.rows > 0 ? tl.rows - 1 : 0);
      // operand pointers; out-of-range M/N indices are clamped to valid
      // memory (outputs not stored), out-of-range k-rows read zeros
      auto a_row = [&](int r) -> const bf16_t* {  // M-ragged A, k-contiguous
        return A + (size_t)min(tl.row0 + r, last_row) * a.lda;
      };
      auto a_elem = [&](int k, int col) -> const bf16_t* {  // TN A(i = m0 + col, k)
        if (k >= Kd) return zero16;
        const int m = (tl.m0 + col + 8 <= a.M) ? tl.m0 + col : 0;
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
      auto b_elem = [&](int k, int col) -> const bf16_t* {  // NN / TN B(k, n = n0 + col)
        const int n = (tl.n0 + col + 8 <= a.N) ? tl.n0 + col : 0;
        if constexpr (K_::MRAG) {
          return B + (size_t)k * a.ldb + n;
        } else {
          if (k >= Kd) return zero16;
          return B + (size_t)(tl.row0 + k) * a.ldb + n;
        }
      };
      // DMA addresses at k-step 0 (k-contiguous operands advance by GK
      // elements, m/n-contiguous ones by GK rows per k-step) and of the
      // ragged tail k-step
      constexpr int DA = Cfg<KIND>::DMA_A, DB = Cfg<KIND>::DMA_B;
      static_assert(DA <= 4 && DB <= 4 && (K_::MRAG || (DA <= 2 && DB <= 2)), "DMA slots");
      DmaPtrs<DA> da, db;
      if constexpr (K_::A_KC) dma_kc_init<GK, NW>(da, a_row, wave, A); else dma_mn_init<NW>(da, a_elem, wave, 0, A);
      if constexpr (K_::B_KC) dma_kc_init<GK, NW>(db, b_row, wave, B); else dma_mn_init<NW>(db, b_elem, wave, 0, B);
#pragma unroll
      for (int x = 0; x < DA; ++x) c.da.p[x] = da.p[x];
#pragma unroll
      for (int x = 0; x < DB; ++x) c.db.p[x] = db.p[x];
      if constexpr (!K_::MRAG) {
        DmaPtrs<DA> ta;
        DmaPtrs<DB> tb;
        dma_mn_init<NW>(ta, a_elem, wave, c.n_full * GK, A);
        dma_mn_init<NW>(tb, b_elem, wave, c.n_full * GK, B);
#pragma unroll
        for (int x = 0; x < DA; ++x) c.ta.p[x] = ta.p[x];
#pragma unroll
        for (int x = 0; x < DB; ++x) c.tb.p[x] = tb.p[x];
      }
      c.rs_a = make_rsrc(A);
      c.rs_b = make_rsrc(B);
      c.a_step = 2u * (K_::A_KC ? GK : (unsigned)GK * a.lda);
      c.b_step = 2u * (K_::B_KC ? GK : (unsigned)GK * a.ldb);
      if constexpr (K_::MRAG) {
        if (ks0 > 0) {
#pragma unroll
          for (int x = 0; x < DA; ++x) c.da.p[x] += (unsigned)ks0 * c.a_step;
#pragma unroll
          for (int x = 0; x < DB; ++x) c.db.p[x] += (unsigned)ks0 * c.b_step;
        }
      }
    });
  };

  // DMA load i of each operand (A: i < DMA_A, B: i < DMA_B) of tile c for
  // k-step ks into stage st
  auto dma = [&](auto kc, const TileCtx& c, int ks, int st, int i) {
    constexpr int KIND = decltype(kc)::value;
    using C_ = Cfg<KIND>;
    constexpr bool MRAG = Kind<KIND>::MRAG;
    char* la = lds + st * C_::STAGE;
    const bool tail = !MRAG && ks >= c.n_full;
    if (i < C_::DMA_A) {
      unsigned pa = c.da.p[i] + ks * c.a_step;
      if constexpr (!MRAG) pa = tail ? c.ta.p[i < 2 ? i : 0] : pa;
      load_to_lds(c.rs_a, pa, la + (i * NW + wave) * 1024);
    }
    if (i < C_::DMA_B) {
      unsigned pb = c.db.p[i] + ks * c.b_step;
      if constexpr (!MRAG) pb = tail ? c.tb.p[i < 2 ? i : 0] : pb;
      load_to_lds(c.rs_b, pb, la + C_::A_BYTES + (i * NW + wave) * 1024);
    }
  };
  // the first NS k-steps of tile c into the ring (only k-steps below nk)
  auto prologue = [&](const TileCtx& c) {
    for_kind(c.kb, [&](auto kc) {
      constexpr int KIND = decltype(kc)::value;
      using C_ = Cfg<KIND>;
#pragma unroll
      for (int p = 0; p < C_::NS; ++p)
        if (p < c.nk) {
#pragma unroll
          for (int q = 0; q < C_::DMA_MAX; ++q) dma(kc, c, p, p, q);
        }
    });
  };

  TileCtx cur;
  if (i < total) {
    make_ctx(i, cur);
    prologue(cur);
  }
  while (i < total) {
    // ---- main loop and epilogue of the current tile
    for_kind(cur.kb, [&](auto kc) {
      constexpr int KIND = decltype(kc)::value;
      using K_ = Kind<KIND>;
      using C_ = Cfg<KIND>;
      constexpr int NS = C_::NS, GK = C_::GK, K32 = C_::K32;
      const int nk = cur.nk;
      f32x4_t acc[MI][NJ];
      bf16x8_t out[16];   // staged bf16 results (epilogue part 1)
      bool late = false;  // results left for part 2's stores
#pragma unroll
      for (int a_ = 0; a_ < MI; ++a_)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[a_][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

      // fragment f of the wave's A rows (wm WM + 16 f ..) or B columns
      // (wn 128 + 16 f ..) at k32-step s of a stage
      auto frag_a = [&](const char* stage, int s, int f) -> bf16x8_t {
        return K_::A_KC ? frag_kc<GK>(stage, wm * WM + f * 16, s)
                        : frag_mn(stage, wm * WM + f * 16, s);
      };
      auto frag_b = [&](const char* stage, int s, int f) -> bf16x8_t {
        const char* lb = stage + C_::A_BYTES;
        return K_::B_KC ? frag_kc<GK>(lb, wn * 128 + f * 16, s)
                        : frag_mn(lb, wn * 128 + f * 16, s);
      };

      // One k32-step s of `stage`: NJ chunks, chunk j issuing the MI MFMAs of
      // B fragment j (acc[i][j] += A_i B_j).  B fragments pass through a ring
      // of four register sets Bq, each read three chunks before its use
      // (chunk j reads fragment j + 3, from the next k32-step - at s_n of
      // stage_n - for j >= NJ - 3); the next k32-step's A fragments are read
      // in chunks 4..7 into A_n.  On a k-step's last k32-step (`last`), chunk
      // 4 first reads the stage's final fragment, then waits for the wave's
      // LDS reads and for its DMA of k-step kt + 1, and takes the barrier
      // after which every wave is done with this stage: the fragments of the
      // next k32-step come from stage_n (k-step kt + 1), and the DMA loads of
      // k-step dma_ks (if >= 0) refill this stage (dma_st) in chunks
      // 4 .. 4 + DMA_MAX - 1.  sched_barrier(0) fences keep this order, so the
      // compiler's LDS waits fall at each fragment's first use.
      static_assert(C_::DMA_MAX <= NJ - 4, "DMA loads per k-step exceed the chunks");
      static_assert(MI == 4, "A fragments are read in chunks 4..7");
      auto k32step = [&](const char* stage, int s, const bf16x8_t* A_c, bf16x8_t* A_n,
                         bf16x8_t* Bq, const char* stage_n, int s_n, bool last, int kt,
                         int dma_ks, int dma_st) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          if (j + 3 < NJ) Bq[(j + 3) % 4] = frag_b(stage, s, j + 3);
          if (last && j == 4) {
            WAIT_LGKMCNT(0);
            // k-step kt + 1 landed (kt + 2 .. min(kt + NS, nk) - 1 may stay in flight)
            wait_vm_groups<C_::DMA_N, NS - 2>(nk - 2 - kt);
            __syncthreads();
          }
          if (j + 3 >= NJ) Bq[(j + 3) % 4] = frag_b(stage_n, s_n, j + 3 - NJ);
          if (j >= 4) A_n[j - 4] = frag_a(stage_n, s_n, j - 4);
          if (last && dma_ks >= 0 && j >= 4 && j - 4 < C_::DMA_MAX) dma(kc, cur, dma_ks, dma_st, j - 4);
#pragma unroll
          for (int ii = 0; ii < MI; ++ii)
            acc[ii][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Bq[j % 4], A_c[ii], acc[ii][j], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      };

      bf16x8_t af0[MI], af1[MI], bq[4];
      if (nk > 0) {
        // own DMA of k-step 0 done (k-steps 1 .. min(NS, nk) - 1 may stay in flight)
        wait_vm_groups<C_::DMA_N, NS - 1>(nk - 1);
        __syncthreads();
#pragma unroll
        for (int f = 0; f < MI; ++f) af0[f] = frag_a(lds, 0, f);
#pragma unroll
        for (int f = 0; f < 3; ++f) bq[f] = frag_b(lds, 0, f);
      }
      // k-step kt: K32 k32-steps, the last of which reads the next stage and
      // refills this one (with k-step kt + NS if there is one).  A fragments
      // alternate between af0 and af1 every k32-step.
      auto kstep = [&](int kt, bf16x8_t* A_even, bf16x8_t* A_odd) {
        const int st = kt % NS;
        const char* stage = lds + st * C_::STAGE;
        const char* stage_next = lds + ((kt + 1) % NS) * C_::STAGE;
        const int refill = kt + NS < nk ? kt + NS : -1;
#pragma unroll
        for (int s = 0; s < K32; ++s) {
          const bool last = s == K32 - 1;
          bf16x8_t* A_c = s % 2 == 0 ? A_even : A_odd;
          bf16x8_t* A_n = s % 2 == 0 ? A_odd : A_even;
          k32step(stage, s, A_c, A_n, bq, last ? stage_next : stage, last ? 0 : s + 1, last, kt,
                  last ? refill : -1, st);
        }
      };
      if constexpr (K32 % 2 == 0) {
        for (int kt = 0; kt < nk; ++kt) kstep(kt, af0, af1);
      } else {
        for (int kt = 0; kt < nk; kt += 2) {
          kstep(kt, af0, af1);
          if (kt + 1 < nk) kstep(kt + 1, af1, af0);
        }
      }
      // (the last k-step's wait took every DMA load of this tile)

      // With dynamic dealing the block takes its next tile now, when this
      // one's main loop is done: the counter's latency passes during the
      // epilogue, and no block holds a tile it has not started while others
      // run out of work.  (Taking it a whole tile ahead let one block hold two
      // of a launch's few long tiles: the mid-size dX + dW_gu launch then ran
      // in 200 instead of 148 us in about half of the calls.)
      if (dyn && threadIdx.x == 0) nxt = atomicAdd(L.counters + xcd, 1);

      // ---- epilogue, part 1: results into registers (or, for the kinds
      // that read memory and the accumulating weight gradients, the whole
      // epilogue).  Accumulator (i, j) register t
      // holds C[wm*WM + 16i + lane%16][wn*128 + 16j + 4(lane/16) + t]
      const GemmArgs& a = L.s[cur.set];
      const Tile tl = cur.tl;
      const int row_lim = tl.rows - wm * WM;  // rows of this wave's sub-tile to store
      char* reg = lds + wave * C_::EPI_WAVE;
      // the lane index, opaque to the compiler from here on: the epilogue's
      // lane-dependent addresses are then computed per tile rather than
      // hoisted out of the tile loop, where they would hold registers across
      // the main loop (or spill)
      int ln = lane;
      asm volatile("" : "+v"(ln));
      if constexpr (KIND == DWD || KIND == DWGU) {
        late = !a.accumulate;
        if (a.accumulate) {
          // fp32 weight gradient added to the caller's values, 16 bytes per
          // lane straight from the accumulators, before the next tile's loads
          const int r_in = ln & 15;
          const int c_in = 4 * (ln >> 4);
#pragma unroll
          for (int ii = 0; ii < MI; ++ii) {
            const int row = wm * WM + ii * 16 + r_in;
            if (tl.m0 + row >= a.M) continue;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
              const int col = tl.n0 + wn * 128 + j * 16 + c_in;
              if (col >= a.N) continue;
              float* c = static_cast<float*>(a.C) + (size_t)tl.g * a.c_gs +
                         (size_t)tl.split * a.c_split + (size_t)(tl.m0 + row) * a.ldc + col;
              *reinterpret_cast<f32x4_t*>(c) = acc[ii][j] + *reinterpret_cast<const f32x4_t*>(c);
            }
          }
        }
      } else if ((KIND == DOWN_FWD || KIND == DX_BWD) && cur.parts > 1) {
        // a K part: its fp32 partial ([cap, N], rows as the output's),
        // straight from the accumulators (here, so that the accumulators
        // and the staged bf16 results of part 2 are never live together)
        const __amdgpu_buffer_rsrc_t rc = store_rsrc(a.part + (size_t)tl.split * a.c_split);
        const int r_in = ln & 15;
        const int c_in = 4 * (ln >> 4);
#pragma unroll
        for (int ii = 0; ii < MI; ++ii) {
          const int row = wm * WM + ii * 16 + r_in;
          const bool rok = row < tl.rows;
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int col = tl.n0 + wn * 128 + j * 16 + c_in;
            const unsigned off = rok && col < a.N
                                     ? 4u * ((unsigned)(tl.row0 + row) * (unsigned)a.N + (unsigned)col)
                                     : kOOB;
            store16<false>(rc, off, __builtin_bit_cast(u32x4_t, acc[ii][j]));
          }
        }
      } else {
        // bf16 outputs go through LDS so that every global access is a whole
        // 16-byte chunk and a wave instruction covers 256 contiguous bytes of
        // a row (4 rows) instead of 32 bytes of 16 rows.  Each wave transposes
        // its 64 x 128 sub-tile in a private 16 KB region of the ring (every
        // wave passed the last k-step's barrier, after which no wave reads the
        // ring's data).  The outputs (and the G/U that the dSwiGLU epilogue
        // reads) are touched once here, so they go past the caches
        // (nontemporal: measured 2-4 % faster for DHH_BWD, DX_BWD and
        // DOWN_FWD; the fp32 weight gradients are not, they were 1.4-1.7x
        // slower that way).
#pragma unroll
        for (int ii = 0; ii < MI; ++ii)
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int row = ii * 16 + (ln & 15);
            const int u = 4 * j + (ln >> 4);
            epi_put(reg, row, u, acc[ii][j][0], acc[ii][j][1], acc[ii][j][2], acc[ii][j][3]);
          }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // region is wave-private
        if constexpr (KIND == GU_FWD) {
          // region row: [G h0..31 | U h0..31 | G h32..63 | U h32..63] of the
          // wave's 64 hidden units; lane -> (row, 8 hidden units)
          const int cg = 8 * ((ln & 7) >> 2) + (ln & 3);
#pragma unroll
          for (int it = 0; it < WM / 8; ++it) {
            const int row = it * 8 + (ln >> 3);
            out[it] = epi_get(reg, row, cg);
            out[8 + it] = epi_get(reg, row, cg + 4);
          }
          late = true;
        } else if constexpr (KIND == DOWN_FWD || KIND == DX_BWD || KIND == UP_FWD) {
          const int c = ln & 15;
#pragma unroll
          for (int it = 0; it < WM / 4; ++it) out[it] = epi_get(reg, it * 4 + (ln >> 4), c);
          late = true;
        } else {
          const int c = ln & 15;
          const int col = tl.n0 + wn * 128 + 8 * c;
          if (col < a.N) {
            if constexpr (KIND == DHH_BWD) {
              // dG = dHh * U * silu'(G), dU = dHh * silu(G); G and U of a batch
              // of rows are loaded before any store of it (all rows at once
              // measured slower: the 128 registers of G and U spill)
              const bf16_t* gu = static_cast<const bf16_t*>(a.aux);
              bf16_t* dgu = static_cast<bf16_t*>(a.C);
              for (int it0 = 0; it0 < WM / 4; it0 += 8) {
                if (it0 * 4 >= row_lim) break;
                bf16x8_t G[8], U[8];
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                  const int row = min((it0 + b) * 4 + (ln >> 4), row_lim - 1);
                  const size_t m = (size_t)(tl.row0 + wm * WM + row);
                  G[b] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(gu + m * 2 * a.H + col));
                  U[b] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(gu + m * 2 * a.H + a.H + col));
                }
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                  const int row = (it0 + b) * 4 + (ln >> 4);
                  const bf16x8_t v = epi_get(reg, row, c);
                  bf16x8_t dG, dU;
#pragma unroll
                  for (int e = 0; e < 8; ++e) {
                    const float g = (float)G[b][e], dh = (float)v[e];
                    const float sg = sigmoid_fast(g);
                    dG[e] = (bf16_t)(dh * (float)U[b][e] * (sg * (1.0f + g * (1.0f - sg))));
                    dU[e] = (bf16_t)(dh * g * sg);
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
                  const int row = min((it0 + b) * 4 + (ln >> 4), row_lim - 1);
                  Av[b] = *reinterpret_cast<const bf16x8_t*>(
                      Ab + (size_t)(tl.row0 + wm * WM + row) * a.H + col);
                }
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                  const int row = (it0 + b) * 4 + (ln >> 4);
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
            }
          }
        }
      }

      // ---- epilogue, part 2: the stores
      if (late) {
      if constexpr (KIND == DWD || KIND == DWGU) {
        // fp32 weight gradient of group g, 16 bytes per lane straight from
        // the accumulators (64 contiguous bytes of 16 rows per instruction)
        const __amdgpu_buffer_rsrc_t rc = store_rsrc(
            static_cast<float*>(a.C) + (size_t)tl.g * a.c_gs + (size_t)tl.split * a.c_split);
        const int r_in = ln & 15;
        const int c_in = 4 * (ln >> 4);
#pragma unroll
        for (int ii = 0; ii < MI; ++ii) {
          const int row = wm * WM + ii * 16 + r_in;
          const bool rok = tl.m0 + row < a.M;
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            const int col = tl.n0 + wn * 128 + j * 16 + c_in;
            const unsigned off = rok && col < a.N
                                     ? 4u * ((unsigned)(tl.m0 + row) * (unsigned)a.ldc + (unsigned)col)
                                     : kOOB;
            store16<false>(rc, off, __builtin_bit_cast(u32x4_t, acc[ii][j]));
          }
        }
      } else if constexpr (KIND == GU_FWD) {
        const int h = cur.tile_n * (GT / 2) + wn * 64 + 32 * ((ln & 7) >> 2) + 8 * (ln & 3);
        const __amdgpu_buffer_rsrc_t rg = store_rsrc(a.C), rh = store_rsrc(a.out2);
        const unsigned H = (unsigned)a.H;
#pragma unroll
        for (int it = 0; it < WM / 8; ++it) {
          const int row = it * 8 + (ln >> 3);
          const bool ok = row < row_lim && h < a.H;
          const unsigned m = (unsigned)(tl.row0 + wm * WM + row);
          const bf16x8_t G = out[it], U = out[8 + it];
          bf16x8_t Hv;
#pragma unroll
          for (int e = 0; e < 8; ++e) Hv[e] = (bf16_t)(silu_fast((float)G[e]) * (float)U[e]);
          store16<true>(rg, ok ? 2u * (m * 2u * H + h) : kOOB, __builtin_bit_cast(u32x4_t, G));
          store16<true>(rg, ok ? 2u * (m * 2u * H + H + h) : kOOB, __builtin_bit_cast(u32x4_t, U));
          store16<true>(rh, ok ? 2u * (m * H + h) : kOOB, __builtin_bit_cast(u32x4_t, Hv));
        }
      } else if constexpr (KIND == DOWN_FWD || KIND == DX_BWD || KIND == UP_FWD) {
        const int c = ln & 15;
        const int col = tl.n0 + wn * 128 + 8 * c;
        const __amdgpu_buffer_rsrc_t rc = store_rsrc(a.C);
#pragma unroll
        for (int it = 0; it < WM / 4; ++it) {
          const int row = it * 4 + (ln >> 4);
          const bool ok = row < row_lim && col < a.N;
          const unsigned m = (unsigned)(tl.row0 + wm * WM + row);
          store16<true>(rc, ok ? 2u * (m * (unsigned)a.ldc + col) : kOOB,
                        __builtin_bit_cast(u32x4_t, out[it]));
          if constexpr (KIND == UP_FWD) {
            // h = silu(A) of the bf16-rounded A
            bf16x8_t Hv;
#pragma unroll
            for (int e = 0; e < 8; ++e) Hv[e] = (bf16_t)silu_fast((float)out[it][e]);
            store16<true>(store_rsrc(a.out2), ok ? 2u * (m * (unsigned)a.H + col) : kOOB,
                          __builtin_bit_cast(u32x4_t, Hv));
          }
        }
      }
      }
    });

    // ---- next tile: the dealt tile is broadcast through LDS; the barrier
    // also frees the ring (every wave has read back its staged results)
    if (dyn) {
      it_parity ^= 1;
      if (threadIdx.x == 0) {
        next_tile[it_parity] = nxt;
      }
    }
    __syncthreads();
    const int i_next = __builtin_amdgcn_readfirstlane(dyn ? next_tile[it_parity] : i + per_xcd);
    TileCtx nx;
    if (i_next < total) {
      make_ctx(i_next, nx);
      prologue(nx);
    }

    cur = nx;
    i = i_next;
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
  return Kind<KIND>::MRAG
             ? (ceil_div(a.cap, BM) + (long)a.n_groups) * n_tiles * std::max(1, a.ksplit_max)
             : (long)a.n_groups * std::max(1, a.ksplit) * ceil_div(a.M, BM) * n_tiles;
}

constexpr const char* kGemmNames[] = {"gemm_gu_fwd", "gemm_down_fwd", "gemm_dhh_bwd",
                                      "gemm_dx_bwd", "gemm_dwd", "gemm_dwgu",
                                      "gemm_up_fwd", "gemm_dh_bwd"};

template <int KA, int KB>
const char* gemm_name() {
  if constexpr (KA == KB) return kGemmNames[KA];
  else if constexpr (KA == DHH_BWD && KB == DWD) return "gemm_dhh_dwd";
  else if constexpr (KA == DH_BWD && KB == DWD) return "gemm_dh_dwd";
  else if constexpr (KA == DX_BWD && KB == DWGU) return "gemm_dx_dwgu";
  else return "gemm_merged";
}

// One bf16 launch over up to kMaxSets sets: sets_a[0..na) of kind KA and
// sets_b[0..nb) of kind KB.  counters: zeroed per-XCD tile counters for
// dynamic dealing (the kernel then deals the sets longest reduction per tile
// first, measured from the device-side group offsets), or NULL for
// round-robin dealing in the given set order.
template <int KA, int KB>
hipError_t run_gemm_bf16(const GemmArgs* sets_a, int na, const GemmArgs* sets_b, int nb,
                         hipStream_t s, int* counters) {
  GemmLaunch L{};
  struct Entry { GemmArgs a; int kb; long tiles; };
  Entry e[kMaxSets];
  int n = 0;
  for (int q = 0; q < na; ++q) e[n++] = Entry{sets_a[q], 0, max_tiles<KA>(sets_a[q])};
  for (int q = 0; q < nb; ++q) e[n++] = Entry{sets_b[q], 1, max_tiles<KB>(sets_b[q])};
  long tiles = 0;
  for (int q = 0; q < n; ++q) {
    L.s[q] = e[q].a;
    L.kind_b[q] = e[q].kb;
    tiles += e[q].tiles;
  }
  L.n_sets = n;
  L.counters = counters;
  if (tiles == 0) return hipSuccess;
  // persistent: at most one block per CU, a multiple of N_XCD blocks
  long blocks = std::min<long>((long)num_cus(), tiles);
  blocks = std::max<long>(N_XCD, (blocks + N_XCD - 1) / N_XCD * N_XCD);
  MOE_TIMED((gemm_name<KA, KB>()), s, gemm_bf16_kernel<KA, KB><<<(int)blocks, 512, 0, s>>>(L));
  return hipGetLastError();
}

// One launch per set group of one GEMM kind (fp32: one SIMT launch per set).
template <int KIND>
hipError_t run_gemm(const GemmArgs* sets, int n_sets, int bf16, hipStream_t s,
                    int* counters = nullptr) {
  if (bf16) return run_gemm_bf16<KIND, KIND>(sets, n_sets, nullptr, 0, s, counters);
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

// counters[0..n) = 0 (the per-XCD tile counters of the next launches)
__global__ __launch_bounds__(64) void zero_counters_kernel(int* counters, int n) {
  if ((int)threadIdx.x < n) counters[threadIdx.x] = 0;
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

// Rows of the set's groups (clamped to [0, cap] as the GEMM's group table
// does) of the bf16 output: out[r, :] = bf16(part_0[r, :] + ... +
// part_{S-1}[r, :]) in that order, S = *parts_used (the K parts the GEMM
// chose; nothing to do when it chose 1).  N % 8 == 0.
__global__ __launch_bounds__(256) void splitk_rows_reduce_kernel(
    bf16_t* out, long ldo, const float* part, long stride, const int* parts_used,
    const int32_t* offsets, int n_groups, int cap, int N) {
  const int S = *parts_used;
  if (S <= 1) return;
  __shared__ int s_hi;
  if (threadIdx.x == 0) s_hi = 0;
  __syncthreads();
  const int lo = clamp_row(offsets[0], cap);
  for (int g = threadIdx.x; g <= n_groups; g += 256) atomicMax(&s_hi, clamp_row(offsets[g], cap));
  __syncthreads();
  const int hi = max(lo, s_hi);
  const int c8 = N / 8;
  const long n = (long)(hi - lo) * c8;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
    const long r = lo + i / c8;
    const int c = (int)(i % c8) * 8;
    f32x4_t q[8][2];  // every part's loads first (S <= 8)
#pragma unroll
    for (int p = 0; p < 8; ++p)
      if (p < S) {
        const f32x4_t* src = reinterpret_cast<const f32x4_t*>(part + p * stride + r * N + c);
        q[p][0] = __builtin_nontemporal_load(src);
        q[p][1] = __builtin_nontemporal_load(src + 1);
      }
    f32x4_t v0 = q[0][0], v1 = q[0][1];
#pragma unroll
    for (int p = 1; p < 8; ++p)
      if (p < S) {
        v0 += q[p][0];
        v1 += q[p][1];
      }
    bf16x8_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = (bf16_t)v0[e];
      o[4 + e] = (bf16_t)v1[e];
    }
    *reinterpret_cast<bf16x8_t*>(out + r * ldo + c) = o;
  }
}

// Largest K split of a DOWN_FWD / DX_BWD set whose fp32 partials ([cap, N]
// each) fit kPartBudget bytes; 1 (no split) when two do not.
constexpr size_t kPartBudget = (size_t)256 << 20;
constexpr int kMaxRowParts = 8;
int row_parts_max(int bf16, long cap, long N) {
  if (!bf16 || cap <= 0) return 1;
  const size_t per = (size_t)cap * N * sizeof(float);
  return (int)std::min<size_t>(kMaxRowParts, kPartBudget / per);
}

// Split-K factor of the weight-gradient GEMM of one set.  A single large
// group (the merged shared experts: one group over all T tokens) is cut into
// parts of its rows, each part writing its own fp32 partial, summed
// afterwards in a fixed order - but only when the whole backward launch that
// holds it (dHh with dW_d, or dX with dW_gu, over every set) has fewer tiles
// than the GPU has CUs; otherwise the other kind's tiles fill the CUs and the
// long tiles simply start first.
long bwd_launch_tiles(const moe_ffn_set* sets, int n_sets, int d, bool second) {
  long t = 0;
  for (int i = 0; i < n_sets; ++i) {
    const moe_ffn_set& f = sets[i];
    const long R1 = f.activation == MOE_ACT_SILU ? 1 : 2;
    const long m_tiles = ceil_div(f.cap, GT) + (long)f.n_groups;  // M-ragged bound
    if (!second)  // dHh (N = H) and dW_d (d x H per group)
      t += m_tiles * ceil_div(f.H, GT) + (long)f.n_groups * ceil_div(d, GT) * ceil_div(f.H, GT);
    else          // dX (N = d) and dW_gu (R1 H x d per group)
      t += m_tiles * ceil_div(d, GT) + (long)f.n_groups * ceil_div((int)(R1 * f.H), GT) * ceil_div(d, GT);
  }
  return t;
}

int ksplit_factor(int bf16, long M, long N, const moe_ffn_set& f, long launch_tiles) {
  if (!bf16 || f.n_groups != 1 || f.cap < 4096 || launch_tiles >= num_cus()) return 1;
  const long tiles = ceil_div((int)M, GT) * (long)ceil_div((int)N, GT);
  const long sp = num_cus() / std::max<long>(tiles, 1);
  return (int)std::max<long>(1, std::min<long>(4, sp));
}

constexpr size_t kWsAlign = 256;
constexpr int kCounterWords = 2 * N_XCD;  // per-XCD counters of the two backward launches
size_t align_up(size_t v) { return (v + kWsAlign - 1) / kWsAlign * kWsAlign; }

// Workspace of the K-part partials of one launch's DOWN_FWD or DX_BWD sets
// (N = d): one int per set (the parts the GEMM chose), then per set that may
// split its row_parts_max [cap, d] fp32 partials.
size_t row_parts_bytes(const moe_ffn_set* sets, int n_sets, int bf16, int d) {
  size_t b = 0;
  for (int i = 0; i < n_sets; ++i) {
    const int S = row_parts_max(bf16, sets[i].cap, d);
    if (S > 1) b += align_up((size_t)S * sets[i].cap * d * sizeof(float));
  }
  return b ? align_up(kMaxSets * sizeof(int)) + b : 0;
}

// Point the DOWN_FWD / DX_BWD arguments of the sets at their partials in the
// workspace region at `p` (row_parts_bytes of it).
void assign_row_parts(GemmArgs* args, const moe_ffn_set* sets, int n_sets, int bf16, int d,
                      char* p) {
  if (!p || row_parts_bytes(sets, n_sets, bf16, d) == 0) return;
  int* used = reinterpret_cast<int*>(p);
  p += align_up(kMaxSets * sizeof(int));
  for (int i = 0; i < n_sets; ++i) {
    const int S = row_parts_max(bf16, sets[i].cap, d);
    if (S <= 1) continue;
    args[i].ksplit_max = S;
    args[i].part = reinterpret_cast<float*>(p);
    args[i].c_split = (long)sets[i].cap * d;
    args[i].ksplit_used = used + i;
    p += align_up((size_t)S * sets[i].cap * d * sizeof(float));
  }
}

// Sum the K parts of the sets that may have split (after their GEMM launch).
hipError_t reduce_row_parts(const GemmArgs* args, int n_sets, hipStream_t s) {
  for (int i = 0; i < n_sets; ++i) {
    const GemmArgs& a = args[i];
    if (a.ksplit_max <= 1) continue;
    const long n8 = (long)a.cap * a.N / 8;
    // grid-stride: 4 blocks per CU stream the partials at full rate, and a call
    // that chose one part (every block returns at once) stays short
    const int blocks = (int)std::max<long>(1, std::min<long>(4L * num_cus(), (n8 + 255) / 256));
    MOE_TIMED("splitk_rows_reduce", s,
              splitk_rows_reduce_kernel<<<blocks, 256, 0, s>>>(
                  static_cast<bf16_t*>(a.C), a.ldc, a.part, a.c_split, a.ksplit_used, a.offsets,
                  a.n_groups, a.cap, a.N));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

// Rows of an expert's first weight per hidden unit: 2 (gate and up) for
// SwiGLU, 1 for the SiLU expert.
long first_rows(const moe_ffn_set& f) { return f.activation == MOE_ACT_SILU ? 1 : 2; }

size_t ffn_fwd_ws_bytes(const moe_ffn_set* sets, int n_sets, int bf16, int d) {
  return row_parts_bytes(sets, n_sets, bf16, d);
}

size_t ffn_bwd_ws_bytes(const moe_ffn_set* sets, int n_sets, int bf16, int d) {
  size_t bytes = align_up(kCounterWords * sizeof(int)) + row_parts_bytes(sets, n_sets, bf16, d);
  for (int i = 0; i < n_sets; ++i) {
    const moe_ffn_set& f = sets[i];
    const long H = f.H, R1 = first_rows(f);
    const int s_wd = ksplit_factor(bf16, d, H, f, bwd_launch_tiles(sets, n_sets, d, false));
    const int s_wgu = ksplit_factor(bf16, R1 * H, d, f, bwd_launch_tiles(sets, n_sets, d, true));
    if (s_wd > 1) bytes += align_up((size_t)s_wd * d * H * sizeof(float));
    if (s_wgu > 1) bytes += align_up((size_t)s_wgu * R1 * H * d * sizeof(float));
  }
  return bytes;
}

hipError_t launch_ffn_fwd_sets(const moe_ffn_set* sets, int n_sets, int bf16, int d, void* ws,
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
  if (bf16) assign_row_parts(o, sets, n_sets, bf16, d, static_cast<char*>(ws));
  hipError_t e = silu ? run_gemm<UP_FWD>(g, n_sets, bf16, s) : run_gemm<GU_FWD>(g, n_sets, bf16, s);
  if (e != hipSuccess) return e;
  if ((e = run_gemm<DOWN_FWD>(o, n_sets, bf16, s)) != hipSuccess) return e;
  return reduce_row_parts(o, n_sets, s);
}

hipError_t launch_ffn_bwd_sets(const moe_ffn_set* sets, int n_sets, int bf16, int d,
                               int accumulate_dw, void* ws, hipStream_t s) {
  GemmArgs hh[2]{}, dx[2]{}, wd[2]{}, wgu[2]{};
  // workspace: per-XCD counters, then the split-K partials
  int* counters = static_cast<int*>(ws);
  char* rows_ws = static_cast<char*>(ws) + (ws ? align_up(kCounterWords * sizeof(int)) : 0);
  char* part = rows_ws + (ws ? row_parts_bytes(sets, n_sets, bf16, d) : 0);
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
        const int S = ksplit_factor(bf16, g->M, g->N, f,
                                    bwd_launch_tiles(sets, n_sets, d, g == &w));
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
  if (bf16 && ws) assign_row_parts(dx, sets, n_sets, bf16, d, rows_ws);
  hipError_t e;
  if (!bf16) {
    e = silu ? run_gemm<DH_BWD>(hh, n_sets, bf16, s) : run_gemm<DHH_BWD>(hh, n_sets, bf16, s);
    if (e != hipSuccess) return e;
    if ((e = run_gemm<DX_BWD>(dx, n_sets, bf16, s)) != hipSuccess) return e;
    if ((e = run_gemm<DWD>(wd, n_sets, bf16, s)) != hipSuccess) return e;
    if ((e = run_gemm<DWGU>(wgu, n_sets, bf16, s)) != hipSuccess) return e;
  } else {
    // two launches of two independent kinds each: dHh with dW_d (both read
    // dY), then dX with dW_gu (both read dG/dU); with a workspace their tiles
    // are dealt dynamically from per-XCD counters, cleared here first
    if (ws) {
      MOE_TIMED("zero_counters", s, zero_counters_kernel<<<1, 64, 0, s>>>(counters, kCounterWords));
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    e = silu ? run_gemm_bf16<DH_BWD, DWD>(hh, n_sets, wd, n_sets, s, ws ? counters : nullptr)
             : run_gemm_bf16<DHH_BWD, DWD>(hh, n_sets, wd, n_sets, s, ws ? counters : nullptr);
    if (e != hipSuccess) return e;
    e = run_gemm_bf16<DX_BWD, DWGU>(dx, n_sets, wgu, n_sets, s, ws ? counters + N_XCD : nullptr);
    if (e != hipSuccess) return e;
    if ((e = reduce_row_parts(dx, n_sets, s)) != hipSuccess) return e;
  }
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
