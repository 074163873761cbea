// Expert placement and migration of a worker's resident experts (Alg. 1).
//
// Sec. 3.3 ("Expert placement modes"): every expert of a layer lives on
// exactly O_e of the M workers and every worker holds N_le = O_e N_e / M
// distinct experts; fixed placement keeps one map, random placement redraws it
// every T rounds.  After a redraw a worker fetches the experts new to it
// (Delta_in), keeps the optimiser state of those it already held and restarts
// the state of the new ones, with a learning-rate warm-up applied only to them
// (Sec. 3.4, "Outer optimization").
//
// Host side: the placement map and the migration map.  Device side: copies of
// expert-sized fp32 rows by index (weights from and to the global store,
// optimiser state from the previous local layout, zeros for restarted state)
// and AdamW over a worker's experts with a step count and learning rate per
// expert.
#include <vector>

#include "common.h"
#include "kernels.h"
#include "timing.h"

namespace moe {

// Placement: the N_e O_e (expert, replica) slots in expert order are dealt to
// the workers in turn, so expert e sits on workers (e O_e + j) mod M, j < O_e
// (distinct since O_e <= M); expert_perm / worker_perm relabel experts and
// workers (random placement).  sets[m * N_le ...] = worker m's sorted ids.
bool gen_placement(int N_e, int O_e, int M, const int32_t* expert_perm,
                   const int32_t* worker_perm, int32_t* sets) {
  if (N_e < 1 || O_e < 1 || M < 1 || O_e > M || ((long)N_e * O_e) % M != 0) return false;
  const int N_le = (int)((long)N_e * O_e / M);
  std::vector<std::vector<int32_t>> held(M);
  for (int e = 0; e < N_e; ++e)
    for (int j = 0; j < O_e; ++j) {
      const int w = (int)(((long)e * O_e + j) % M);
      held[worker_perm ? worker_perm[w] : w].push_back(expert_perm ? expert_perm[e] : e);
    }
  for (int m = 0; m < M; ++m) {
    std::sort(held[m].begin(), held[m].end());
    if ((int)held[m].size() != N_le) return false;
    std::copy(held[m].begin(), held[m].end(), sets + (size_t)m * N_le);
  }
  return true;
}

namespace {

constexpr int kMaxRows = 256;

struct CopyRowsArgs {
  const float* src;
  float* dst;
  bf16_t* dst_bf16;  // or NULL: bf16 copy of the written rows (dst's layout)
  size_t row_len;
  int src_row[kMaxRows];  // -1: zero row
  int dst_row[kMaxRows];
};

// dst[dst_row[r], :] = src[src_row[r], :] (or 0); one block column per row
__global__ __launch_bounds__(256) void copy_expert_rows_kernel(CopyRowsArgs a) {
  const int r = blockIdx.y;
  const int s = a.src_row[r];
  const size_t o = (size_t)a.dst_row[r] * a.row_len;
  float* d = a.dst + o;
  bf16_t* lp = a.dst_bf16 ? a.dst_bf16 + o : nullptr;
  const float* src = s >= 0 ? a.src + (size_t)s * a.row_len : nullptr;
  const size_t n4 = a.row_len / 4;
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    const f32x4_t v = src ? __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(src) + i)
                          : f32x4_t{0.f, 0.f, 0.f, 0.f};
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t*>(d) + i);
    if (lp) {
      const bf16x4_t b = {(bf16_t)v[0], (bf16_t)v[1], (bf16_t)v[2], (bf16_t)v[3]};
      reinterpret_cast<bf16x4_t*>(lp)[i] = b;
    }
  }
  for (size_t i = n4 * 4 + (size_t)blockIdx.x * 256 + threadIdx.x; i < a.row_len; i += stride) {
    const float v = src ? src[i] : 0.f;
    d[i] = v;
    if (lp) lp[i] = (bf16_t)v;
  }
}

}  // namespace

hipError_t launch_copy_expert_rows(const float* src, const int32_t* src_row, float* dst,
                                   const int32_t* dst_row, int n_rows, size_t row_len,
                                   void* dst_bf16, hipStream_t s) {
  if (n_rows == 0 || row_len == 0) return hipSuccess;
  CopyRowsArgs a{};
  a.src = src;
  a.dst = dst;
  a.dst_bf16 = static_cast<bf16_t*>(dst_bf16);
  a.row_len = row_len;
  for (int r = 0; r < n_rows; ++r) {
    a.src_row[r] = src_row[r];
    a.dst_row[r] = dst_row ? dst_row[r] : r;
  }
  const size_t want = (row_len / 4 + 255) / 256;
  dim3 grid((unsigned)std::max<size_t>(1, std::min<size_t>(want, 1024)), (unsigned)n_rows);
  MOE_TIMED("copy_expert_rows", s, copy_expert_rows_kernel<<<grid, 256, 0, s>>>(a));
  return hipGetLastError();
}

}  // namespace moe
