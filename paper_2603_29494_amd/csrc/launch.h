// Internal launch interface between the C ABI (vecattn_api.cpp) and the HIP
// kernels.  Arguments are already validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace vecattn {

struct Tensor4 {
  const void* ptr;
  int64_t B, H, N, D;
  int64_t sB, sH, sN;
};

hipError_t launch_pool(const Tensor4& q, int32_t block, void* qp, int64_t qp_sB, int64_t qp_sH,
                       int64_t qp_sN, hipStream_t stream);

struct SparseAttnArgs {
  Tensor4 q, k, v;
  void* o;
  int64_t o_sB, o_sH, o_sN;
  float* lse;
  const int32_t* idx;
  const int32_t* counts;
  int64_t cap;
  int32_t block;
  int32_t causal;
  float scale;
  const int32_t* order;  // [B, Hq, N_p] block order per (b, h), or NULL (ascending)
};

hipError_t launch_sparse_attn(const SparseAttnArgs& a, hipStream_t stream);

// Block order per (b, h) for the attention: blocks sorted by count (largest
// first), then by a sampled mean key, then by index, within consecutive
// segments of kOrderMaxBlocks blocks.  rows = B * Hq (fits the grid).
constexpr int32_t kOrderMaxBlocks = 16384;
hipError_t launch_attn_order(const int32_t* idx, int64_t cap, const int32_t* counts, int64_t rows,
                             int32_t Np, int64_t N, int32_t* order, hipStream_t stream);

struct SelectArgs {
  Tensor4 q, k;
  int32_t block;
  int32_t causal;
  int32_t keep_diag;  // every block also keeps the keys of its own rows
  int32_t unpadded;   // entries past a row's count are left unwritten
  int32_t mode;
  double param;
  const double* head_params;  // NULL, or one parameter per query head (host memory, Hq <= 128)
  int32_t tile;         // cross-tile minS: keys per tile (16 or 32)
  int32_t group_tiles;  // cross-tile minS: tiles per group (a power of two)
  int32_t* idx;
  int64_t cap;
  int32_t* counts;
  int32_t* n_clamped;
  void* workspace;
  size_t workspace_bytes;
};

// The library's own selection workspace (one copy per GPU, for callers that
// cannot allocate): its size, and this GPU's copy (the current device's).
constexpr size_t kStaticWorkspaceBytes = size_t(64) << 20;
hipError_t static_workspace(void** ptr);

size_t select_workspace_bytes(int64_t B, int64_t Hq, int64_t Hkv, int64_t N, int64_t D,
                              int32_t block, int32_t mode, int64_t cap);
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);

// Rows whose list breaks the attention's input contract, counted into *n_bad
// (cleared first).  rows <= 2^31 - 1 fits the grid.
hipError_t launch_check_lists(const int32_t* idx, const int32_t* counts, int64_t rows, int64_t cap,
                              int64_t n_keys, int32_t* n_bad, hipStream_t stream);

// Sparsity per query head from the counts of a selection (Eq. 5's sp_h):
// sparsity[h] = 1 - sum_{b,i} C[b,h,i] / (B * sum_i L_i), as fp64.
hipError_t launch_head_sparsity(const int32_t* counts, int64_t B, int64_t Hq, int64_t N,
                                int32_t block, int32_t causal, double* sparsity,
                                hipStream_t stream);

// Attention mass each query row's block list keeps (the recall of Sec. 2.2):
// kept[b,h,r] = sum over the listed visible keys of the row's softmax over
// all its visible keys.  N <= kRecallMaxN.
constexpr int64_t kRecallMaxN = int64_t(1) << 18;
struct RecallArgs {
  Tensor4 q, k;
  const int32_t* idx;
  const int32_t* counts;
  int64_t cap;
  int32_t block;
  int32_t causal;
  float scale;
  float* kept;
};
hipError_t launch_recall(const RecallArgs& a, hipStream_t stream);

// Host: per-head filter ratios by dynamic programming (Eq. 5).  Returns 0, or
// 1 when no choice reaches the target.
int plan_filter_ratios(int32_t H, int32_t C, const double* sp, const double* perf, double target,
                       int32_t grid, int32_t* choice, double* best);

}  // namespace vecattn
