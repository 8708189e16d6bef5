// C ABI of libvecattn: argument validation and dispatch to the HIP kernels.
// Every check happens on the host before any launch; see include/vecattn.h for
// the contract of each entry point.
#include "vecattn.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "launch.h"

namespace {

using vecattn::Tensor4;

constexpr int64_t kMaxN = int64_t(1) << 30;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Sizes positive, D contiguous, rows 16-byte aligned.
vecattn_status check_desc(const void* ptr, const vecattn_tdesc* d) {
  if (!ptr || !d) return VECATTN_ERR_INVALID_ARG;
  if (d->B < 1 || d->H < 1 || d->N < 1 || d->D < 1 || d->N > kMaxN) return VECATTN_ERR_INVALID_ARG;
  if (d->sB < 0 || d->sH < 0 || d->sN < d->D) return VECATTN_ERR_INVALID_ARG;
  if ((d->sB % 8) || (d->sH % 8) || (d->sN % 8) || !aligned16(ptr)) return VECATTN_ERR_INVALID_ARG;
  if (d->D != 64 && d->D != 128) return VECATTN_ERR_UNSUPPORTED;
  return VECATTN_OK;
}

Tensor4 to_tensor(const void* p, const vecattn_tdesc* d) {
  return Tensor4{p, d->B, d->H, d->N, d->D, d->sB, d->sH, d->sN};
}

int64_t num_blocks(int64_t N, int32_t P) { return (N + P - 1) / P; }

int64_t topk_count(double ratio, int64_t L) {
  int64_t k = static_cast<int64_t>(std::ceil(ratio * static_cast<double>(L) - 1e-9));
  if (k < 1) k = 1;
  if (k > L) k = L;
  return k;
}

bool mode_ok(int32_t mode) {
  return mode == VECATTN_SEL_TOPK || mode == VECATTN_SEL_TOPP || mode == VECATTN_SEL_MINS ||
         mode == VECATTN_SEL_MINS_TILED;
}

bool param_ok(int32_t mode, double param) {
  if (mode == VECATTN_SEL_TOPK || mode == VECATTN_SEL_TOPP) return param > 0.0 && param <= 1.0;
  if (mode == VECATTN_SEL_MINS || mode == VECATTN_SEL_MINS_TILED) return param >= 0.0;
  return false;
}

// Tile of 16 or 32 keys; a power-of-two number of tiles per group, at most
// 2^30 keys per group.
bool tiling_ok(int32_t tile, int32_t group_tiles) {
  if (tile != 16 && tile != 32) return false;
  if (group_tiles < 1 || (group_tiles & (group_tiles - 1)) != 0) return false;
  return static_cast<int64_t>(tile) * group_tiles <= (int64_t(1) << 30);
}

// Bits of the `causal` argument of the selection entry points.
constexpr int32_t kCausal = VECATTN_CAUSAL, kKeepDiag = VECATTN_KEEP_DIAG,
                  kUnpadded = VECATTN_UNPADDED;
// Bits the selection entry points accept.
constexpr int32_t kSelBits = kCausal | kKeepDiag | kUnpadded;

// Largest count any block can produce.  Without the diagonal, k_i is
// non-decreasing in L_i, so the largest L_i decides; with it (block i adds
// its own n_i rows' keys), the largest min(L_i, k_i + n_i).  Every block but
// the last has n_i = P and L_i, k_i non-decreasing in i, so that value is
// non-decreasing over them: the last two blocks decide.
int64_t max_count(int64_t N, int32_t P, int32_t flags, int32_t mode, double param) {
  const bool causal = (flags & kCausal) != 0;
  const int64_t Np = num_blocks(N, P);
  const int64_t Lmax = causal ? std::min<int64_t>(N, Np * static_cast<int64_t>(P)) : N;
  if (mode != VECATTN_SEL_TOPK) return Lmax;
  if (!(flags & kKeepDiag)) return topk_count(param, Lmax);
  int64_t best = 0;
  for (int64_t i = std::max<int64_t>(0, Np - 2); i < Np; ++i) {
    const int64_t n_i = std::min<int64_t>(N, (i + 1) * P) - i * P;
    const int64_t L = causal ? std::min<int64_t>(N, (i + 1) * P) : N;
    best = std::max(best, std::min(L, topk_count(param, L) + n_i));
  }
  return best;
}

constexpr int64_t kMaxHeadParams = 128;  // query heads a per-head parameter list may cover

// The attention gathers K and V rows with 32-bit byte offsets inside one
// head: key j of a head sits at j * row_bytes, computed with a 24-bit
// multiply, and the head's rows must span < 2^31 bytes.  Heads beyond that
// are rejected (UNSUPPORTED) instead of gathering wrong rows.
bool gather_offsets_ok(const vecattn_tdesc* d) {
  const int64_t rowb = d->sN * 2;
  if (d->N >= (int64_t(1) << 24)) return false;
  if (d->N > 1 && rowb >= (int64_t(1) << 24)) return false;
  return (d->N - 1) * rowb + 2 * d->D < (int64_t(1) << 31);
}

// Every check of vecattn_sparse_attn, without launching anything.
vecattn_status check_attn(const void* q, const vecattn_tdesc* qd, const void* k,
                          const vecattn_tdesc* kd, const void* v, const vecattn_tdesc* vd,
                          const int32_t* idx, int64_t cap, const int32_t* counts, int32_t block,
                          int32_t causal, float scale, const void* o, const vecattn_tdesc* od) {
  vecattn_status st;
  if ((st = check_desc(q, qd)) != VECATTN_OK) return st;
  if ((st = check_desc(k, kd)) != VECATTN_OK) return st;
  if ((st = check_desc(v, vd)) != VECATTN_OK) return st;
  if ((st = check_desc(o, od)) != VECATTN_OK) return st;
  if (kd->B != qd->B || kd->N != qd->N || kd->D != qd->D || qd->H % kd->H != 0)
    return VECATTN_ERR_INVALID_ARG;
  if (vd->B != kd->B || vd->H != kd->H || vd->N != kd->N || vd->D != kd->D)
    return VECATTN_ERR_INVALID_ARG;
  if (od->B != qd->B || od->H != qd->H || od->N != qd->N || od->D != qd->D)
    return VECATTN_ERR_INVALID_ARG;
  if (!idx || !counts || block < 1 || cap < 1 || cap > kMaxN) return VECATTN_ERR_INVALID_ARG;
  if (!std::isfinite(scale) || scale < 0.0f) return VECATTN_ERR_INVALID_ARG;
  if ((causal & ~kSelBits) != 0) return VECATTN_ERR_INVALID_ARG;
  if (!gather_offsets_ok(kd) || !gather_offsets_ok(vd)) return VECATTN_ERR_UNSUPPORTED;
  return VECATTN_OK;
}

// Every argument check of the selection entry points except the workspace's;
// *need receives the workspace bytes the call needs.
vecattn_status select_check(const void* q, const vecattn_tdesc* qd, const void* k,
                            const vecattn_tdesc* kd, int32_t block, int32_t causal, int32_t mode,
                            double param, const double* head_params, int32_t tile,
                            int32_t group_tiles, const int32_t* idx, int64_t cap,
                            const int32_t* counts, size_t* need) {
  vecattn_status st = check_desc(q, qd);
  if (st != VECATTN_OK) return st;
  st = check_desc(k, kd);
  if (st != VECATTN_OK) return st;
  if (kd->B != qd->B || kd->N != qd->N || kd->D != qd->D || qd->H % kd->H != 0)
    return VECATTN_ERR_INVALID_ARG;
  if (!idx || !counts || block < 1 || cap < 1 || cap > kMaxN) return VECATTN_ERR_INVALID_ARG;
  if (!mode_ok(mode) || (causal & ~kSelBits) != 0) return VECATTN_ERR_INVALID_ARG;
  if (head_params) {
    if (qd->H > kMaxHeadParams) return VECATTN_ERR_UNSUPPORTED;
    for (int64_t h = 0; h < qd->H; ++h) {
      if (!param_ok(mode, head_params[h])) return VECATTN_ERR_INVALID_ARG;
      if (mode == VECATTN_SEL_TOPK && cap < max_count(qd->N, block, causal, mode, head_params[h]))
        return VECATTN_ERR_CAPACITY;
    }
    param = head_params[0];
  } else if (!param_ok(mode, param)) {
    return VECATTN_ERR_INVALID_ARG;
  }
  if (mode == VECATTN_SEL_MINS_TILED && !tiling_ok(tile, group_tiles))
    return VECATTN_ERR_INVALID_ARG;
  if (!head_params && mode == VECATTN_SEL_TOPK &&
      cap < max_count(qd->N, block, causal, mode, param))
    return VECATTN_ERR_CAPACITY;
  // With the diagonal kept, no block may be clamped: cap covers every count.
  if ((causal & kKeepDiag) && mode != VECATTN_SEL_TOPK &&
      cap < max_count(qd->N, block, causal, mode, param))
    return VECATTN_ERR_CAPACITY;
  *need = vecattn::select_workspace_bytes(qd->B, qd->H, kd->H, qd->N, qd->D, block, mode, cap);
  return VECATTN_OK;
}

vecattn_status select_impl(const void* q, const vecattn_tdesc* qd, const void* k,
                           const vecattn_tdesc* kd, int32_t block, int32_t causal, int32_t mode,
                           double param, const double* head_params, int32_t tile,
                           int32_t group_tiles, int32_t* idx, int64_t cap, int32_t* counts,
                           int32_t* n_clamped, void* workspace, size_t workspace_bytes,
                           void* stream) {
  size_t need = 0;
  const vecattn_status st = select_check(q, qd, k, kd, block, causal, mode, param, head_params,
                                         tile, group_tiles, idx, cap, counts, &need);
  if (st != VECATTN_OK) return st;
  if (need > 0 && (!workspace || workspace_bytes < need)) return VECATTN_ERR_CAPACITY;
  if (workspace && !aligned16(workspace)) return VECATTN_ERR_INVALID_ARG;
  if (head_params) param = head_params[0];
  vecattn::SelectArgs a{to_tensor(q, qd), to_tensor(k, kd), block, (causal & kCausal) ? 1 : 0,
                        (causal & kKeepDiag) ? 1 : 0, (causal & kUnpadded) ? 1 : 0, mode, param,
                        head_params, tile, group_tiles,
                        idx, cap, counts, n_clamped, workspace, workspace_bytes};
  hipError_t e = vecattn::launch_select(a, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

}  // namespace

extern "C" {

int32_t vecattn_version(void) { return 101; }

const char* vecattn_status_string(vecattn_status s) {
  switch (s) {
    case VECATTN_OK: return "ok";
    case VECATTN_ERR_INVALID_ARG: return "invalid argument";
    case VECATTN_ERR_UNSUPPORTED: return "unsupported";
    case VECATTN_ERR_CAPACITY: return "capacity too small";
    case VECATTN_ERR_DEVICE: return "device error";
  }
  return "unknown status";
}

vecattn_status vecattn_pool(const void* q, const vecattn_tdesc* qd, int32_t block, void* qp,
                            const vecattn_tdesc* qpd, void* stream) {
  vecattn_status st = check_desc(q, qd);
  if (st != VECATTN_OK) return st;
  if (block < 1) return VECATTN_ERR_INVALID_ARG;
  st = check_desc(qp, qpd);
  if (st != VECATTN_OK) return st;
  if (qpd->B != qd->B || qpd->H != qd->H || qpd->D != qd->D || qpd->N != num_blocks(qd->N, block))
    return VECATTN_ERR_INVALID_ARG;
  hipError_t e = vecattn::launch_pool(to_tensor(q, qd), block, qp, qpd->sB, qpd->sH, qpd->sN,
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

vecattn_status vecattn_select_max_count(int64_t N, int32_t block, int32_t causal, int32_t mode,
                                        double param, int64_t* out) {
  if (!out || N < 1 || N > kMaxN || block < 1 || !mode_ok(mode) || !param_ok(mode, param) ||
      (causal & ~kSelBits) != 0)
    return VECATTN_ERR_INVALID_ARG;
  *out = max_count(N, block, causal, mode, param);
  return VECATTN_OK;
}

vecattn_status vecattn_select_workspace_size(const vecattn_tdesc* qd, const vecattn_tdesc* kd,
                                             int32_t block, int32_t causal, int32_t mode,
                                             int64_t cap, size_t* bytes) {
  (void)causal;
  if (!qd || !kd || !bytes || block < 1 || cap < 1) return VECATTN_ERR_INVALID_ARG;
  if (!mode_ok(mode) || qd->B < 1 || qd->H < 1 || qd->N < 1 || qd->N > kMaxN || kd->H < 1 ||
      qd->H % kd->H != 0 || (qd->D != 64 && qd->D != 128))
    return VECATTN_ERR_INVALID_ARG;
  *bytes = vecattn::select_workspace_bytes(qd->B, qd->H, kd->H, qd->N, qd->D, block, mode, cap);
  return VECATTN_OK;
}

size_t vecattn_select_workspace_bytes(const vecattn_tdesc* qd, const vecattn_tdesc* kd,
                                      int32_t block, int32_t mode, int64_t cap) {
  size_t n = 0;
  return vecattn_select_workspace_size(qd, kd, block, 0, mode, cap, &n) == VECATTN_OK ? n : 0;
}

vecattn_status vecattn_head_sparsity(const int32_t* counts, int64_t B, int64_t Hq, int64_t N,
                                     int32_t block, int32_t causal, double* sparsity,
                                     void* stream) {
  if (!counts || !sparsity || B < 1 || Hq < 1 || Hq > INT32_MAX || N < 1 || N > kMaxN ||
      block < 1 || (causal & ~kSelBits) != 0)
    return VECATTN_ERR_INVALID_ARG;
  hipError_t e = vecattn::launch_head_sparsity(counts, B, Hq, N, block, (causal & kCausal) ? 1 : 0,
                                               sparsity, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

vecattn_status vecattn_recall(const void* q, const vecattn_tdesc* qd, const void* k,
                              const vecattn_tdesc* kd, const int32_t* idx, int64_t cap,
                              const int32_t* counts, int32_t block, int32_t causal, float scale,
                              float* kept, void* stream) {
  vecattn_status st = check_desc(q, qd);
  if (st != VECATTN_OK) return st;
  if ((st = check_desc(k, kd)) != VECATTN_OK) return st;
  if (kd->B != qd->B || kd->N != qd->N || kd->D != qd->D || qd->H % kd->H != 0)
    return VECATTN_ERR_INVALID_ARG;
  if (!idx || !counts || !kept || block < 1 || cap < 1 || cap > kMaxN)
    return VECATTN_ERR_INVALID_ARG;
  if (!std::isfinite(scale) || scale < 0.0f) return VECATTN_ERR_INVALID_ARG;
  if ((causal & ~kSelBits) != 0) return VECATTN_ERR_INVALID_ARG;
  if (qd->N > vecattn::kRecallMaxN) return VECATTN_ERR_UNSUPPORTED;
  vecattn::RecallArgs a{to_tensor(q, qd), to_tensor(k, kd), idx, counts, cap, block,
                        (causal & kCausal) ? 1 : 0, scale, kept};
  hipError_t e = vecattn::launch_recall(a, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

vecattn_status vecattn_select(const void* q, const vecattn_tdesc* qd, const void* k,
                              const vecattn_tdesc* kd, int32_t block, int32_t causal, int32_t mode,
                              double param, int32_t* idx, int64_t cap, int32_t* counts,
                              int32_t* n_clamped, void* workspace, size_t workspace_bytes,
                              void* stream) {
  // Cross-tile minS through this entry point uses the paper's B_K = G_K = 16.
  return select_impl(q, qd, k, kd, block, causal, mode, param, nullptr, 16, 16, idx, cap, counts,
                     n_clamped, workspace, workspace_bytes, stream);
}

vecattn_status vecattn_select_noalloc(const void* q, const vecattn_tdesc* qd, const void* k,
                                      const vecattn_tdesc* kd, int32_t block, int32_t causal,
                                      int32_t mode, double param, int32_t* idx, int64_t cap,
                                      int32_t* counts, int32_t* n_clamped, void* stream) {
  // All checks first (no device call on an error), then the size limit, then
  // this GPU's copy of the library's workspace.
  size_t need = 0;
  vecattn_status st = select_check(q, qd, k, kd, block, causal, mode, param, nullptr, 16, 16, idx,
                                   cap, counts, &need);
  if (st != VECATTN_OK) return st;
  if (need > vecattn::kStaticWorkspaceBytes) return VECATTN_ERR_CAPACITY;
  void* ws = nullptr;
  if (vecattn::static_workspace(&ws) != hipSuccess) return VECATTN_ERR_DEVICE;
  return select_impl(q, qd, k, kd, block, causal, mode, param, nullptr, 16, 16, idx, cap, counts,
                     n_clamped, ws, vecattn::kStaticWorkspaceBytes, stream);
}

vecattn_status vecattn_select_per_head(const void* q, const vecattn_tdesc* qd, const void* k,
                                       const vecattn_tdesc* kd, int32_t block, int32_t causal,
                                       int32_t mode, const double* params, int32_t tile,
                                       int32_t group_tiles, int32_t* idx, int64_t cap,
                                       int32_t* counts, int32_t* n_clamped, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  if (!params) return VECATTN_ERR_INVALID_ARG;
  return select_impl(q, qd, k, kd, block, causal, mode, 0.0, params, tile, group_tiles, idx, cap,
                     counts, n_clamped, workspace, workspace_bytes, stream);
}

vecattn_status vecattn_select_mins_tiled(const void* q, const vecattn_tdesc* qd, const void* k,
                                         const vecattn_tdesc* kd, int32_t block, int32_t causal,
                                         double alpha, int32_t tile, int32_t group_tiles,
                                         int32_t* idx, int64_t cap, int32_t* counts,
                                         int32_t* n_clamped, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  return select_impl(q, qd, k, kd, block, causal, VECATTN_SEL_MINS_TILED, alpha, nullptr, tile,
                     group_tiles, idx, cap, counts, n_clamped, workspace, workspace_bytes, stream);
}

vecattn_status vecattn_sparse_attn_ordered(const void* q, const vecattn_tdesc* qd, const void* k,
                                           const vecattn_tdesc* kd, const void* v,
                                           const vecattn_tdesc* vd, const int32_t* idx,
                                           int64_t cap, const int32_t* counts,
                                           const int32_t* order, int32_t block, int32_t causal,
                                           float scale, void* o, const vecattn_tdesc* od,
                                           float* lse, void* stream) {
  const vecattn_status st =
      check_attn(q, qd, k, kd, v, vd, idx, cap, counts, block, causal, scale, o, od);
  if (st != VECATTN_OK) return st;
  vecattn::SparseAttnArgs a{to_tensor(q, qd), to_tensor(k, kd), to_tensor(v, vd),
                            o, od->sB, od->sH, od->sN, lse, idx, counts, cap, block,
                            (causal & kCausal) ? 1 : 0, scale, order};
  hipError_t e = vecattn::launch_sparse_attn(a, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

vecattn_status vecattn_sparse_attn(const void* q, const vecattn_tdesc* qd, const void* k,
                                   const vecattn_tdesc* kd, const void* v, const vecattn_tdesc* vd,
                                   const int32_t* idx, int64_t cap, const int32_t* counts,
                                   int32_t block, int32_t causal, float scale, void* o,
                                   const vecattn_tdesc* od, float* lse, void* stream) {
  return vecattn_sparse_attn_ordered(q, qd, k, kd, v, vd, idx, cap, counts, nullptr, block, causal,
                                     scale, o, od, lse, stream);
}

vecattn_status vecattn_attn_order(const int32_t* idx, int64_t cap, const int32_t* counts,
                                  int64_t B, int32_t Hq, int64_t N, int32_t block, int32_t* order,
                                  void* stream) {
  if (!idx || !counts || !order || B < 1 || Hq < 1 || N < 1 || N > kMaxN || block < 1 ||
      cap < 1 || cap > kMaxN || B * Hq > INT32_MAX)
    return VECATTN_ERR_INVALID_ARG;
  const int64_t Np = (N + block - 1) / block;
  hipError_t e = vecattn::launch_attn_order(idx, cap, counts, B * Hq, static_cast<int32_t>(Np), N,
                                            order, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

vecattn_status vecattn_check_lists(const int32_t* idx, int64_t rows, int64_t cap,
                                   const int32_t* counts, int64_t n_keys, int32_t* n_bad,
                                   void* stream) {
  if (!n_bad || rows < 0 || rows > INT32_MAX || cap < 1 || cap > kMaxN || n_keys < 1 ||
      n_keys > kMaxN)
    return VECATTN_ERR_INVALID_ARG;
  if (rows > 0 && (!idx || !counts)) return VECATTN_ERR_INVALID_ARG;
  hipError_t e = vecattn::launch_check_lists(idx, counts, rows, cap, n_keys, n_bad,
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? VECATTN_OK : VECATTN_ERR_DEVICE;
}

}  // extern "C"

namespace {

// Packed variable-length batches: sequence s is rows [cu[s], cu[s+1]) of the
// B = 1 tensors; its blocks, lists and counts follow those of the sequences
// before it.
bool cu_ok(const int64_t* cu, int32_t nseq, int64_t total) {
  if (!cu || nseq < 1 || cu[0] != 0 || cu[nseq] != total) return false;
  for (int32_t s = 0; s < nseq; ++s)
    if (cu[s + 1] < cu[s]) return false;
  return true;
}

vecattn_tdesc seq_desc(const vecattn_tdesc* d, int64_t n) {
  vecattn_tdesc r = *d;
  r.N = n;
  return r;
}

const void* seq_ptr(const void* p, const vecattn_tdesc* d, int64_t row) {
  return static_cast<const char*>(p) + row * d->sN * 2;  // bf16 elements
}

}  // namespace

extern "C" {

vecattn_status vecattn_select_varlen(const void* q, const vecattn_tdesc* qd, const void* k,
                                     const vecattn_tdesc* kd, const int64_t* cu_seqlens,
                                     int32_t nseq, int32_t block, int32_t causal, int32_t mode,
                                     double param, int32_t* idx, int64_t cap, int32_t* counts,
                                     int32_t* n_clamped, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  vecattn_status st = check_desc(q, qd);
  if (st != VECATTN_OK) return st;
  if ((st = check_desc(k, kd)) != VECATTN_OK) return st;
  if (qd->B != 1 || kd->B != 1 || kd->N != qd->N || kd->D != qd->D || qd->H % kd->H != 0)
    return VECATTN_ERR_INVALID_ARG;
  if (!cu_ok(cu_seqlens, nseq, qd->N) || !idx || !counts || block < 1 || cap < 1 || cap > kMaxN)
    return VECATTN_ERR_INVALID_ARG;
  if (!mode_ok(mode) || !param_ok(mode, param) || (causal & ~kSelBits) != 0)
    return VECATTN_ERR_INVALID_ARG;
  // Every sequence's checks first, so that an error launches nothing.
  for (int32_t s = 0; s < nseq; ++s) {
    const int64_t n = cu_seqlens[s + 1] - cu_seqlens[s];
    if (n == 0) continue;
    if ((mode == VECATTN_SEL_TOPK || (causal & kKeepDiag)) &&
        cap < max_count(n, block, causal, mode, param))
      return VECATTN_ERR_CAPACITY;
    const size_t need = vecattn::select_workspace_bytes(1, qd->H, kd->H, n, qd->D, block, mode, cap);
    if (need > 0 && (!workspace || workspace_bytes < need)) return VECATTN_ERR_CAPACITY;
  }
  int64_t blocks = 0;  // blocks of the sequences before s
  for (int32_t s = 0; s < nseq; ++s) {
    const int64_t n = cu_seqlens[s + 1] - cu_seqlens[s];
    if (n == 0) continue;
    const vecattn_tdesc qs = seq_desc(qd, n), ks = seq_desc(kd, n);
    st = select_impl(seq_ptr(q, qd, cu_seqlens[s]), &qs, seq_ptr(k, kd, cu_seqlens[s]), &ks, block,
                     causal, mode, param, nullptr, 16, 16, idx + blocks * qd->H * cap, cap,
                     counts + blocks * qd->H, n_clamped, workspace, workspace_bytes, stream);
    if (st != VECATTN_OK) return st;
    blocks += num_blocks(n, block);
  }
  return VECATTN_OK;
}

vecattn_status vecattn_sparse_attn_varlen(const void* q, const vecattn_tdesc* qd, const void* k,
                                          const vecattn_tdesc* kd, const void* v,
                                          const vecattn_tdesc* vd, const int64_t* cu_seqlens,
                                          int32_t nseq, const int32_t* idx, int64_t cap,
                                          const int32_t* counts, int32_t block, int32_t causal,
                                          float scale, void* o, const vecattn_tdesc* od,
                                          float* lse, void* stream) {
  // The whole packed tensors first (sizes, strides, the relations between
  // Q, K, V and O), then every sequence's view, so that an error launches
  // nothing.
  vecattn_status st = check_attn(q, qd, k, kd, v, vd, idx, cap, counts, block, causal, scale, o, od);
  if (st != VECATTN_OK) return st;
  if (qd->B != 1 || kd->B != 1 || vd->B != 1 || od->B != 1) return VECATTN_ERR_INVALID_ARG;
  if (!cu_ok(cu_seqlens, nseq, qd->N)) return VECATTN_ERR_INVALID_ARG;
  for (int32_t s = 0; s < nseq; ++s) {
    const int64_t n = cu_seqlens[s + 1] - cu_seqlens[s];
    if (n == 0) continue;
    const int64_t r0 = cu_seqlens[s];
    const vecattn_tdesc qs = seq_desc(qd, n), ks = seq_desc(kd, n), vs = seq_desc(vd, n),
                        os = seq_desc(od, n);
    st = check_attn(seq_ptr(q, qd, r0), &qs, seq_ptr(k, kd, r0), &ks, seq_ptr(v, vd, r0), &vs, idx,
                    cap, counts, block, causal, scale, seq_ptr(o, od, r0), &os);
    if (st != VECATTN_OK) return st;
  }
  int64_t blocks = 0;
  for (int32_t s = 0; s < nseq; ++s) {
    const int64_t n = cu_seqlens[s + 1] - cu_seqlens[s];
    if (n == 0) continue;
    const int64_t r0 = cu_seqlens[s];
    const vecattn_tdesc qs = seq_desc(qd, n), ks = seq_desc(kd, n), vs = seq_desc(vd, n),
                        os = seq_desc(od, n);
    st = vecattn_sparse_attn(seq_ptr(q, qd, r0), &qs, seq_ptr(k, kd, r0), &ks, seq_ptr(v, vd, r0),
                             &vs, idx + blocks * qd->H * cap, cap, counts + blocks * qd->H, block,
                             causal, scale, const_cast<void*>(seq_ptr(o, od, r0)), &os,
                             lse ? lse + qd->H * r0 : nullptr, stream);
    if (st != VECATTN_OK) return st;
    blocks += num_blocks(n, block);
  }
  return VECATTN_OK;
}

vecattn_status vecattn_plan_filter_ratios(int32_t heads, int32_t n_cand, const double* sparsity,
                                          const double* perf, double target, int32_t grid,
                                          int32_t* choice, double* best_perf) {
  if (heads < 1 || n_cand < 1 || !sparsity || !perf || !choice || !best_perf)
    return VECATTN_ERR_INVALID_ARG;
  if (grid < 1 || grid > (1 << 20) || !(target >= 0.0 && target <= 1.0))
    return VECATTN_ERR_INVALID_ARG;
  if (static_cast<int64_t>(heads) * grid > (int64_t(1) << 26)) return VECATTN_ERR_INVALID_ARG;
  for (int64_t t = 0; t < static_cast<int64_t>(heads) * n_cand; ++t)
    if (!(sparsity[t] >= 0.0 && sparsity[t] <= 1.0) || !std::isfinite(perf[t]))
      return VECATTN_ERR_INVALID_ARG;
  return vecattn::plan_filter_ratios(heads, n_cand, sparsity, perf, target, grid, choice,
                                     best_perf) == 0
             ? VECATTN_OK
             : VECATTN_ERR_CAPACITY;
}

}  // extern "C"
