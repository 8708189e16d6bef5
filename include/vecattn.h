/*
 * vecattn.h -- C ABI of libvecattn, vertical-vector sparse attention for
 * AMD Instinct MI355X (gfx950), after VecAttention (arXiv 2603.29494).
 *
 * The method has two stages (paper, Sec. 3 and appendix algorithms 1-2):
 *   1. vecattn_select: for every query block of P rows, pool the block's
 *      queries (Eq. 2), score every eligible key with the pooled query
 *      (estimated map A_p, Sec. 3.1.1) and keep the important key columns
 *      ("vertical vectors") by a budget (row-wise topK) or a cumulative-mass
 *      threshold (row-wise topP), Sec. 3.1.2.  Output: the index matrix I and
 *      count vector C of Algorithm 1.
 *   2. vecattn_sparse_attn: attention of each query block restricted to the
 *      gathered K/V rows of its selected keys (Eq. 4, Algorithm 2).
 *
 * Conventions shared by every entry point
 *   - Tensors are caller-owned device memory.  The library never allocates,
 *     frees or synchronises; every call is asynchronous on `stream` (a
 *     hipStream_t; NULL means the default stream) and keeps no state, so calls
 *     on different streams may run concurrently.
 *   - Q, K, V, O are bf16 with logical shape [B, H, N, D] described by a
 *     vecattn_tdesc: sizes plus element strides sB, sH, sN; the D dimension is
 *     contiguous (stride 1).  Every row start must be 16-byte aligned (base
 *     pointer 16-byte aligned, sB, sH, sN multiples of 8).  D must be 64 or 128.
 *   - Query heads Hq and key/value heads Hkv: Hq % Hkv == 0, and query head h
 *     reads key/value head h / (Hq / Hkv) (grouped-query attention).
 *   - Blocks: block = P >= 1 query rows; N_p = ceil(N / P); block i holds rows
 *     [i*P, min(N, (i+1)*P)) (the last block may be ragged).
 *   - I (idx) is int32 [B, Hq, N_p, cap], contiguous.  Row (b, h, i) lists the
 *     selected keys of block i in strictly ascending order in its first C[b,h,i]
 *     entries; the remaining entries are -1.  C (counts) is int32 [B, Hq, N_p].
 *   - Argument errors are detected on the host before any launch and return a
 *     status without touching memory.  Launch failures return
 *     VECATTN_ERR_DEVICE.
 */
#ifndef VECATTN_H
#define VECATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum vecattn_status {
  VECATTN_OK = 0,
  VECATTN_ERR_INVALID_ARG = 1, /* null pointer, bad size/stride/alignment, bad parameter */
  VECATTN_ERR_UNSUPPORTED = 2, /* valid request this build does not implement (e.g. D=96) */
  VECATTN_ERR_CAPACITY = 3,    /* cap smaller than a topK budget, or workspace too small */
  VECATTN_ERR_DEVICE = 4       /* a HIP call or kernel launch failed */
} vecattn_status;

typedef enum vecattn_sel_mode {
  VECATTN_SEL_TOPK = 0, /* param = keep ratio r in (0, 1]: block i keeps
                           k_i = min(L_i, max(1, ceil(r * L_i - 1e-9))) keys */
  VECATTN_SEL_TOPP = 1, /* param = mass p in (0, 1]: block i keeps the shortest
                           prefix, in (score desc, index asc) order, whose softmax
                           mass over its eligible keys is >= p */
  VECATTN_SEL_MINS = 2  /* param = alpha >= 0 (Eq. 3, minS): block i keeps every
                           eligible key whose score is >= its largest score
                           minus alpha (alpha = +inf keeps all) */
} vecattn_sel_mode;

typedef struct vecattn_tdesc {
  int64_t B, H, N, D; /* logical sizes */
  int64_t sB, sH, sN; /* element strides of the B, H and N dimensions */
} vecattn_tdesc;

/* Version of this ABI (major * 100 + minor). */
int32_t vecattn_version(void);

/* Human-readable name of a status code (static storage, never NULL). */
const char* vecattn_status_string(vecattn_status s);

/*
 * Query pooling, Eq. 2 (Sec. 3.1.1): qp[b, h, i, :] = bf16 rounding (nearest,
 * ties to even, applied once) of the exact mean of q's rows in block i.  The
 * ragged last block averages the rows it has.
 *   q  : bf16 [B, H, N, D] (qd)          qp : bf16 [B, H, N_p, D] (qpd, N = N_p)
 * Errors: INVALID_ARG for null pointers, block < 1, or qpd not matching
 * (B, H, N_p, D); UNSUPPORTED for D not in {64, 128}.
 */
vecattn_status vecattn_pool(const void* q, const vecattn_tdesc* qd, int32_t block, void* qp,
                            const vecattn_tdesc* qpd, void* stream);

/*
 * Largest number of keys any block can select, for sizing cap.  topK: max_i k_i;
 * topP: max_i L_i, where L_i = N (non-causal) or min(N, (i+1)*P) (causal).
 * Errors: INVALID_ARG for N < 1, block < 1, out == NULL, or param outside the
 * mode's range.
 */
vecattn_status vecattn_select_max_count(int64_t N, int32_t block, int32_t causal, int32_t mode,
                                        double param, int64_t* out);

/*
 * Workspace bytes vecattn_select needs for these shapes (device memory the
 * caller allocates and passes in; contents need not be initialised).
 */
vecattn_status vecattn_select_workspace_size(const vecattn_tdesc* qd, const vecattn_tdesc* kd,
                                             int32_t block, int32_t causal, int32_t mode,
                                             int64_t cap, size_t* bytes);

/*
 * Important-vector selection (Sec. 3.1; Algorithm 1's outputs I and C).
 *   q : bf16 [B, Hq, N, D]    k : bf16 [B, Hkv, N, D]
 *   Block i's eligible keys are j in [0, N) (causal = 0) or j in
 *   [0, min(N, (i+1)*P)) (causal != 0).  Scores are <Q_p[i], k_j> / sqrt(D)
 *   with Q_p from vecattn_pool, computed from bf16 products accumulated in
 *   fp32.  Ties in score are broken toward the lower key index.
 *   idx    : int32 [B, Hq, N_p, cap] output (ascending lists, -1 padded)
 *   counts : int32 [B, Hq, N_p] output
 *   n_clamped : optional device int32; when not NULL, the number of blocks
 *            whose threshold-mode selection exceeded cap is ADDED to it
 *            (those blocks keep their cap highest-scoring keys).
 *   workspace : device memory of at least vecattn_select_workspace_size bytes.
 * Errors: INVALID_ARG (null pointer, shape mismatch between q and k, block < 1,
 * param outside (0, 1] for topK / topP or negative / NaN for minS, cap < 1);
 * CAPACITY (topK with cap < max_i k_i, or a workspace that is too small);
 * UNSUPPORTED (D not in {64, 128}).
 */
vecattn_status vecattn_select(const void* q, const vecattn_tdesc* qd, const void* k,
                              const vecattn_tdesc* kd, int32_t block, int32_t causal, int32_t mode,
                              double param, int32_t* idx, int64_t cap, int32_t* counts,
                              int32_t* n_clamped, void* workspace, size_t workspace_bytes,
                              void* stream);

/*
 * Vector-sparse attention, Eq. 4 (Sec. 3.2) and Algorithm 2.  For query row r
 * of block i (head h), the visible keys are V_r = { j in I[b,h,i,0:C[b,h,i]] :
 * causal == 0 or j <= r }, and
 *   o[r] = sum_{j in V_r} softmax_j(scale * <q_r, k_j>) v_j,
 *   lse[r] = log sum_{j in V_r} exp(scale * <q_r, k_j>)   (natural log).
 * A row with no visible key gets o[r] = 0 and lse[r] = -inf.
 *   q, o : bf16 [B, Hq, N, D]      k, v : bf16 [B, Hkv, N, D]
 *   idx, counts : as produced by vecattn_select (any source is accepted if
 *   every listed key is in [0, N) and the lists are strictly ascending;
 *   other contents are undefined behaviour).
 *   scale : softmax scale; 0 means 1 / sqrt(D).
 *   lse   : optional fp32 [B, Hq, N] contiguous output, may be NULL.
 * Errors: INVALID_ARG (null pointer, shape mismatch, block < 1, cap < 1,
 * misalignment); UNSUPPORTED (D not in {64, 128}).
 */
vecattn_status vecattn_sparse_attn(const void* q, const vecattn_tdesc* qd, const void* k,
                                   const vecattn_tdesc* kd, const void* v, const vecattn_tdesc* vd,
                                   const int32_t* idx, int64_t cap, const int32_t* counts,
                                   int32_t block, int32_t causal, float scale, void* o,
                                   const vecattn_tdesc* od, float* lse, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* VECATTN_H */
