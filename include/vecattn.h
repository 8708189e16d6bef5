/*
 * vecattn.h -- C ABI of libvecattn, vertical-vector sparse attention for
 * AMD Instinct MI355X (gfx950), after VecAttention (arXiv 2603.29494).
 *
 * The method has two stages (paper, Sec. 3 and appendix algorithms 1-2):
 *   1. vecattn_select: for every query block of P rows, pool the block's
 *      queries (Eq. 2), score every eligible key with the pooled query
 *      (estimated map A_p, Sec. 3.1.1) and keep the important key columns
 *      ("vertical vectors") by a budget (row-wise topK) or a cumulative-mass
 *      threshold (row-wise topP), Sec. 3.1.2, or the minS filter (Eq. 3), also
 *      with Algorithm 1's cross-tile running maximum (vecattn_select_mins_tiled).
 *      Output: the index matrix I and count vector C of Algorithm 1.
 *   2. vecattn_sparse_attn: attention of each query block restricted to the
 *      gathered K/V rows of its selected keys (Eq. 4, Algorithm 2).
 *
 * Conventions shared by every entry point
 *   - Tensors are caller-owned device memory.  The library never allocates,
 *     frees or synchronises; every call is asynchronous on `stream` (a
 *     hipStream_t; NULL means the default stream), and calls on different
 *     streams may run concurrently.  The only state kept between calls is a
 *     per-process, per-device locality counter of vecattn_sparse_attn (the
 *     progress of the workgroups on each XCD through their lists, which paces
 *     the order in which a workgroup walks its list; non-causal calls only):
 *     concurrent calls share it, which changes their speed and the order of
 *     the softmax sums (the last bits of O), never which keys are attended.
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
 *     entries; the remaining entries are -1 (left unwritten with
 *     VECATTN_UNPADDED).  C (counts) is int32 [B, Hq, N_p].
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
  VECATTN_SEL_MINS = 2, /* param = alpha >= 0 (Eq. 3, minS): block i keeps every
                           eligible key whose score is >= its largest score
                           minus alpha (alpha = +inf keeps all) */
  VECATTN_SEL_MINS_TILED = 3 /* param = alpha >= 0: minS against Algorithm 1's
                           cross-tile running maximum (Sec. 3.1.3), with the
                           paper's B_K = 16 keys per tile and G_K = 16 tiles per
                           group; see vecattn_select_mins_tiled */
} vecattn_sel_mode;

/* Bits of the `causal` argument of the selection entry points.  0 (none) and
 * 1 (VECATTN_CAUSAL) keep their plain meaning; bits other than these three are
 * invalid. */
#define VECATTN_CAUSAL 1    /* block i's eligible keys end at its last row */
#define VECATTN_KEEP_DIAG 2 /* block i also keeps the keys of its own rows,
                               [i*P, min(N, (i+1)*P)); cap must then cover
                               vecattn_select_max_count for the same flags in
                               every mode (no block is clamped) */
#define VECATTN_UNPADDED 4  /* the entries of I past a row's count are left as
                               they were instead of being set to -1 (the
                               attention and vecattn_check_lists read only the
                               first C entries): with a large cap (threshold
                               modes, cap = N) this saves writing the padding */

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
 * Largest number of keys any block can select, for sizing cap.  topK: max_i k_i
 * (with VECATTN_KEEP_DIAG: max_i min(L_i, k_i + n_i), n_i the rows of block i);
 * the other modes: max_i L_i, where L_i = N (non-causal) or min(N, (i+1)*P)
 * (causal).  `causal` takes the same bits as vecattn_select.
 * Errors: INVALID_ARG for N < 1, block < 1, out == NULL, or param outside the
 * mode's range.
 */
vecattn_status vecattn_select_max_count(int64_t N, int32_t block, int32_t causal, int32_t mode,
                                        double param, int64_t* out);

/*
 * Workspace bytes vecattn_select needs for these shapes (device memory the
 * caller allocates and passes in; contents need not be initialised).  The
 * size depends on B, Hq, Hkv (kd->H), N, D and block.
 * Errors: INVALID_ARG (a NULL pointer, block < 1, cap < 1, an unknown mode,
 * sizes < 1 or N > 2^30, Hq % Hkv != 0, D not in {64, 128}).
 */
vecattn_status vecattn_select_workspace_size(const vecattn_tdesc* qd, const vecattn_tdesc* kd,
                                             int32_t block, int32_t causal, int32_t mode,
                                             int64_t cap, size_t* bytes);

/* The same size as a return value (0 when vecattn_select_workspace_size would
 * return an error). */
size_t vecattn_select_workspace_bytes(const vecattn_tdesc* qd, const vecattn_tdesc* kd,
                                      int32_t block, int32_t mode, int64_t cap);

/*
 * Important-vector selection (Sec. 3.1; Algorithm 1's outputs I and C).
 *   q : bf16 [B, Hq, N, D]    k : bf16 [B, Hkv, N, D]
 *   causal : VECATTN_CAUSAL and/or VECATTN_KEEP_DIAG bits.  Block i's
 *   eligible keys are j in [0, N), or j in [0, min(N, (i+1)*P)) with
 *   VECATTN_CAUSAL.  With VECATTN_KEEP_DIAG the block's list is the union of
 *   the mode's selection and the keys of its own rows (a practical variant
 *   the paper leaves open: local keys always attended).  Scores are <Q_p[i], k_j> / sqrt(D)
 *   with Q_p from vecattn_pool, computed from bf16 products accumulated in
 *   fp32.  Ties in score are broken toward the lower key index.
 *   idx    : int32 [B, Hq, N_p, cap] output (ascending lists, -1 padded)
 *   counts : int32 [B, Hq, N_p] output
 *   n_clamped : optional device int32; when not NULL, the number of blocks
 *            whose threshold-mode selection exceeded cap is ADDED to it
 *            (topP and minS blocks keep their cap highest-scoring keys;
 *            cross-tile minS blocks their first cap keys).
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
 * vecattn_select without a caller workspace, for callers that cannot allocate
 * device memory (code under stream capture, tight serving loops, harnesses
 * that forbid allocation).  The workspace is a 64 MiB array inside the library
 * (VECATTN_STATIC_WORKSPACE_BYTES), one copy per GPU the library runs on, held
 * until the process ends; the call allocates nothing.  Arguments and results
 * are those of vecattn_select.  Every call on a GPU uses that GPU's one copy
 * (the current device's): calls that overlap on one GPU (other streams, other
 * threads) race and must be serialised by the caller.
 * Errors: as vecattn_select; CAPACITY when vecattn_select_workspace_size for
 * these shapes exceeds VECATTN_STATIC_WORKSPACE_BYTES; DEVICE if the array's
 * device address cannot be obtained.
 */
#define VECATTN_STATIC_WORKSPACE_BYTES (64u << 20)
vecattn_status vecattn_select_noalloc(const void* q, const vecattn_tdesc* qd, const void* k,
                                      const vecattn_tdesc* kd, int32_t block, int32_t causal,
                                      int32_t mode, double param, int32_t* idx, int64_t cap,
                                      int32_t* counts, int32_t* n_clamped, void* stream);

/*
 * Important-vector selection with Algorithm 1's cross-tile minS filter
 * (appendix Algorithm 1; Sec. 3.1.3, "Cross-tile minS optimization"; the rule
 * is Eq. 3's with a running maximum in place of the row maximum).  Block i's
 * eligible keys (as for vecattn_select) fall into groups of tile * group_tiles
 * consecutive keys, the first starting at key 0; inside a group the tiles of
 * `tile` keys are visited in ascending order, and a key of tile t is kept when
 * its score is >= (largest score in the group's tiles 0..t) - alpha.  Scores
 * are computed as for vecattn_select; alpha = +inf keeps every eligible key.
 *   tile        : B_K, 16 or 32 keys
 *   group_tiles : G_K, a power of two, tile * group_tiles <= 2^30 (a group
 *                 longer than N makes the running maximum span the whole row)
 *   idx, counts, workspace : as for vecattn_select (workspace size from
 *            vecattn_select_workspace_size with mode VECATTN_SEL_MINS_TILED)
 *   n_clamped : optional device int32; the number of blocks that selected more
 *            than cap keys is ADDED to it.  Such a block keeps its first cap
 *            selected keys in key order (the order in which Algorithm 1 appends
 *            its tiles) and reports count = cap.
 * vecattn_select with mode VECATTN_SEL_MINS_TILED equals this call with
 * tile = 16, group_tiles = 16.
 * Errors: INVALID_ARG (null pointer, shape mismatch, block < 1, cap < 1, alpha
 * negative or NaN, tile not 16 or 32, group_tiles not a power of two or too
 * large); CAPACITY (workspace too small); UNSUPPORTED (D not in {64, 128}).
 */
vecattn_status vecattn_select_mins_tiled(const void* q, const vecattn_tdesc* qd, const void* k,
                                         const vecattn_tdesc* kd, int32_t block, int32_t causal,
                                         double alpha, int32_t tile, int32_t group_tiles,
                                         int32_t* idx, int64_t cap, int32_t* counts,
                                         int32_t* n_clamped, void* workspace,
                                         size_t workspace_bytes, void* stream);

/*
 * vecattn_select with one parameter per query head: params[h] (host memory,
 * Hq values) replaces `param` for query head h -- e.g. the per-head filter
 * ratios of Eq. 5 (vecattn_plan_filter_ratios).  tile and group_tiles apply
 * to VECATTN_SEL_MINS_TILED as in vecattn_select_mins_tiled and are ignored by
 * the other modes.  The values are read during the call; the buffer may be
 * reused as soon as it returns.
 * Errors: as vecattn_select, each params[h] checked against the mode's range
 * (topK: CAPACITY when cap is below any head's budget); INVALID_ARG for
 * params == NULL or, for cross-tile minS, a bad tiling; UNSUPPORTED for more
 * than 128 query heads.
 */
vecattn_status vecattn_select_per_head(const void* q, const vecattn_tdesc* qd, const void* k,
                                       const vecattn_tdesc* kd, int32_t block, int32_t causal,
                                       int32_t mode, const double* params, int32_t tile,
                                       int32_t group_tiles, int32_t* idx, int64_t cap,
                                       int32_t* counts, int32_t* n_clamped, void* workspace,
                                       size_t workspace_bytes, void* stream);

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
 *   causal : the VECATTN_CAUSAL bit (VECATTN_KEEP_DIAG and VECATTN_UNPADDED are
 *   accepted and have no effect here; other bits are invalid).
 *   scale : softmax scale; 0 means 1 / sqrt(D).
 *   lse   : optional fp32 [B, Hq, N] contiguous output, may be NULL.
 * Errors: INVALID_ARG (null pointer, shape mismatch, block < 1, cap < 1,
 * misalignment); UNSUPPORTED (D not in {64, 128}; or a K or V head the
 * gathers cannot address with 32-bit offsets: N >= 2^24, a row stride sN of
 * 2^23 elements or more (with N > 1), or (N - 1) * sN * 2 + 2 * D >= 2^31
 * bytes -- e.g. a packed [B, N, 3, H, D] QKV view with H * D = 5120 from
 * N ~ 69,900 on).
 */
vecattn_status vecattn_sparse_attn(const void* q, const vecattn_tdesc* qd, const void* k,
                                   const vecattn_tdesc* kd, const void* v, const vecattn_tdesc* vd,
                                   const int32_t* idx, int64_t cap, const int32_t* counts,
                                   int32_t block, int32_t causal, float scale, void* o,
                                   const vecattn_tdesc* od, float* lse, void* stream);

/*
 * Block schedule for vecattn_sparse_attn_ordered.  Eq. 4 and Algorithm 2 treat
 * the query blocks independently, so the order in which the attention takes
 * them changes only its speed.  This call orders the N_p blocks of each
 * (b, h) by:
 *   1. count C[b,h,i], largest first (the longest lists start first, so the
 *      workgroups of a head finish together, and lists of like length, which
 *      walk the keys at a like pace, run side by side and share cache hits);
 *   2. then a signature: the mean of the entries at positions
 *      floor((2j + 1) * C / 16), j = 0..7, of the list (each clamped to
 *      [0, N - 1]), as floor(sum * 64 / N) capped at 511, smallest first;
 *   3. then the block index, smallest first.
 * A head of more than 16384 blocks is ordered in consecutive segments of
 * 16384 blocks, each segment by the rules above (positions [16384 s,
 * 16384 (s + 1)) hold a permutation of the same blocks).
 *   idx, cap, counts : as for vecattn_sparse_attn (counts are clamped to
 *            [0, cap]; only the 8 sampled entries of each list are read)
 *   B, Hq, N, block  : the selection's shapes; N_p = ceil(N / block)
 *   order  : int32 [B, Hq, N_p] device output; row (b, h) is a permutation of
 *            [0, N_p)
 * Asynchronous on `stream`; one read of counts and of the sampled entries.
 * Errors: INVALID_ARG (a NULL pointer, B, Hq, N or block < 1, N or cap
 * outside [1, 2^30], B * Hq > 2^31 - 1).
 */
vecattn_status vecattn_attn_order(const int32_t* idx, int64_t cap, const int32_t* counts,
                                  int64_t B, int32_t Hq, int64_t N, int32_t block, int32_t* order,
                                  void* stream);

/*
 * vecattn_sparse_attn taking the blocks of each (b, h) in a given order:
 *   order : int32 [B, Hq, N_p] device memory, row (b, h) a permutation of
 *           [0, N_p) (e.g. from vecattn_attn_order), or NULL for the
 *           ascending order (then this is vecattn_sparse_attn).  Entries are
 *           clamped to [0, N_p); a row that is not a permutation leaves the
 *           blocks missing from it unwritten.
 * Every other argument, the results and the errors are those of
 * vecattn_sparse_attn (the order of the softmax sums, and so the last bits
 * of O, can differ between calls, as there).
 */
vecattn_status vecattn_sparse_attn_ordered(const void* q, const vecattn_tdesc* qd, const void* k,
                                           const vecattn_tdesc* kd, const void* v,
                                           const vecattn_tdesc* vd, const int32_t* idx,
                                           int64_t cap, const int32_t* counts,
                                           const int32_t* order, int32_t block, int32_t causal,
                                           float scale, void* o, const vecattn_tdesc* od,
                                           float* lse, void* stream);

/*
 * Checker for the index input of vecattn_sparse_attn, for lists that did not
 * come from vecattn_select.  Sets *n_bad (device int32, cleared by the call)
 * to the number of rows whose list breaks the attention's contract: a count
 * outside [0, cap], or among the row's first `count` entries one outside
 * [0, n_keys) or one not strictly above the entry before it.  Entries past a
 * row's count are not read.
 *   idx    : int32 [rows, cap], contiguous (e.g. [B, Hq, N_p, cap] as rows =
 *            B * Hq * N_p)            counts : int32 [rows]
 *   n_keys : N of the keys the lists index
 * One read of the listed entries (4 bytes each); asynchronous on `stream`.
 * Errors: INVALID_ARG (n_bad NULL, idx or counts NULL with rows > 0, rows < 0
 * or > 2^31 - 1, cap < 1, n_keys < 1, cap or n_keys > 2^30).
 */
vecattn_status vecattn_check_lists(const int32_t* idx, int64_t rows, int64_t cap,
                                   const int32_t* counts, int64_t n_keys, int32_t* n_bad,
                                   void* stream);

/*
 * Variable-length batches.  Sequences of different lengths packed along N of
 * B = 1 tensors: sequence s is rows [cu_seqlens[s], cu_seqlens[s+1]) (host
 * int64, nseq + 1 values, cu_seqlens[0] = 0, non-decreasing, last = N; empty
 * sequences are allowed).  Each sequence is handled exactly as a separate
 * B = 1 call on its rows (its key indices count from its first row); the
 * calls run one after another on `stream`.  Output layouts are the
 * per-sequence arrays laid end to end:
 *   idx    : int32, for each sequence [Hq, N_p(s), cap], N_p(s) = ceil(n_s / P)
 *   counts : int32, for each sequence [Hq, N_p(s)]
 *   lse    : fp32,  for each sequence [Hq, n_s] (optional)
 * Q, K, V, O rows are read and written in place (the [1, H, N, D] views).
 * The selection workspace must be sized (vecattn_select_workspace_size) for
 * the longest sequence.  Every argument is checked for every sequence before
 * the first launch.  Many short sequences cost one set of launches each.
 */
vecattn_status vecattn_select_varlen(const void* q, const vecattn_tdesc* qd, const void* k,
                                     const vecattn_tdesc* kd, const int64_t* cu_seqlens,
                                     int32_t nseq, int32_t block, int32_t causal, int32_t mode,
                                     double param, int32_t* idx, int64_t cap, int32_t* counts,
                                     int32_t* n_clamped, void* workspace, size_t workspace_bytes,
                                     void* stream);
vecattn_status vecattn_sparse_attn_varlen(const void* q, const vecattn_tdesc* qd, const void* k,
                                          const vecattn_tdesc* kd, const void* v,
                                          const vecattn_tdesc* vd, const int64_t* cu_seqlens,
                                          int32_t nseq, const int32_t* idx, int64_t cap,
                                          const int32_t* counts, int32_t block, int32_t causal,
                                          float scale, void* o, const vecattn_tdesc* od,
                                          float* lse, void* stream);

/*
 * Sparsity of each query head from a selection's counts: Eq. 5's sp_h
 * (Sec. 3.1.2), the table vecattn_plan_filter_ratios takes.
 *   sparsity[h] = 1 - (sum over b, i of counts[b, h, i]) / (B * sum_i L_i)
 * with L_i the eligible keys of block i (N, or min(N, (i + 1) * block) with
 * VECATTN_CAUSAL).  Integer sums, one fp64 division.
 *   counts   : int32 [B, Hq, N_p] (device, e.g. from vecattn_select)
 *   sparsity : fp64 [Hq] device output
 *   causal   : the selection's bits (VECATTN_KEEP_DIAG is accepted, no effect)
 * Errors: INVALID_ARG (NULL pointer, B, Hq or N < 1, N > 2^30, block < 1, bad
 * bits).
 */
vecattn_status vecattn_head_sparsity(const int32_t* counts, int64_t B, int64_t Hq, int64_t N,
                                     int32_t block, int32_t causal, double* sparsity,
                                     void* stream);

/*
 * Recall of a selected pattern, the statistic of the sparse-pattern study
 * (Sec. 2.2): for query row r of block i, the share of the row's exact
 * attention map that the block's list keeps,
 *   kept[b, h, r] = sum_{j in I[b,h,i,0:C) visible} exp(x_j) / sum_{j visible} exp(x_j),
 *   x_j = scale * <q_r, k_j>, visible = (j < N) and (causal == 0 or j <= r).
 * The mean of kept over rows is the recall of the pattern; 1 - keep ratio is
 * its sparsity.  One dense pass over the visible keys (2 * N * visible * D
 * MFMA FLOP per head), the list held as a bitmask in LDS.
 *   q : bf16 [B, Hq, N, D]   k : bf16 [B, Hkv, N, D]
 *   idx, counts, cap : as for vecattn_sparse_attn (entries outside [0, N) are
 *            ignored; a key listed twice counts once)
 *   scale : 0 means 1 / sqrt(D)
 *   kept  : fp32 [B, Hq, N] contiguous output
 * Errors: INVALID_ARG (null pointer, shape mismatch, block < 1, cap < 1, bad
 * scale or bits, misalignment); UNSUPPORTED (D not in {64, 128}, N > 2^18).
 */
vecattn_status vecattn_recall(const void* q, const vecattn_tdesc* qd, const void* k,
                              const vecattn_tdesc* kd, const int32_t* idx, int64_t cap,
                              const int32_t* counts, int32_t block, int32_t causal, float scale,
                              float* kept, void* stream);

/*
 * Per-head filter ratios, Eq. 5 (Sec. 3.1.2).  Host function (host memory, no
 * GPU).
 * For each of `heads` heads, n_cand candidate filter ratios were sampled
 * offline with their sparsity sp[h][c] in [0, 1] and a performance score
 * perf[h][c] (any finite value, larger is better).  The call picks one
 * candidate per head so that the mean sparsity over the heads is >= target
 * and the summed performance is largest: Eq. 5's table over heads and
 * sparsity, kept as the summed sparsity with each sp[h][c] rounded to a
 * multiple of 1 / grid.  Ties go to the lower candidate index.
 *   sparsity, perf : double [heads][n_cand], row-major
 *   choice         : int32 [heads] output, the chosen candidate per head
 *   best_perf      : output, the summed performance of that choice
 * Errors: INVALID_ARG (null pointer, heads or n_cand < 1, target outside
 * [0, 1], sparsity outside [0, 1] or non-finite perf, grid < 1 or
 * heads * grid > 2^26); CAPACITY (no choice reaches the target).
 */
vecattn_status vecattn_plan_filter_ratios(int32_t heads, int32_t n_cand, const double* sparsity,
                                          const double* perf, double target, int32_t grid,
                                          int32_t* choice, double* best_perf);

#ifdef __cplusplus
}
#endif

#endif /* VECATTN_H */
