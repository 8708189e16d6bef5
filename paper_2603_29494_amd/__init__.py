"""vecattn: vertical-vector sparse attention for AMD MI355X (gfx950).

After VecAttention (arXiv 2603.29494): per query block, pool the queries
(Eq. 2), score every key with the pooled query and keep the important key
columns (row-wise topK budget, topP mass threshold, or the minS filter of
Eq. 3, also with Algorithm 1's cross-tile running maximum; Sec. 3.1), then run
attention restricted to the gathered K/V rows of those columns (Eq. 4,
Algorithm 2).  Both stages are HIP kernels in libvecattn.so behind the C ABI
of include/vecattn.h; this package only marshals torch tensors to it.
"""
from ._lib import (SEL_MINS, SEL_MINS_TILED, SEL_TOPK, SEL_TOPP, VecattnError, attn_order,
                   check_lists,
                   head_sparsity, head_sparsity_of, load, max_count, plan_filter_ratios, pool,
                   recall, select, select_varlen, sparse_attn, sparse_attn_varlen, varlen_blocks,
                   workspace_bytes)

__all__ = ["SEL_TOPK", "SEL_TOPP", "SEL_MINS", "SEL_MINS_TILED", "VecattnError", "attn_order",
           "check_lists",
           "head_sparsity", "head_sparsity_of", "recall",
           "load", "max_count", "plan_filter_ratios", "pool", "select", "select_varlen",
           "sparse_attn", "sparse_attn_varlen", "varlen_blocks", "workspace_bytes"]
