"""ctypes binding of libvecattn.so (include/vecattn.h).

Argument marshalling only: torch tensors become device pointers, tensor
descriptors and the current HIP stream; every step of the computation runs in
the library's HIP kernels.  There is no fallback: if the library is missing or
cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvecattn.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_DEVICE = range(5)
CAUSAL, KEEP_DIAG, UNPADDED = 1, 2, 4  # bits of the selection entry points' `causal` argument
SEL_TOPK, SEL_TOPP, SEL_MINS, SEL_MINS_TILED = 0, 1, 2, 3
_MODES = {"topk": SEL_TOPK, "topp": SEL_TOPP, "mins": SEL_MINS, "mins_tiled": SEL_MINS_TILED}


class VecattnError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


class TDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("H", ctypes.c_int64), ("N", ctypes.c_int64),
                ("D", ctypes.c_int64), ("sB", ctypes.c_int64), ("sH", ctypes.c_int64),
                ("sN", ctypes.c_int64)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libvecattn.so from the package directory (raises if not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(or python paper_2603_29494_amd/build.py) first")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f64, f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double,
                            ctypes.c_float)
    D = ctypes.POINTER(TDesc)
    lib.vecattn_version.restype = i32
    lib.vecattn_status_string.argtypes = [ctypes.c_int]
    lib.vecattn_status_string.restype = ctypes.c_char_p
    lib.vecattn_pool.argtypes = [P, D, i32, P, D, P]
    lib.vecattn_select_max_count.argtypes = [i64, i32, i32, i32, f64, ctypes.POINTER(i64)]
    lib.vecattn_select_workspace_size.argtypes = [D, D, i32, i32, i32, i64,
                                                  ctypes.POINTER(ctypes.c_size_t)]
    lib.vecattn_select.argtypes = [P, D, P, D, i32, i32, i32, f64, P, i64, P, P, P,
                                   ctypes.c_size_t, P]
    lib.vecattn_select_mins_tiled.argtypes = [P, D, P, D, i32, i32, f64, i32, i32, P, i64, P, P,
                                              P, ctypes.c_size_t, P]
    lib.vecattn_sparse_attn.argtypes = [P, D, P, D, P, D, P, i64, P, i32, i32, f32, P, D, P, P]
    lib.vecattn_sparse_attn_ordered.argtypes = [P, D, P, D, P, D, P, i64, P, P, i32, i32, f32, P, D,
                                                P, P]
    lib.vecattn_attn_order.argtypes = [P, i64, P, i64, i32, i64, i32, P, P]
    lib.vecattn_check_lists.argtypes = [P, i64, i64, P, i64, P, P]
    lib.vecattn_plan_filter_ratios.argtypes = [i32, i32, P, P, f64, i32, P, ctypes.POINTER(f64)]
    lib.vecattn_select_per_head.argtypes = [P, D, P, D, i32, i32, i32, P, i32, i32, P, i64, P, P,
                                            P, ctypes.c_size_t, P]
    lib.vecattn_select_varlen.argtypes = [P, D, P, D, P, i32, i32, i32, i32, f64, P, i64, P, P, P,
                                          ctypes.c_size_t, P]
    lib.vecattn_sparse_attn_varlen.argtypes = [P, D, P, D, P, D, P, i32, P, i64, P, i32, i32, f32,
                                               P, D, P, P]
    lib.vecattn_select_workspace_bytes.argtypes = [D, D, i32, i32, i64]
    lib.vecattn_select_workspace_bytes.restype = ctypes.c_size_t
    lib.vecattn_head_sparsity.argtypes = [P, i64, i64, i64, i32, i32, P, P]
    lib.vecattn_recall.argtypes = [P, D, P, D, P, i64, P, i32, i32, f32, P, P]
    lib.vecattn_select_noalloc.argtypes = [P, D, P, D, i32, i32, i32, f64, P, i64, P, P, P]
    for name in ("vecattn_pool", "vecattn_select_max_count", "vecattn_select_workspace_size",
                 "vecattn_select", "vecattn_select_mins_tiled", "vecattn_sparse_attn",
                 "vecattn_plan_filter_ratios", "vecattn_select_per_head",
                 "vecattn_select_varlen", "vecattn_sparse_attn_varlen", "vecattn_check_lists",
                 "vecattn_head_sparsity", "vecattn_recall", "vecattn_select_noalloc",
                 "vecattn_sparse_attn_ordered", "vecattn_attn_order"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    try:
        return load().vecattn_status_string(int(status)).decode()
    except ImportError:
        return "unknown"


def _check(status: int, what: str):
    if status != OK:
        raise VecattnError(status, what)


def desc(t: torch.Tensor) -> TDesc:
    if t.dim() != 4:
        raise ValueError("expected a [B, H, N, D] tensor")
    B, H, N, Dd = t.shape
    sB, sH, sN, sD = t.stride()
    if sD != 1:
        raise ValueError("the D dimension must be contiguous")
    return TDesc(B, H, N, Dd, sB, sH, sN)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _bf16_cuda(t: torch.Tensor, name: str):
    if not t.is_cuda or t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be a bfloat16 CUDA tensor")


def mode_id(mode) -> int:
    return _MODES[mode] if isinstance(mode, str) else int(mode)


def _per_head(param) -> bool:
    import numpy as np
    return np.ndim(param) > 0


def _flags(causal: bool, keep_diag: bool, unpadded: bool = False) -> int:
    return (CAUSAL if causal else 0) | (KEEP_DIAG if keep_diag else 0) | (UNPADDED if unpadded else 0)


def max_count(N: int, block: int, causal: bool, mode, param, keep_diag: bool = False) -> int:
    """Largest count a block can select (a per-head parameter list: over its heads)."""
    if _per_head(param):
        return max(max_count(N, block, causal, mode, float(x), keep_diag) for x in param)
    out = ctypes.c_int64(0)
    _check(load().vecattn_select_max_count(int(N), int(block), _flags(causal, keep_diag),
                                           mode_id(mode),
                                           float(param), ctypes.byref(out)), "select_max_count")
    return int(out.value)


def pool(q: torch.Tensor, block: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Pooled queries, Eq. 2: bf16 [B, H, ceil(N/block), D]."""
    _bf16_cuda(q, "q")
    B, H, N, Dd = q.shape
    Np = (N + block - 1) // block
    if out is None:
        out = torch.empty((B, H, Np, Dd), dtype=torch.bfloat16, device=q.device)
    qd, od = desc(q), desc(out)
    _check(load().vecattn_pool(_ptr(q), ctypes.byref(qd), int(block), _ptr(out), ctypes.byref(od),
                               _stream(q)), "pool")
    return out


def workspace_bytes(q: torch.Tensor, k: torch.Tensor, block: int, causal: bool, mode,
                    cap: int) -> int:
    n = ctypes.c_size_t(0)
    qd, kd = desc(q), desc(k)
    _check(load().vecattn_select_workspace_size(ctypes.byref(qd), ctypes.byref(kd), int(block),
                                                int(bool(causal)), mode_id(mode), int(cap),
                                                ctypes.byref(n)), "select_workspace_size")
    return int(n.value)


def select(q: torch.Tensor, k: torch.Tensor, block: int, mode, param: float,
           causal: bool = False, cap: Optional[int] = None,
           idx: Optional[torch.Tensor] = None, counts: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None,
           n_clamped: Optional[torch.Tensor] = None, tile: Optional[int] = None,
           group_tiles: Optional[int] = None,
           keep_diag: bool = False, unpadded: bool = False) -> Tuple[torch.Tensor, torch.Tensor]:
    """Per-block key-index lists (I, C) of Algorithm 1 for topK / topP / minS (Eq. 3)
    selection, or minS with Algorithm 1's cross-tile running maximum ("mins_tiled":
    ``tile`` = B_K and ``group_tiles`` = G_K, both 16 when not given).  ``param``
    may be one value per query head (a sequence of Hq values, e.g. from
    plan_filter_ratios).  ``keep_diag``: every block also keeps the keys of its own
    rows (cap must then cover max_count(..., keep_diag=True)).  ``unpadded``: list
    entries past a block's count are left unwritten instead of -1."""
    _bf16_cuda(q, "q")
    _bf16_cuda(k, "k")
    B, Hq, N, Dd = q.shape
    Np = (N + block - 1) // block
    if cap is None:
        cap = max_count(N, block, causal, mode, param, keep_diag)
    flags = _flags(causal, keep_diag, unpadded)
    dev = q.device
    if idx is None:
        idx = torch.empty((B, Hq, Np, cap), dtype=torch.int32, device=dev)
    if counts is None:
        counts = torch.empty((B, Hq, Np), dtype=torch.int32, device=dev)
    if idx.shape != (B, Hq, Np, cap) or not idx.is_contiguous() or idx.dtype != torch.int32:
        raise ValueError("idx must be contiguous int32 [B, Hq, N_p, cap]")
    if counts.shape != (B, Hq, Np) or not counts.is_contiguous() or counts.dtype != torch.int32:
        raise ValueError("counts must be contiguous int32 [B, Hq, N_p]")
    need = workspace_bytes(q, k, block, causal, mode, cap)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    qd, kd = desc(q), desc(k)
    nws = 0 if workspace is None else workspace.numel()
    if _per_head(param):
        import numpy as np
        hp = np.ascontiguousarray(np.asarray(param, dtype=np.float64).reshape(-1))
        if hp.size != Hq:
            raise ValueError("a per-head parameter list needs one value per query head")
        _check(load().vecattn_select_per_head(
            _ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), int(block), flags,
            mode_id(mode), hp.ctypes.data_as(ctypes.c_void_p), 16 if tile is None else int(tile),
            16 if group_tiles is None else int(group_tiles), _ptr(idx), int(cap), _ptr(counts),
            _ptr(n_clamped), _ptr(workspace), nws, _stream(q)), "select_per_head")
        return idx, counts
    if mode_id(mode) == SEL_MINS_TILED:
        _check(load().vecattn_select_mins_tiled(
            _ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), int(block), flags,
            float(param), 16 if tile is None else int(tile),
            16 if group_tiles is None else int(group_tiles), _ptr(idx), int(cap), _ptr(counts),
            _ptr(n_clamped), _ptr(workspace), nws, _stream(q)), "select_mins_tiled")
        return idx, counts
    if tile is not None or group_tiles is not None:
        raise ValueError("tile / group_tiles apply to mode 'mins_tiled' only")
    _check(load().vecattn_select(_ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), int(block),
                                 flags, mode_id(mode), float(param), _ptr(idx),
                                 int(cap), _ptr(counts), _ptr(n_clamped), _ptr(workspace), nws,
                                 _stream(q)),
           "select")
    return idx, counts


STATIC_WORKSPACE_BYTES = 64 << 20


def select_noalloc(q: torch.Tensor, k: torch.Tensor, block: int, mode, param: float,
                   causal: bool, cap: int, idx: torch.Tensor, counts: torch.Tensor,
                   n_clamped: Optional[torch.Tensor] = None, keep_diag: bool = False):
    """select() on the library's own workspace (vecattn_select_noalloc): no device
    memory is allocated by this call; the caller provides idx [B, Hq, N_p, cap]
    and counts [B, Hq, N_p] (contiguous int32).  Calls overlapping on one GPU
    race on that workspace."""
    _bf16_cuda(q, "q")
    _bf16_cuda(k, "k")
    B, Hq, N, _ = q.shape
    Np = (N + block - 1) // block
    if idx.shape != (B, Hq, Np, cap) or not idx.is_contiguous() or idx.dtype != torch.int32:
        raise ValueError("idx must be contiguous int32 [B, Hq, N_p, cap]")
    if counts.shape != (B, Hq, Np) or not counts.is_contiguous() or counts.dtype != torch.int32:
        raise ValueError("counts must be contiguous int32 [B, Hq, N_p]")
    qd, kd = desc(q), desc(k)
    _check(load().vecattn_select_noalloc(_ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd),
                                         int(block), _flags(causal, keep_diag), mode_id(mode),
                                         float(param), _ptr(idx), int(cap), _ptr(counts),
                                         _ptr(n_clamped), _stream(q)), "select_noalloc")
    return idx, counts


def sparse_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, idx: torch.Tensor,
                counts: torch.Tensor, block: int, causal: bool = False, scale: float = 0.0,
                out: Optional[torch.Tensor] = None, return_lse: bool = False,
                order: Optional[torch.Tensor] = None):
    """Vector-sparse attention, Eq. 4: O (bf16, like q) and optionally LSE (fp32 [B,Hq,N]).
    ``order`` (int32 [B, Hq, N_p], e.g. from attn_order) sets the order in which
    the blocks of each head are taken (speed only)."""
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _bf16_cuda(t, n)
    if idx.dtype != torch.int32 or counts.dtype != torch.int32 or not idx.is_contiguous() \
            or not counts.is_contiguous():
        raise ValueError("idx and counts must be contiguous int32")
    B, Hq, N, Dd = q.shape
    Np = (N + block - 1) // block
    if idx.dim() != 4 or tuple(idx.shape[:3]) != (B, Hq, Np) or tuple(counts.shape) != (B, Hq, Np):
        raise ValueError("idx must be [B, Hq, N_p, cap] and counts [B, Hq, N_p]")
    if order is not None and (order.dtype != torch.int32 or not order.is_contiguous()
                              or tuple(order.shape) != (B, Hq, Np)):
        raise ValueError("order must be a contiguous int32 [B, Hq, N_p] tensor")
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    lse = torch.empty((B, Hq, N), dtype=torch.float32, device=q.device) if return_lse else None
    qd, kd, vd, od = desc(q), desc(k), desc(v), desc(out)
    if order is None:
        rc = load().vecattn_sparse_attn(_ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd),
                                        _ptr(v), ctypes.byref(vd), _ptr(idx), int(idx.shape[-1]),
                                        _ptr(counts), int(block), int(bool(causal)), float(scale),
                                        _ptr(out), ctypes.byref(od), _ptr(lse), _stream(q))
    else:
        rc = load().vecattn_sparse_attn_ordered(
            _ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), _ptr(v), ctypes.byref(vd),
            _ptr(idx), int(idx.shape[-1]), _ptr(counts), _ptr(order), int(block),
            int(bool(causal)), float(scale), _ptr(out), ctypes.byref(od), _ptr(lse), _stream(q))
    _check(rc, "sparse_attn")
    return (out, lse) if return_lse else out


def attn_order(idx: torch.Tensor, counts: torch.Tensor, n_keys: int, block: int,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Block order for sparse_attn (int32 [B, Hq, N_p]): per head, count
    descending, then a sampled mean key, then block index."""
    if idx.dtype != torch.int32 or counts.dtype != torch.int32 or not idx.is_cuda \
            or not counts.is_cuda or not idx.is_contiguous() or not counts.is_contiguous():
        raise ValueError("idx and counts must be contiguous int32 CUDA tensors")
    if idx.dim() != 4 or counts.dim() != 3 or tuple(idx.shape[:3]) != tuple(counts.shape):
        raise ValueError("idx must be [B, Hq, N_p, cap] and counts [B, Hq, N_p]")
    B, Hq, Np = counts.shape
    if Np != (int(n_keys) + int(block) - 1) // int(block):
        raise ValueError("counts hold N_p = ceil(n_keys / block) blocks per head")
    if out is None:
        out = torch.empty((B, Hq, Np), dtype=torch.int32, device=idx.device)
    elif out.dtype != torch.int32 or not out.is_contiguous() or tuple(out.shape) != (B, Hq, Np):
        raise ValueError("out must be a contiguous int32 [B, Hq, N_p] tensor")
    _check(load().vecattn_attn_order(_ptr(idx), int(idx.shape[-1]), _ptr(counts), int(B), int(Hq),
                                     int(n_keys), int(block), _ptr(out), _stream(idx)),
           "attn_order")
    return out


def check_lists(idx: torch.Tensor, counts: torch.Tensor, n_keys: int) -> int:
    """Number of rows of (idx [..., cap], counts [...]) that break sparse_attn's
    input contract (count outside [0, cap], a listed key outside [0, n_keys), or a
    list not strictly ascending); 0 for any output of select.  Synchronises."""
    if idx.dtype != torch.int32 or counts.dtype != torch.int32 or not idx.is_cuda \
            or not counts.is_cuda or not idx.is_contiguous() or not counts.is_contiguous():
        raise ValueError("idx and counts must be contiguous int32 CUDA tensors")
    if idx.dim() < 1 or tuple(idx.shape[:-1]) != tuple(counts.shape):
        raise ValueError("idx must be [..., cap] with counts of shape [...]")
    n_bad = torch.empty(1, dtype=torch.int32, device=idx.device)
    _check(load().vecattn_check_lists(_ptr(idx), int(counts.numel()), int(idx.shape[-1]),
                                      _ptr(counts), int(n_keys), _ptr(n_bad), _stream(idx)),
           "check_lists")
    return int(n_bad.item())


def plan_filter_ratios(sparsity, perf, target: float, grid: int = 1000):
    """Per-head filter ratios by Eq. 5's dynamic programme (host computation).

    ``sparsity`` and ``perf`` are [heads, candidates] tables sampled offline
    (sparsity in [0, 1], larger perf is better).  Returns (choice, best): the
    chosen candidate per head (int32 [heads]) reaching mean sparsity >= target
    with the largest summed perf, and that sum.  Raises VecattnError
    (capacity) when no choice reaches the target."""
    import numpy as np
    sp = np.ascontiguousarray(sparsity, dtype=np.float64)
    pf = np.ascontiguousarray(perf, dtype=np.float64)
    if sp.ndim != 2 or sp.shape != pf.shape:
        raise ValueError("sparsity and perf must be [heads, candidates] tables of one shape")
    choice = np.empty(sp.shape[0], dtype=np.int32)
    best = ctypes.c_double(0.0)
    _check(load().vecattn_plan_filter_ratios(int(sp.shape[0]), int(sp.shape[1]),
                                             sp.ctypes.data_as(ctypes.c_void_p),
                                             pf.ctypes.data_as(ctypes.c_void_p), float(target),
                                             int(grid), choice.ctypes.data_as(ctypes.c_void_p),
                                             ctypes.byref(best)), "plan_filter_ratios")
    return choice, float(best.value)


def head_sparsity_of(counts: torch.Tensor, N: int, block: int, causal: bool = False,
                     out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Eq. 5's sp_h of one selection: float64 [Hq] on the device, from its
    counts [B, Hq, N_p] (vecattn_head_sparsity)."""
    if counts.dtype != torch.int32 or not counts.is_cuda or not counts.is_contiguous() \
            or counts.dim() != 3:
        raise ValueError("counts must be a contiguous int32 CUDA tensor [B, Hq, N_p]")
    B, Hq, _ = counts.shape
    if out is None:
        out = torch.empty(Hq, dtype=torch.float64, device=counts.device)
    _check(load().vecattn_head_sparsity(_ptr(counts), int(B), int(Hq), int(N), int(block),
                                        int(bool(causal)), _ptr(out), _stream(counts)),
           "head_sparsity")
    return out


def head_sparsity(q: torch.Tensor, k: torch.Tensor, block: int, mode, params, causal: bool = False,
                  cap: Optional[int] = None, **tiling) -> "torch.Tensor":
    """Sparsity per query head for each candidate parameter (an sp_h table for
    plan_filter_ratios): one selection per parameter, each reduced to its
    per-head sparsity by vecattn_head_sparsity.  Returns float64 [Hq,
    len(params)] on the host.  Extra keyword arguments (tile, group_tiles) go
    to select."""
    B, Hq, N, _ = q.shape
    table = torch.empty((len(params), Hq), dtype=torch.float64, device=q.device)
    ws = None
    for c, prm in enumerate(params):
        cp = max_count(N, block, causal, mode, prm) if cap is None else cap
        need = workspace_bytes(q, k, block, causal, mode, cp)
        if ws is None or ws.numel() < need:
            ws = torch.empty(need, dtype=torch.uint8, device=q.device)
        _, cnt = select(q, k, block, mode, prm, causal, cap=cp, workspace=ws, **tiling)
        head_sparsity_of(cnt, N, block, causal, out=table[c])
    return table.cpu().t().contiguous()


def recall(q: torch.Tensor, k: torch.Tensor, idx: torch.Tensor, counts: torch.Tensor, block: int,
           causal: bool = False, scale: float = 0.0) -> torch.Tensor:
    """Attention mass each query row's block list keeps (the recall of the
    pattern study, vecattn_recall): fp32 [B, Hq, N]."""
    _bf16_cuda(q, "q")
    _bf16_cuda(k, "k")
    if idx.dtype != torch.int32 or counts.dtype != torch.int32 or not idx.is_contiguous() \
            or not counts.is_contiguous():
        raise ValueError("idx and counts must be contiguous int32")
    B, Hq, N, _ = q.shape
    kept = torch.empty((B, Hq, N), dtype=torch.float32, device=q.device)
    qd, kd = desc(q), desc(k)
    _check(load().vecattn_recall(_ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), _ptr(idx),
                                 int(idx.shape[-1]), _ptr(counts), int(block), int(bool(causal)),
                                 float(scale), _ptr(kept), _stream(q)), "recall")
    return kept


def varlen_blocks(cu_seqlens, block: int):
    """Query blocks of each packed sequence and their offsets: (per-sequence
    N_p, first block of each sequence, total blocks)."""
    import numpy as np
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    nb = (np.diff(cu) + block - 1) // block
    first = np.concatenate([[0], np.cumsum(nb)[:-1]]) if len(nb) else np.zeros(0, np.int64)
    return nb, first, int(nb.sum())


def select_varlen(q: torch.Tensor, k: torch.Tensor, cu_seqlens, block: int, mode, param: float,
                  causal: bool = False, cap: Optional[int] = None,
                  workspace: Optional[torch.Tensor] = None, n_clamped: Optional[torch.Tensor] = None,
                  keep_diag: bool = False) -> Tuple[torch.Tensor, torch.Tensor]:
    """Selection over packed variable-length sequences (q, k: [1, H, total, D];
    cu_seqlens: nseq + 1 row offsets).  Returns flat (idx, counts): the
    per-sequence [Hq, N_p(s), cap] and [Hq, N_p(s)] arrays laid end to end."""
    import numpy as np
    _bf16_cuda(q, "q")
    _bf16_cuda(k, "k")
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int64))
    Hq = q.shape[1]
    lens = np.diff(cu)
    longest = int(lens.max()) if lens.size else 0
    if cap is None:
        cap = max(max_count(int(n), block, causal, mode, param, keep_diag) for n in lens if n > 0)
    _, _, total_blocks = varlen_blocks(cu, block)
    idx = torch.empty(total_blocks * Hq * cap, dtype=torch.int32, device=q.device)
    counts = torch.empty(total_blocks * Hq, dtype=torch.int32, device=q.device)
    if workspace is None:
        qv = q[:, :, :max(longest, 1)]
        kv = k[:, :, :max(longest, 1)]
        workspace = torch.empty(workspace_bytes(qv, kv, block, causal, mode, cap), dtype=torch.uint8,
                                device=q.device)
    qd, kd = desc(q), desc(k)
    _check(load().vecattn_select_varlen(
        _ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), cu.ctypes.data_as(ctypes.c_void_p),
        int(len(cu) - 1), int(block), _flags(causal, keep_diag), mode_id(mode), float(param),
        _ptr(idx), int(cap), _ptr(counts), _ptr(n_clamped), _ptr(workspace), workspace.numel(),
        _stream(q)), "select_varlen")
    return idx, counts


def sparse_attn_varlen(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, cu_seqlens,
                       idx: torch.Tensor, counts: torch.Tensor, cap: int, block: int,
                       causal: bool = False, scale: float = 0.0,
                       out: Optional[torch.Tensor] = None, return_lse: bool = False):
    """Vector-sparse attention over packed variable-length sequences, with the
    lists of select_varlen.  Returns out (and the flat per-sequence
    [Hq, n_s] LSE arrays laid end to end when return_lse)."""
    import numpy as np
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _bf16_cuda(t, n)
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int64))
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    lse = (torch.empty(q.shape[1] * q.shape[2], dtype=torch.float32, device=q.device)
           if return_lse else None)
    qd, kd, vd, od = desc(q), desc(k), desc(v), desc(out)
    _check(load().vecattn_sparse_attn_varlen(
        _ptr(q), ctypes.byref(qd), _ptr(k), ctypes.byref(kd), _ptr(v), ctypes.byref(vd),
        cu.ctypes.data_as(ctypes.c_void_p), int(len(cu) - 1), _ptr(idx), int(cap), _ptr(counts),
        int(block), int(bool(causal)), float(scale), _ptr(out), ctypes.byref(od), _ptr(lse),
        _stream(q)), "sparse_attn_varlen")
    return (out, lse) if return_lse else out
