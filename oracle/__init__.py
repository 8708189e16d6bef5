"""CPU oracle for vertical-vector sparse attention (VecAttention, arXiv 2603.29494).

TEST INFRASTRUCTURE ONLY.  Plain fp64 C++ (``vecattn_ref.cpp``) behind ctypes,
used by ``tests/``, the smoke check and the CPU-baseline leg of the benchmark to
check the GPU library.  The product path never imports this package; this
package never imports the product.  Inputs are bf16 bit patterns held in
``numpy.uint16`` arrays, laid out contiguous ``[B, H, N, D]``.

Functions and the passages they follow:

* :func:`pool`            -- Eq. 2 (query pooling), Sec. 3.1.1.
* :func:`pooled_scores`   -- the estimated map's scores Q_p K^T / sqrt(D), Sec. 3.1.1.
* :func:`select`          -- row-wise topK / topP (Sec. 3.1.2) and minS (Eq. 3).
* :func:`mins_progressive`-- Eq. 3 as Algorithm 1 applies it (running max per K-group).
* :func:`select_mins_tiled` -- Algorithm 1's selection (cross-tile minS, Sec. 3.1.3) per block.
* :func:`sparse_attn`     -- Eq. 4 (materialised softmax over the selected keys).
* :func:`sparse_attn_online` -- Algorithm 2's online recurrence (second route to Eq. 4).
* :func:`dense_attn`      -- Eq. 1, textbook dense attention.
* :func:`plan_filter_ratios` -- Eq. 5's optimum by exhaustive search (tiny tables only).
* :func:`kept_mass`       -- Sec. 2.2's recall: the exact attention mass a pattern keeps.
* :func:`head_sparsity`   -- Eq. 5's sp_h: the share of a head's eligible keys left out.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vecattn_ref.cpp")
_LIB_PATH = os.path.join(_HERE, "libvecattn_ref.so")

TOPK, TOPP, MINS, MINS_TILED = 0, 1, 2, 3

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (OpenMP, -O2, strict IEEE double)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", _SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64, i32, f64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    lib.ora_bf16_round.argtypes = [P, i64, P]
    lib.ora_pool.argtypes = [P, i64, i64, i64, i64, i32, P, i32]
    lib.ora_pooled_scores.argtypes = [P, P, i64, i64, i64, i64, i64, i32, i32, i64, i64, i64, P, P]
    lib.ora_topk_count.argtypes = [f64, i64]
    lib.ora_topk_count.restype = i64
    lib.ora_select.argtypes = [P, P, i64, i64, i64, i64, i64, i32, i32, i32, f64, i64,
                               P, P, P, P, i64, i32, i32]
    lib.ora_mins_progressive_row.argtypes = [P, i64, f64, i64, i64, P, P]
    lib.ora_select_mins_tiled.argtypes = [P, P, i64, i64, i64, i64, i64, i32, i32, f64, i64, i64,
                                          i64, P, P, P, P, i64, i32, i32]
    lib.ora_sparse_attn.argtypes = [P, P, P, i64, i64, i64, i64, i64, i32, i32, f64,
                                    P, i64, P, P, P, P, i64, i32, i32]
    lib.ora_dense_attn.argtypes = [P, P, P, i64, i64, i64, i64, i64, i32, f64, P, P, i32]
    lib.ora_sparse_attn_online.argtypes = [P, P, P, i64, i64, i64, i64, i64, i32, i32, f64,
                                           P, i64, P, i32, P, P, i32]
    lib.ora_pooled_scores_rows.argtypes = [P, P, i64, i64, i64, i64, i64, i32, i32, P, i64, P,
                                           i32]
    lib.ora_kept_mass.argtypes = [P, P, i64, i64, i64, i64, i64, i32, i32, f64, P, i64, P, P, P,
                                  i64, i32]
    for name in ("ora_bf16_round", "ora_pool", "ora_pooled_scores", "ora_select",
                 "ora_mins_progressive_row", "ora_select_mins_tiled", "ora_sparse_attn", "ora_dense_attn",
                 "ora_sparse_attn_online", "ora_kept_mass", "ora_pooled_scores_rows"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _bits(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("oracle inputs are bf16 bit patterns (numpy.uint16)")
    return a


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round doubles to bf16 (nearest, ties to even) in one step; returns bits."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _check(_load().ora_bf16_round(_ptr(x), x.size, _ptr(out)), "bf16_round")
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def num_blocks(N: int, block: int) -> int:
    return (N + block - 1) // block


def eligible_keys(N: int, block: int, i: int, causal: bool) -> int:
    return min(N, (i + 1) * block) if causal else N


def topk_count(ratio: float, L: int) -> int:
    return int(_load().ora_topk_count(float(ratio), int(L)))


def pool(q: np.ndarray, block: int, nthreads: int = 0) -> np.ndarray:
    q = _bits(q)
    B, H, N, D = q.shape
    out = np.empty((B, H, num_blocks(N, block), D), dtype=np.uint16)
    _check(_load().ora_pool(_ptr(q), B, H, N, D, block, _ptr(out), nthreads), "pool")
    return out


def pooled_scores(q: np.ndarray, k: np.ndarray, block: int, causal: bool, b: int, h: int,
                  i: int) -> np.ndarray:
    q, k = _bits(q), _bits(k)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    out = np.empty(N, dtype=np.float64)
    L = ctypes.c_int64(0)
    _check(_load().ora_pooled_scores(_ptr(q), _ptr(k), B, Hq, Hkv, N, D, block, int(causal),
                                     b, h, i, _ptr(out), ctypes.byref(L)), "pooled_scores")
    return out[:L.value].copy()


def pooled_scores_rows(q: np.ndarray, k: np.ndarray, block: int, causal: bool, rows,
                       nthreads: int = 0):
    """pooled_scores of several blocks (flat ids (b * Hq + h) * Np + i), computed
    in parallel: a list of 1-D arrays, one per listed block (L_i values each)."""
    q, k = _bits(q), _bits(k)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((rows_arr.size, N), dtype=np.float64)
    _check(_load().ora_pooled_scores_rows(_ptr(q), _ptr(k), B, Hq, Hkv, N, D, block, int(causal),
                                          _ptr(rows_arr), rows_arr.size, _ptr(out), nthreads),
           "pooled_scores_rows")
    Np = num_blocks(N, block)
    return [out[t, :eligible_keys(N, block, int(w) % Np, causal)] for t, w in enumerate(rows_arr)]


def with_diagonal(idx: np.ndarray, counts: np.ndarray, N: int, block: int, cap: int,
                  rows: Optional[Sequence[int]] = None, compact: bool = False):
    """The keep-the-diagonal variant: each block's list united with the keys of
    its own rows [i P, min(N, (i+1) P)), ascending, -1 padded to cap."""
    Np = num_blocks(N, block)
    flat = idx.reshape(-1, idx.shape[-1])
    cnt = counts.reshape(-1)
    out = np.full((flat.shape[0], cap), -1, dtype=np.int32)
    ocnt = np.zeros(flat.shape[0], dtype=np.int32)
    # t: output row; w: its flat block id (compact outputs hold the listed rows in order)
    todo = range(flat.shape[0]) if rows is None else (range(len(rows)) if compact else list(rows))
    for t in todo:
        w = int(rows[t]) if compact else int(t)
        i = w % Np
        keys = sorted(set(flat[t, :cnt[t]].tolist()) | set(range(i * block, min(N, (i + 1) * block))))
        if len(keys) > cap:
            raise ValueError("capacity too small for the kept diagonal")
        out[t, :len(keys)] = keys
        ocnt[t] = len(keys)
    return out.reshape(idx.shape[:-1] + (cap,)), ocnt.reshape(counts.shape)


def select(q: np.ndarray, k: np.ndarray, block: int, mode: int, param: float, causal: bool,
           cap: int, rows: Optional[Sequence[int]] = None,
           nthreads: int = 0, compact: bool = False,
           keep_diag: bool = False) -> Tuple[np.ndarray, np.ndarray, int]:
    """Selected key lists (ascending, -1 padded), counts and number of clamped rows.

    ``rows`` lists flat block ids w = (b * Hq + h) * Np + i to compute; other rows
    of the outputs are left as -1 / 0.  ``compact`` (with ``rows``): outputs of
    shape [len(rows), cap] and [len(rows)], in the order of ``rows``.
    ``keep_diag``: each list united with the keys of its block's own rows
    (:func:`with_diagonal`; no clamping then: cap must cover every union).
    """
    q, k = _bits(q), _bits(k)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    Np = num_blocks(N, block)
    if compact:
        if rows is None:
            raise ValueError("compact output needs rows")
        idx = np.full((len(rows), cap), -1, dtype=np.int32)
        counts = np.zeros(len(rows), dtype=np.int32)
    else:
        idx = np.full((B, Hq, Np, cap), -1, dtype=np.int32)
        counts = np.zeros((B, Hq, Np), dtype=np.int32)
    ncl = ctypes.c_int64(0)
    rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    rc = _load().ora_select(_ptr(q), _ptr(k), B, Hq, Hkv, N, D, block, int(causal), int(mode),
                            float(param), int(cap), _ptr(idx), _ptr(counts), ctypes.byref(ncl),
                            _ptr(rows_arr), 0 if rows_arr is None else rows_arr.size,
                            int(bool(compact)), nthreads)
    if rc == 3:
        raise ValueError("capacity too small for topK")
    _check(rc, "select")
    if keep_diag:
        if ncl.value:
            raise ValueError("capacity too small: a block was clamped")
        idx, counts = with_diagonal(idx, counts, N, block, cap, rows, compact)
    return idx, counts, int(ncl.value)


def select_mins_tiled(q: np.ndarray, k: np.ndarray, block: int, alpha: float, causal: bool,
                      cap: int, bk: int = 16, gk: int = 16, rows: Optional[Sequence[int]] = None,
                      nthreads: int = 0,
                      compact: bool = False) -> Tuple[np.ndarray, np.ndarray, int]:
    """Algorithm 1's selection: per block, the eligible keys kept by the cross-tile
    minS rule (groups of gk tiles of bk keys, running maximum within a group;
    Sec. 3.1.3), ascending; a block keeping more than cap keys keeps its first
    cap and is counted.  Outputs as :func:`select`."""
    q, k = _bits(q), _bits(k)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    Np = num_blocks(N, block)
    if compact:
        if rows is None:
            raise ValueError("compact output needs rows")
        idx = np.full((len(rows), cap), -1, dtype=np.int32)
        counts = np.zeros(len(rows), dtype=np.int32)
    else:
        idx = np.full((B, Hq, Np, cap), -1, dtype=np.int32)
        counts = np.zeros((B, Hq, Np), dtype=np.int32)
    ncl = ctypes.c_int64(0)
    rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    _check(_load().ora_select_mins_tiled(_ptr(q), _ptr(k), B, Hq, Hkv, N, D, block, int(causal),
                                         float(alpha), int(bk), int(gk), int(cap), _ptr(idx),
                                         _ptr(counts), ctypes.byref(ncl), _ptr(rows_arr),
                                         0 if rows_arr is None else rows_arr.size,
                                         int(bool(compact)), nthreads), "select_mins_tiled")
    return idx, counts, int(ncl.value)


def mins_progressive(scores: np.ndarray, alpha: float, bk: int, gk: int) -> np.ndarray:
    s = np.ascontiguousarray(scores, dtype=np.float64)
    out = np.empty(max(1, s.size), dtype=np.int32)
    n = ctypes.c_int64(0)
    _check(_load().ora_mins_progressive_row(_ptr(s), s.size, float(alpha), bk, gk, _ptr(out),
                                            ctypes.byref(n)), "mins_progressive")
    return out[:n.value].copy()


def sparse_attn(q: np.ndarray, k: np.ndarray, v: np.ndarray, idx: np.ndarray, counts: np.ndarray,
                block: int, causal: bool, scale: float = 0.0,
                blocks: Optional[Sequence[int]] = None,
                nthreads: int = 0, compact: bool = False) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 4 in fp64.  Returns (O [B,Hq,N,D] f64, LSE [B,Hq,N] f64); rows of
    blocks not listed in ``blocks`` are left NaN.  ``compact`` (with
    ``blocks``): idx [len(blocks), cap] and counts [len(blocks)] hold the listed
    blocks' lists in order, and the outputs are O [len(blocks), block, D] and
    LSE [len(blocks), block] (rows past N in a ragged last block stay NaN)."""
    q, k, v = _bits(q), _bits(k), _bits(v)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    cap = idx.shape[-1]
    if compact:
        if blocks is None:
            raise ValueError("compact layout needs blocks")
        o = np.full((len(blocks), block, D), np.nan, dtype=np.float64)
        lse = np.full((len(blocks), block), np.nan, dtype=np.float64)
    else:
        o = np.full((B, Hq, N, D), np.nan, dtype=np.float64)
        lse = np.full((B, Hq, N), np.nan, dtype=np.float64)
    blk = None if blocks is None else np.ascontiguousarray(blocks, dtype=np.int64)
    _check(_load().ora_sparse_attn(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, D, block,
                                   int(causal), float(scale), _ptr(idx), cap, _ptr(counts),
                                   _ptr(o), _ptr(lse), _ptr(blk),
                                   0 if blk is None else blk.size, int(bool(compact)), nthreads),
           "sparse_attn")
    return o, lse


def sparse_attn_online(q, k, v, idx, counts, block, causal, bk, scale=0.0, nthreads=0):
    q, k, v = _bits(q), _bits(k), _bits(v)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    o = np.zeros((B, Hq, N, D), dtype=np.float64)
    lse = np.zeros((B, Hq, N), dtype=np.float64)
    _check(_load().ora_sparse_attn_online(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, D, block,
                                          int(causal), float(scale), _ptr(idx), idx.shape[-1],
                                          _ptr(counts), int(bk), _ptr(o), _ptr(lse), nthreads),
           "sparse_attn_online")
    return o, lse


def dense_attn(q, k, v, causal, scale=0.0, nthreads=0):
    q, k, v = _bits(q), _bits(k), _bits(v)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    o = np.zeros((B, Hq, N, D), dtype=np.float64)
    lse = np.zeros((B, Hq, N), dtype=np.float64)
    _check(_load().ora_dense_attn(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, D, int(causal),
                                  float(scale), _ptr(o), _ptr(lse), nthreads), "dense_attn")
    return o, lse


def kept_mass(q, k, idx, counts, block, causal, scale=0.0, blocks=None, nthreads=0):
    """Sec. 2.2's recall of the lists' pattern, per query row: the share of the
    row's exact attention distribution (softmax over the keys it sees) that
    falls on its block's listed keys.  Returns [B, Hq, N] f64 (NaN for rows of
    blocks not in ``blocks``)."""
    q, k = _bits(q), _bits(k)
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    kept = np.full((B, Hq, N), np.nan, dtype=np.float64)
    blk = None if blocks is None else np.ascontiguousarray(blocks, dtype=np.int64)
    _check(_load().ora_kept_mass(_ptr(q), _ptr(k), B, Hq, Hkv, N, D, block, int(causal),
                                 float(scale), _ptr(idx), idx.shape[-1], _ptr(counts), _ptr(kept),
                                 _ptr(blk), 0 if blk is None else blk.size, nthreads),
           "kept_mass")
    return kept


def head_sparsity(counts, N: int, block: int, causal: bool) -> np.ndarray:
    """Eq. 5's sp_h from a selection's counts [B, Hq, N_p]: 1 - (keys kept by the
    head's blocks over the batch) / (B * the blocks' eligible keys), per head."""
    c = np.asarray(counts, dtype=np.int64)
    B, Hq, Np = c.shape
    L = sum(eligible_keys(N, block, i, causal) for i in range(Np))
    return 1.0 - c.sum(axis=(0, 2)).astype(np.float64) / float(B * L)


def plan_filter_ratios(sparsity, perf, target: float):
    """Eq. 5 (Sec. 3.1.2, per-head filter ratios) by its definition: over every
    choice of one candidate per head, the largest summed performance among the
    choices whose mean sparsity is at least ``target``.  Plain exhaustive search
    (candidates ** heads choices), for tiny tables.  Returns (best, optima):
    the optimum (None if no choice reaches the target) and every optimal
    choice."""
    import itertools
    sp = np.asarray(sparsity, dtype=np.float64)
    pf = np.asarray(perf, dtype=np.float64)
    H, C = sp.shape
    best, optima = None, []
    for ch in itertools.product(range(C), repeat=H):
        mean_sp = sum(sp[h, c] for h, c in enumerate(ch)) / H
        if mean_sp < target - 1e-12:
            continue
        val = sum(pf[h, c] for h, c in enumerate(ch))
        if best is None or val > best + 1e-12:
            best, optima = val, [ch]
        elif abs(val - best) <= 1e-12:
            optima.append(ch)
    return best, optima
