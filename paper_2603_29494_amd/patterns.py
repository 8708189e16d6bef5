"""Sparsity-recall statistics of sparse attention patterns (paper Sec. 2.2,
"Statistical Comparison of Different Sparse Patterns").

An analysis tool, not part of the selection / attention path: it takes one
head's dense attention map and, for each pattern, partitions the map into
regions of that pattern's shape, ranks the regions by their mean attention
weight, selects them in that order and records after each step the sparsity
(fraction of the map's entries left out) and the recall (fraction of the
attention mass kept):

  oracle             single entries (the best any mask can do at a sparsity)
  block              P x P tiles
  vertical_vector    P consecutive query rows x 1 key column
  horizontal_vector  1 query row x P consecutive keys
  line               whole key columns and whole diagonals (slash lines),
                     which overlap: a step adds only the entries not yet kept

Causal maps count only the entries on or below the diagonal.  The dense map
is computed with plain torch operations (float32), on whatever device the
inputs are on.
"""
from __future__ import annotations

from typing import Dict, Tuple

import numpy as np
import torch

PATTERNS = ("oracle", "block", "vertical_vector", "horizontal_vector", "line")


def attention_map(q: torch.Tensor, k: torch.Tensor, causal: bool) -> torch.Tensor:
    """softmax(q k^T / sqrt(D)) of one head (q, k: [N, D]), float32, causal
    entries above the diagonal set to 0."""
    q, k = q.float(), k.float()
    s = (q @ k.t()) / float(q.shape[1]) ** 0.5
    if causal:
        n = s.shape[0]
        s = s.masked_fill(torch.ones(n, n, dtype=torch.bool, device=s.device).triu(1), float("-inf"))
    return torch.softmax(s, dim=1)


def _curve_from_regions(mass: torch.Tensor, size: torch.Tensor, total_mass: float,
                        total_size: float) -> Tuple[np.ndarray, np.ndarray]:
    """Disjoint regions: rank by mean weight (mass / size), accumulate."""
    keep = size > 0
    mass, size = mass[keep].double(), size[keep].double()
    order = torch.argsort(mass / size, descending=True, stable=True)
    cm = torch.cumsum(mass[order], 0) / total_mass
    cs = torch.cumsum(size[order], 0) / total_size
    return (np.concatenate([[1.0], (1.0 - cs).cpu().numpy()]),
            np.concatenate([[0.0], cm.cpu().numpy()]))


def _valid(n: int, causal: bool, device) -> torch.Tensor:
    v = torch.ones(n, n, dtype=torch.bool, device=device)
    return v.tril() if causal else v


def _tiles(x: torch.Tensor, rp: int, cp: int) -> torch.Tensor:
    """Sum over rp x cp tiles (the map padded with zeros to whole tiles)."""
    n, m = x.shape
    pr, pc = (-n) % rp, (-m) % cp
    x = torch.nn.functional.pad(x, (0, pc, 0, pr))
    return x.reshape((n + pr) // rp, rp, (m + pc) // cp, cp).sum(dim=(1, 3))


def sparsity_recall(a: torch.Tensor, pattern: str, size: int, causal: bool,
                    max_lines: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """The sparsity-recall curve of one pattern on attention map ``a`` [N, N]
    (region size ``size`` = P for the tiled patterns).  Returns (sparsity,
    recall), starting at (1, 0) and ending at (0, 1) for the disjoint
    patterns.  ``max_lines`` (line pattern) stops after that many lines (0: all)."""
    n = a.shape[0]
    valid = _valid(n, causal, a.device).to(torch.float64)
    a = a.double() * valid
    total_mass = float(a.sum())
    total_size = float(valid.sum())
    if pattern == "oracle":
        return _curve_from_regions(a[valid > 0], torch.ones_like(a[valid > 0]), total_mass,
                                   total_size)
    if pattern in ("block", "vertical_vector", "horizontal_vector"):
        rp, cp = {"block": (size, size), "vertical_vector": (size, 1),
                  "horizontal_vector": (1, size)}[pattern]
        return _curve_from_regions(_tiles(a, rp, cp).reshape(-1), _tiles(valid, rp, cp).reshape(-1),
                                   total_mass, total_size)
    if pattern != "line":
        raise ValueError(f"unknown pattern {pattern}")
    # Lines: key columns j and diagonals d = i - j (slash lines), ranked by
    # their mean weight; each step keeps the line's entries not kept yet.
    col_mass, col_size = a.sum(0), valid.sum(0)
    idx_i = torch.arange(n, device=a.device).view(-1, 1)
    idx_j = torch.arange(n, device=a.device).view(1, -1)
    dg = (idx_i - idx_j + (n - 1)).reshape(-1)                   # 0 .. 2n - 2
    diag_mass = torch.zeros(2 * n - 1, dtype=torch.float64, device=a.device)
    diag_size = torch.zeros_like(diag_mass)
    diag_mass.index_add_(0, dg, a.reshape(-1))
    diag_size.index_add_(0, dg, valid.reshape(-1))
    mass = torch.cat([col_mass, diag_mass])
    sz = torch.cat([col_size, diag_size])
    live = sz > 0
    order = torch.argsort(torch.where(live, mass / sz.clamp(min=1), torch.full_like(mass, -1.0)),
                          descending=True, stable=True)
    order = order[: int(live.sum())]
    if max_lines > 0:
        order = order[:max_lines]
    kept = torch.zeros(n, n, dtype=torch.bool, device=a.device)
    km, ks = 0.0, 0.0
    sp, rc = [1.0], [0.0]
    for t in order.tolist():
        if t < n:
            sel = ~kept[:, t] & (valid[:, t] > 0)
            km += float(a[:, t][sel].sum())
            ks += float(sel.sum())
            kept[:, t] |= sel
        else:
            d = t - n - (n - 1)                                   # i - j
            i = torch.arange(max(0, d), min(n, n + d), device=a.device)
            j = i - d
            sel = ~kept[i, j] & (valid[i, j] > 0)
            km += float(a[i, j][sel].sum())
            ks += float(sel.sum())
            kept[i[sel], j[sel]] = True
        sp.append(1.0 - ks / total_size)
        rc.append(km / total_mass)
    return np.array(sp), np.array(rc)


def recall_at(curve: Tuple[np.ndarray, np.ndarray], sparsity: float) -> float:
    """Recall of a curve at a given sparsity (the largest recall among the
    steps whose sparsity is at least that)."""
    sp, rc = curve
    ok = sp >= sparsity - 1e-12
    return float(rc[ok].max()) if ok.any() else 0.0


def compare(q: torch.Tensor, k: torch.Tensor, size: int, causal: bool,
            sparsities=(0.5, 0.8, 0.9, 0.95), max_lines: int = 0) -> Dict[str, Dict[float, float]]:
    """Recall of every pattern at the given sparsities for one head."""
    a = attention_map(q, k, causal)
    out = {}
    for p in PATTERNS:
        c = sparsity_recall(a, p, size, causal, max_lines=max_lines)
        out[p] = {s: recall_at(c, s) for s in sparsities}
    return out
