"""Parity rule for selected index sets (GPU vs oracle), shared by the GPU tests.

Scores are the oracle's fp64 values of the estimated map (Sec. 3.1.1).  The
GPU computes them from the same bf16 inputs with fp32 accumulation, so sets
may differ only where two keys' scores are within 1e-5 * max|s| of the cut:
  topK: equal counts; every key in the symmetric difference lies within the
        tolerance of the oracle's k-th score.
  minS: every key in the symmetric difference lies within the tolerance of
        rowmax - alpha (rows clamped to cap follow the topK rule);
  cross-tile minS (Algorithm 1): every key in the symmetric difference lies
        within the tolerance of its own threshold, the running maximum of its
        group's tiles up to its tile, minus alpha;
  topP: every key in the symmetric difference lies within the tolerance of
        the oracle's cut score, or the oracle's cumulative mass at the cut is
        within 1e-5 of p (then the counts differ by at most one); the GPU set's
        oracle mass is >= p - 1e-5 unless the row was clamped to cap.
Lists must be strictly ascending, in [0, L_i), and -1 padded.
"""
import numpy as np

import oracle

REL_TOL = 1e-5
MASS_TOL = 1e-5


def check_rows(q, k, block, mode, param, causal, cap, idx_gpu, cnt_gpu, rows, compact=False):
    """Returns the number of rows whose sets differ (all within the rule).

    compact: idx_gpu [len(rows), cap] / cnt_gpu [len(rows)] hold only the
    sampled rows, in the order of ``rows`` (full-size layers)."""
    B, Hq, N, D = q.shape
    Np = (N + block - 1) // block
    if compact:
        idx_o, cnt_o, _ = oracle.select(q, k, block, mode, param, causal, cap, rows=rows,
                                        compact=True)
        pos = {int(w): t for t, w in enumerate(rows)}
    else:
        idx_o, cnt_o, _ = oracle.select(q, k, block, mode, param, causal, cap, rows=rows)
        pos = {int(w): int(w) for w in rows}
    idx_o = idx_o.reshape(-1, cap)
    cnt_o = cnt_o.reshape(-1)
    idx_gpu = idx_gpu.reshape(-1, idx_gpu.shape[-1])
    cnt_gpu = cnt_gpu.reshape(-1)
    mismatched = 0
    for w, s in zip(rows, _scores(q, k, block, causal, rows)):
        w = int(w)
        pw = pos[w]
        L = len(s)
        tol = REL_TOL * np.abs(s).max()
        cg, co = int(cnt_gpu[pw]), int(cnt_o[pw])
        g = idx_gpu[pw, :cg]
        o = idx_o[pw, :co]
        assert 0 <= cg <= idx_gpu.shape[1], (w, cg)
        assert np.all(np.diff(g) > 0), f"row {w}: not strictly ascending"
        assert cg == 0 or (g[0] >= 0 and g[-1] < L), f"row {w}: index out of range"
        assert np.all(idx_gpu[pw, cg:] == -1), f"row {w}: padding"
        diff = np.setxor1d(g, o)
        if mode == oracle.MINS and co < cap:   # minS: keys at or above rowmax - alpha
            if diff.size:
                mismatched += 1
                thr = s.max() - param
                assert np.all(np.abs(s[diff] - thr) <= tol), \
                    f"row {w}: minS differs beyond near-threshold: {np.abs(s[diff] - thr).max()}"
            continue
        if mode == oracle.TOPK or co == cap:   # topK, or a threshold row clamped to cap
            assert cg == co, f"row {w}: count {cg} != {co}"
            if diff.size:
                vk = s[o].min()
                assert np.all(np.abs(s[diff] - vk) <= tol), \
                    f"row {w}: topK differs beyond near-tie: {np.abs(s[diff] - vk).max()}"
                mismatched += 1
        else:
            if diff.size:
                mismatched += 1
                vcut = s[o].min()
                e = np.exp(s - s.max())
                Z = e.sum()
                order = np.lexsort((np.arange(L), -s))
                cum = np.cumsum(e[order]) / Z
                mass_at_cut = cum[co - 1]
                prev = cum[co - 2] if co >= 2 else 0.0
                near_mass = abs(mass_at_cut - param) <= MASS_TOL or abs(prev - param) <= MASS_TOL
                near_score = np.all(np.abs(s[diff] - vcut) <= tol)
                assert near_score or (near_mass and abs(cg - co) <= 1), \
                    f"row {w}: topP differs: counts {cg} vs {co}, gap {np.abs(s[diff] - vcut).max()}"
            if cg < cap:
                e = np.exp(s - s.max())
                assert e[g].sum() / e.sum() >= param - MASS_TOL, f"row {w}: mass below p"
    return mismatched


def check_rows_keep_diag(q, k, block, mode, param, causal, cap, idx_gpu, cnt_gpu, rows,
                         compact=False, tiling=(16, 16)):
    """Parity of lists selected with the block's own rows kept (the keep-diagonal
    variant): the GPU list holds every key of the block's rows, and its
    difference from the oracle's list (the oracle's selection united with those
    keys) lies outside the block's rows, within the near-tie tolerance of the
    oracle's cut (the score of its last kept key; minS: rowmax - alpha;
    cross-tile minS: the key's own running threshold, with ``tiling`` = (B_K,
    G_K)).  Returns the number of rows whose lists differ."""
    B, Hq, N, D = q.shape
    Np = (N + block - 1) // block
    kw = dict(rows=rows, compact=True)
    if mode == oracle.MINS_TILED:
        plain_i, plain_c, ncl = oracle.select_mins_tiled(q, k, block, param, causal, cap,
                                                         tiling[0], tiling[1], **kw)
        assert ncl == 0
        kd_i, kd_c = oracle.with_diagonal(plain_i, plain_c, N, block, cap, rows, compact=True)
    else:
        plain_i, plain_c, _ = oracle.select(q, k, block, mode, param, causal, cap, **kw)
        kd_i, kd_c, _ = oracle.select(q, k, block, mode, param, causal, cap, keep_diag=True, **kw)
    idx_gpu = idx_gpu.reshape(-1, idx_gpu.shape[-1])
    cnt_gpu = cnt_gpu.reshape(-1)
    mismatched = 0
    for t, (w, s) in enumerate(zip(rows, _scores(q, k, block, causal, rows))):
        w = int(w)
        pw = t if compact else w
        i = w % Np
        diag = np.arange(i * block, min(N, (i + 1) * block))
        cg = int(cnt_gpu[pw])
        g = idx_gpu[pw, :cg]
        assert np.all(np.diff(g) > 0) and (cg == 0 or (g[0] >= 0 and g[-1] < len(s))), w
        assert np.all(idx_gpu[pw, cg:] == -1), f"row {w}: padding"
        assert np.isin(diag, g).all(), f"row {w}: a key of the block's own rows is missing"
        diff = np.setxor1d(g, kd_i[t, :kd_c[t]])
        if diff.size:
            mismatched += 1
            assert not np.isin(diff, diag).any()
            if mode == oracle.MINS_TILED:
                cut = running_threshold(s, param, tiling[0], tiling[1])[diff]
            elif mode == oracle.MINS:
                cut = s.max() - param
            else:
                cut = s[plain_i[t, :plain_c[t]]].min()
            tol = REL_TOL * np.abs(s).max()
            assert np.all(np.abs(s[diff] - cut) <= tol), \
                f"row {w}: keep-diagonal lists differ beyond near-tie: {np.abs(s[diff] - cut).max()}"
    return mismatched


def _scores(q, k, block, causal, rows, chunk=256):
    """The oracle's scores of the listed blocks, computed a chunk at a time."""
    rows = [int(w) for w in rows]
    for c0 in range(0, len(rows), chunk):
        yield from oracle.pooled_scores_rows(q, k, block, causal, rows[c0:c0 + chunk])


def running_threshold(s, alpha, bk, gk):
    """Per key: (maximum over its group's tiles up to its own tile) - alpha,
    the threshold Algorithm 1 compares it with (used only to place the
    tolerance of the cross-tile minS rule; the reference set is the oracle's)."""
    L = len(s)
    thr = np.empty(L)
    gs = bk * gk
    for g0 in range(0, L, gs):
        run = -np.inf
        for t0 in range(g0, min(L, g0 + gs), bk):
            t1 = min(L, t0 + bk)
            run = max(run, s[t0:t1].max())
            thr[t0:t1] = run - alpha
    return thr


def check_rows_tiled(q, k, block, alpha, causal, bk, gk, idx_gpu, cnt_gpu, rows, compact=False):
    """Cross-tile minS parity for rows none of which exceeded the GPU's cap.
    Returns the number of rows whose sets differ (all within the rule)."""
    B, Hq, N, D = q.shape
    Np = (N + block - 1) // block
    cap_o = N
    if compact:
        idx_o, cnt_o, ncl = oracle.select_mins_tiled(q, k, block, alpha, causal, cap_o, bk, gk,
                                                     rows=rows, compact=True)
        pos = {int(w): t for t, w in enumerate(rows)}
    else:
        idx_o, cnt_o, ncl = oracle.select_mins_tiled(q, k, block, alpha, causal, cap_o, bk, gk,
                                                     rows=rows)
        pos = {int(w): int(w) for w in rows}
    assert ncl == 0
    idx_o = idx_o.reshape(-1, cap_o)
    cnt_o = cnt_o.reshape(-1)
    idx_gpu = idx_gpu.reshape(-1, idx_gpu.shape[-1])
    cnt_gpu = cnt_gpu.reshape(-1)
    mismatched = 0
    for w, s in zip(rows, _scores(q, k, block, causal, rows)):
        w = int(w)
        pw = pos[w]
        L = len(s)
        tol = REL_TOL * np.abs(s).max()
        cg, co = int(cnt_gpu[pw]), int(cnt_o[pw])
        g = idx_gpu[pw, :cg]
        o = idx_o[pw, :co]
        assert cg < idx_gpu.shape[1] or cg == co, (w, cg)
        assert np.all(np.diff(g) > 0), f"row {w}: not strictly ascending"
        assert cg == 0 or (g[0] >= 0 and g[-1] < L), f"row {w}: index out of range"
        assert np.all(idx_gpu[pw, cg:] == -1), f"row {w}: padding"
        diff = np.setxor1d(g, o)
        if diff.size:
            mismatched += 1
            thr = running_threshold(s, alpha, bk, gk)
            gap = np.abs(s[diff] - thr[diff])
            assert np.all(gap <= tol), f"row {w}: cross-tile minS differs beyond near-threshold: {gap.max()}"
    return mismatched
