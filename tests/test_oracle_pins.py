"""Pins of the CPU oracle against facts fixed by the paper's definitions and by
mathematics: brute force on tiny inputs, library routines, closed forms and
invariants.  None of these re-types the oracle's own arithmetic.

Passages: Eq. 1 and Eq. 2, the estimated map and topK/topP of Sec. 3.1,
Eq. 3 (minS) and Algorithm 1's per-group running max, Eq. 4 and Algorithm 2.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2603_29494_amd import synth


def _bf16_nearest_by_search(x: float) -> int:
    """Nearest bf16 to x by searching neighbouring bit patterns (ties: even)."""
    if x == 0.0:
        return 0x8000 if math.copysign(1.0, x) < 0 else 0
    f32 = np.array([x], dtype=np.float32)
    base = int(f32.view(np.uint32)[0] >> 16)
    best = None
    for cand in range(base - 3, base + 4):
        if not 0 <= cand <= 0xFFFF:
            continue
        val = float(oracle.bf16_to_f64(np.array([cand], dtype=np.uint16))[0])
        if not math.isfinite(val):
            continue
        err = abs(val - x)
        key = (err, cand & 1)
        if best is None or key < best[0]:
            best = (key, cand)
    return best[1]


def test_bf16_round_is_nearest_even():
    r = np.random.Generator(np.random.PCG64(1))
    xs = list(r.standard_normal(400) * 10.0 ** r.uniform(-40, 30, 400))
    # exact midpoints between neighbouring bf16 values, both parities
    for bits in (0x3F80, 0x3F81, 0x4049, 0x404A, 0xC123, 0x0001, 0x0080, 0x7F7E):
        lo = float(oracle.bf16_to_f64(np.array([bits], dtype=np.uint16))[0])
        hi = float(oracle.bf16_to_f64(np.array([bits + 1], dtype=np.uint16))[0])
        xs += [(lo + hi) / 2, lo + (hi - lo) * 0.4999, lo + (hi - lo) * 0.5001]
    xs += [1e-45, -3e-41, 2.0 ** -133, 1.5 * 2.0 ** -133]
    got = oracle.bf16_round(np.array(xs))
    for x, g in zip(xs, got):
        assert int(g) == _bf16_nearest_by_search(x), (x, hex(int(g)))


def test_bf16_round_agrees_with_torch_on_fp32_values():
    # torch rounds fp32 -> bf16 to nearest even; on fp32 inputs one rounding step
    # is the same as ours.
    r = np.random.Generator(np.random.PCG64(2))
    x = (r.standard_normal(20000) * 3).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.bf16_round(x.astype(np.float64)), ref)


@pytest.mark.parametrize("N,P", [(64, 16), (70, 16), (5, 1), (33, 64), (130, 128)])
def test_pool_is_rounded_block_mean(N, P):
    q = synth.random_bits(10 + N, (1, 2, N, 8))
    qp = oracle.pool(q, P)
    qf = oracle.bf16_to_f64(q)
    Np = (N + P - 1) // P
    assert qp.shape == (1, 2, Np, 8)
    for i in range(Np):
        mean = qf[:, :, i * P:min(N, (i + 1) * P), :].mean(axis=2)   # numpy mean (library)
        expect = np.array([_bf16_nearest_by_search(float(m)) for m in mean.ravel()], dtype=np.uint16)
        assert np.array_equal(qp[:, :, i, :].ravel(), expect)


def test_pool_special_cases():
    q = synth.random_bits(3, (1, 1, 40, 16))
    assert np.array_equal(oracle.pool(q, 1), q)                      # P = 1: Q_p = Q
    same = np.repeat(q[:, :, :1, :], 40, axis=2)
    assert np.array_equal(oracle.pool(same, 16)[0, 0], np.repeat(q[0, 0, :1], 3, axis=0))


@pytest.mark.parametrize("causal", [False, True])
def test_scores_match_numpy(causal):
    q = synth.random_bits(4, (1, 4, 100, 32))
    k = synth.random_bits(5, (1, 2, 100, 32))
    P = 16
    qp = oracle.bf16_to_f64(oracle.pool(q, P))
    kf = oracle.bf16_to_f64(k)
    for h in range(4):
        for i in range(7):
            s = oracle.pooled_scores(q, k, P, causal, 0, h, i)
            L = min(100, (i + 1) * P) if causal else 100
            ref = (kf[0, h // 2, :L] @ qp[0, h, i]) / math.sqrt(32)    # numpy matmul
            assert s.shape == (L,)
            np.testing.assert_allclose(s, ref, rtol=1e-12, atol=1e-14)


def test_topk_count_values():
    assert oracle.topk_count(0.15, 75600) == 11340
    assert oracle.topk_count(0.125, 1024) == 128
    assert oracle.topk_count(0.10, 64) == 7
    assert oracle.topk_count(0.10, 32768) == 3277
    assert oracle.topk_count(0.1, 640) == 64
    assert 0.07 * 100 > 7.0 and oracle.topk_count(0.07, 100) == 7   # rounding guard
    assert oracle.topk_count(1e-9, 50) == 1
    assert oracle.topk_count(1.0, 50) == 50


def _tiny_layer(seed, N, D=16, dup=False):
    q = synth.random_bits(seed, (1, 1, N, D))
    k = synth.random_bits(seed + 1, (1, 1, N, D))
    if dup:  # identical key rows create exact score ties
        k[0, 0, 5] = k[0, 0, 2]
        k[0, 0, 9] = k[0, 0, 2]
        k[0, 0, 11] = k[0, 0, 7]
    return q, k


def _brute_topk(s, kk):
    best = None
    for sub in itertools.combinations(range(len(s)), kk):
        key = (-sum(s[j] for j in sub), sub)     # max sum, then lexicographically smallest
        if best is None or key < best:
            best = key
    return list(best[1])


@pytest.mark.parametrize("seed,N,ratio,dup", [(11, 12, 0.25, False), (12, 12, 0.5, True),
                                              (13, 14, 0.3, True), (14, 9, 0.6, False)])
def test_topk_matches_brute_force(seed, N, ratio, dup):
    q, k = _tiny_layer(seed, N, dup=dup)
    idx, cnt, _ = oracle.select(q, k, N, oracle.TOPK, ratio, False, N)
    s = oracle.pooled_scores(q, k, N, False, 0, 0, 0)
    kk = oracle.topk_count(ratio, N)
    assert cnt[0, 0, 0] == kk
    assert list(idx[0, 0, 0, :kk]) == _brute_topk(list(s), kk)
    assert np.all(idx[0, 0, 0, kk:] == -1)


def test_topk_invariants_and_scale():
    q, k = _tiny_layer(21, 200, D=32)
    P = 50
    idx, cnt, _ = oracle.select(q, k, P, oracle.TOPK, 0.2, True, 200)
    for i in range(4):
        s = oracle.pooled_scores(q, k, P, True, 0, 0, i)
        L = len(s)
        c = cnt[0, 0, i]
        assert c == oracle.topk_count(0.2, L)
        sel = idx[0, 0, i, :c]
        assert np.all(np.diff(sel) > 0) and sel.min() >= 0 and sel.max() < L
        rest = np.setdiff1d(np.arange(L), sel)
        assert s[sel].min() >= s[rest].max()
    k2 = oracle.bf16_round(oracle.bf16_to_f64(k) * 2.0)    # exact rescale of every score
    idx2, cnt2, _ = oracle.select(q, k2, P, oracle.TOPK, 0.2, True, 200)
    assert np.array_equal(idx, idx2) and np.array_equal(cnt, cnt2)
    idx3, cnt3, _ = oracle.select(q, k, P, oracle.TOPK, 1.0, True, 200)
    for i in range(4):
        L = min(200, (i + 1) * P)
        assert list(idx3[0, 0, i, :cnt3[0, 0, i]]) == list(range(L))


def _brute_topp(s, p):
    s = np.asarray(s)
    e = np.exp(s - s.max())
    Z = e.sum()
    best = None
    for n in range(1, len(s) + 1):
        for sub in itertools.combinations(range(len(s)), n):
            m = e[list(sub)].sum() / Z
            if m >= p:
                key = (n, -m, sub)
                if best is None or key < best:
                    best = key
        if best is not None:
            return list(best[2])
    return list(range(len(s)))


@pytest.mark.parametrize("seed,N,p", [(31, 10, 0.5), (32, 12, 0.8), (33, 11, 0.95), (34, 12, 0.3)])
def test_topp_matches_brute_force(seed, N, p):
    q, k = _tiny_layer(seed, N, D=16)
    k = oracle.bf16_round(oracle.bf16_to_f64(k) * 3.0)   # spread the scores
    idx, cnt, _ = oracle.select(q, k, N, oracle.TOPP, p, False, N)
    s = oracle.pooled_scores(q, k, N, False, 0, 0, 0)
    assert list(idx[0, 0, 0, :cnt[0, 0, 0]]) == sorted(_brute_topp(s, p))


@pytest.mark.parametrize("L,p", [(100, 0.333), (640, 0.9512), (77, 0.5)])
def test_topp_uniform_scores(L, p):
    # Q = 0 makes every score 0: the mass is uniform and topP keeps ceil(p L)
    # keys, the lowest indices first.
    q = np.zeros((1, 1, L, 16), dtype=np.uint16)
    k = synth.random_bits(41, (1, 1, L, 16))
    idx, cnt, _ = oracle.select(q, k, L, oracle.TOPP, p, False, L)
    t = math.ceil(p * L)
    assert abs(p * L - round(p * L)) > 1e-6
    assert cnt[0, 0, 0] == t and list(idx[0, 0, 0, :t]) == list(range(t))


def test_topp_mass_reaching_p_exactly_stops():
    # uniform scores, p * L an integer: the cumulative mass equals p exactly
    # after p * L keys, and "reaches p" means >= p, so no further key is taken
    L, p = 100, 0.25
    q = np.zeros((1, 1, L, 16), dtype=np.uint16)
    k = synth.random_bits(42, (1, 1, L, 16))
    idx, cnt, _ = oracle.select(q, k, L, oracle.TOPP, p, False, L)
    assert cnt[0, 0, 0] == 25 and list(idx[0, 0, 0, :25]) == list(range(25))


def test_topp_mass_invariants():
    q, k = _tiny_layer(51, 300, D=32)
    k = oracle.bf16_round(oracle.bf16_to_f64(k) * 4.0)
    for p in (0.5, 0.9, 0.99):
        idx, cnt, _ = oracle.select(q, k, 100, oracle.TOPP, p, False, 300)
        for i in range(3):
            s = oracle.pooled_scores(q, k, 100, False, 0, 0, i)
            e = np.exp(s - s.max())
            sel = idx[0, 0, i, :cnt[0, 0, i]]
            mass = e[sel].sum() / e.sum()
            assert mass >= p - 1e-12
            weakest = sel[np.argmin(s[sel])]
            assert (e[sel].sum() - e[weakest]) / e.sum() < p
            rest = np.setdiff1d(np.arange(300), sel)
            assert s[sel].min() >= s[rest].max()


def test_threshold_cap_keeps_best():
    q, k = _tiny_layer(52, 256, D=32)
    idx, cnt, ncl = oracle.select(q, k, 64, oracle.TOPP, 0.99, False, 20)
    assert ncl == 4 and np.all(cnt == 20)
    for i in range(4):
        s = oracle.pooled_scores(q, k, 64, False, 0, 0, i)
        top = np.argsort(-s, kind="stable")[:20]
        assert set(idx[0, 0, i]) == set(top)
    with pytest.raises(ValueError):
        oracle.select(q, k, 64, oracle.TOPK, 0.5, False, 20)


def test_mins_special_cases():
    r = np.random.Generator(np.random.PCG64(61))
    s = r.standard_normal(1000)
    s[[17, 400]] = s.max() + 1.0
    q, k = _tiny_layer(62, 64)
    assert list(oracle.mins_progressive(s, 0.0, 1000, 1)) == [17, 400]     # alpha = 0: argmax ties
    assert list(oracle.mins_progressive(s, np.inf, 16, 16)) == list(range(1000))
    for alpha in (0.1, 0.5, 2.0):
        glob = set(np.nonzero(s >= s.max() - alpha)[0])
        prog = set(oracle.mins_progressive(s, alpha, 16, 16))
        assert glob <= prog            # a running max never exceeds the global max
    # when each group's max sits in its first tile the running max is the group max
    s2 = r.standard_normal(512)
    for g0 in range(0, 512, 64):
        s2[g0] = s2[g0:g0 + 64].max() + 0.5
    prog = oracle.mins_progressive(s2, 0.7, 16, 4)
    expect = [j for j in range(512) if s2[j] >= s2[(j // 64) * 64:(j // 64) * 64 + 64].max() - 0.7]
    assert list(prog) == expect
    # global minS through select(): alpha = 0 keeps the argmax
    idx, cnt, _ = oracle.select(q, k, 64, oracle.MINS, 0.0, False, 64)
    sc = oracle.pooled_scores(q, k, 64, False, 0, 0, 0)
    assert list(idx[0, 0, 0, :cnt[0, 0, 0]]) == [int(np.argmax(sc))]


def test_mins_tiled_worked_examples():
    # Algorithm 1 by hand, bk = 2, gk = 2 (groups of 4 keys), alpha = 1.5:
    #   group {0..3}: tile {0,1} running max 3 -> keep s >= 1.5: key 1;
    #                 tile {2,3} running max 5 -> keep s >= 3.5: key 3;
    #   group {4,5}:  running max restarts, 3.2 -> keep s >= 1.7: key 5.
    # (A running max over earlier tiles only would keep key 0; one never reset
    # would drop key 5; the row maximum of Eq. 3 keeps only key 3.)
    s = np.array([1.0, 3.0, 2.0, 5.0, 0.0, 3.2])
    assert list(oracle.mins_progressive(s, 1.5, 2, 2)) == [1, 3, 5]
    # comparator >= (Eq. 3): a key exactly alpha below the running max stays
    assert list(oracle.mins_progressive(np.array([2.0, 1.0]), 1.0, 2, 1)) == [0, 1]


def test_mins_tiled_single_group_is_prefix_max():
    # one group, one-key tiles: key j is kept iff s_j >= max(s_0..s_j) - alpha
    r = np.random.Generator(np.random.PCG64(71))
    s = r.standard_normal(3000)
    for alpha in (0.0, 0.3, 1.0):
        expect = np.nonzero(s >= np.maximum.accumulate(s) - alpha)[0]
        assert np.array_equal(oracle.mins_progressive(s, alpha, 1, 10 ** 6), expect)


@pytest.mark.parametrize("causal", [False, True])
def test_select_mins_tiled_per_block(causal):
    q, k = _tiny_layer(73, 300, D=32)
    Np = 5
    idx, cnt, ncl = oracle.select_mins_tiled(q, k, 64, 0.05, causal, 300, bk=16, gk=4)
    assert ncl == 0
    gidx, gcnt, _ = oracle.select(q, k, 64, oracle.MINS, 0.05, causal, 300)
    for i in range(Np):
        s = oracle.pooled_scores(q, k, 64, causal, 0, 0, i)
        row = idx[0, 0, i, :cnt[0, 0, i]]
        assert np.array_equal(row, oracle.mins_progressive(s, 0.05, 16, 4))
        assert np.all(idx[0, 0, i, cnt[0, 0, i]:] == -1)
        assert set(gidx[0, 0, i, :gcnt[0, 0, i]]) <= set(row)   # running max <= row max
    # alpha = inf keeps every eligible key
    idx, cnt, _ = oracle.select_mins_tiled(q, k, 64, np.inf, causal, 300, bk=16, gk=16)
    for i in range(Np):
        L = min(300, 64 * (i + 1)) if causal else 300
        assert list(idx[0, 0, i, :cnt[0, 0, i]]) == list(range(L))
    # a block keeping more than cap keys keeps its first cap keys and is counted
    full, fcnt, _ = oracle.select_mins_tiled(q, k, 64, 0.05, causal, 300, bk=16, gk=4)
    cap = int(np.median(fcnt))
    idx, cnt, ncl = oracle.select_mins_tiled(q, k, 64, 0.05, causal, cap, bk=16, gk=4)
    assert ncl == int(np.sum(fcnt > cap))
    assert np.array_equal(cnt, np.minimum(fcnt, cap))
    assert np.array_equal(idx[0, 0], full[0, 0, :, :cap])


def _all_keys(N, P, causal, Np, B=1, H=1):
    cap = N
    idx = np.full((B, H, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, H, Np), dtype=np.int32)
    for i in range(Np):
        L = min(N, (i + 1) * P) if causal else N
        idx[:, :, i, :L] = np.arange(L)
        cnt[:, :, i] = L
    return idx, cnt


@pytest.mark.parametrize("causal", [False, True])
def test_full_keep_equals_dense_and_sdpa(causal):
    B, Hq, Hkv, N, D, P = 1, 4, 2, 70, 16, 16
    q = synth.random_bits(71, (B, Hq, N, D))
    k = synth.random_bits(72, (B, Hkv, N, D))
    v = synth.random_bits(73, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    idx, cnt = _all_keys(N, P, causal, Np, B, Hq)
    o, lse = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
    od, lsed = oracle.dense_attn(q, k, v, causal)
    np.testing.assert_allclose(o, od, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lsed, rtol=0, atol=1e-12)
    tq, tk, tv = (torch.from_numpy(oracle.bf16_to_f64(x)) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal,
                                                           enable_gqa=True)
    np.testing.assert_allclose(o, ref.numpy(), rtol=0, atol=1e-12)


def test_single_key_and_zero_query():
    B, H, N, D, P = 1, 1, 48, 16, 16
    q = synth.random_bits(81, (B, H, N, D))
    k = synth.random_bits(82, (B, H, N, D))
    v = synth.random_bits(83, (B, H, N, D))
    idx = np.full((1, 1, 3, 4), -1, dtype=np.int32)
    cnt = np.array([[[1, 1, 1]]], dtype=np.int32)
    idx[0, 0, :, 0] = [5, 30, 40]
    o, lse = oracle.sparse_attn(q, k, v, idx, cnt, P, False)
    vf = oracle.bf16_to_f64(v)
    qf, kf = oracle.bf16_to_f64(q), oracle.bf16_to_f64(k)
    for i, j in enumerate([5, 30, 40]):
        assert np.array_equal(o[0, 0, i * P:(i + 1) * P], np.repeat(vf[0, 0, j:j + 1], P, 0))
        # one visible key: LSE is that key's scaled score, q_r . k_j / sqrt(D)
        np.testing.assert_allclose(lse[0, 0, i * P:(i + 1) * P],
                                   qf[0, 0, i * P:(i + 1) * P] @ kf[0, 0, j] / np.sqrt(D),
                                   rtol=0, atol=1e-12)
    z = np.zeros_like(q)
    idx2 = np.array([[[[1, 4, 9, 20]] * 3]], dtype=np.int32).reshape(1, 1, 3, 4)
    cnt2 = np.full((1, 1, 3), 4, dtype=np.int32)
    o2, lse2 = oracle.sparse_attn(z, k, v, idx2, cnt2, P, False)
    np.testing.assert_allclose(o2[0, 0], np.repeat(vf[0, 0, [1, 4, 9, 20]].mean(0)[None], N, 0),
                               rtol=0, atol=1e-14)
    # Q = 0: every score is 0, so LSE = log(number of visible keys)
    np.testing.assert_allclose(lse2[0, 0], np.full(N, np.log(4.0)), rtol=0, atol=1e-14)


def test_lse_matches_torch_logsumexp():
    # LSE over each row's visible listed keys (causal: j <= r) against torch's
    # logsumexp in fp64 on the same scaled scores; rows with nothing visible are -inf.
    import torch
    B, H, N, D, P = 1, 2, 40, 16, 8
    q = synth.random_bits(91, (B, H, N, D))
    k = synth.random_bits(92, (B, H, N, D))
    v = synth.random_bits(93, (B, H, N, D))
    r = np.random.default_rng(94)
    Np, cap = N // P, 12
    idx = np.full((B, H, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, H, Np), dtype=np.int32)
    for h in range(H):
        for i in range(Np):
            c = int(r.integers(0, cap + 1))
            idx[0, h, i, :c] = np.sort(r.choice(N, size=c, replace=False))
            cnt[0, h, i] = c
    _, lse = oracle.sparse_attn(q, k, v, idx, cnt, P, True)
    qf = torch.from_numpy(oracle.bf16_to_f64(q))
    kf = torch.from_numpy(oracle.bf16_to_f64(k))
    for h in range(H):
        for row in range(N):
            keys = [j for j in idx[0, h, row // P, :cnt[0, h, row // P]] if j <= row]
            if not keys:
                assert np.isneginf(lse[0, h, row])
                continue
            s = (kf[0, h, keys] @ qf[0, h, row]) / np.sqrt(D)
            assert abs(lse[0, h, row] - torch.logsumexp(s, 0).item()) <= 1e-12


def test_empty_causal_rows():
    B, H, N, D, P = 1, 1, 32, 16, 16
    q, k, v = (synth.random_bits(s, (B, H, N, D)) for s in (91, 92, 93))
    idx = np.array([[[[10, 12, -1], [3, 20, 31]]]], dtype=np.int32)
    cnt = np.array([[[2, 3]]], dtype=np.int32)
    o, lse = oracle.sparse_attn(q, k, v, idx, cnt, P, True)
    assert np.all(o[0, 0, :10] == 0) and np.all(np.isneginf(lse[0, 0, :10]))
    assert np.all(np.isfinite(lse[0, 0, 10:]))
    oo, lo = oracle.sparse_attn_online(q, k, v, idx, cnt, P, True, 2)
    np.testing.assert_array_equal(oo[0, 0, :10], 0.0)
    assert np.all(np.isneginf(lo[0, 0, :10]))


@pytest.mark.parametrize("bk", [1, 3, 16, 64])
@pytest.mark.parametrize("causal", [False, True])
def test_online_recurrence_equals_materialised(bk, causal):
    B, Hq, Hkv, N, D, P = 1, 2, 1, 150, 16, 32
    q, k, v = (synth.random_bits(s, (B, h, N, D)) for s, h in ((101, Hq), (102, Hkv), (103, Hkv)))
    r = np.random.Generator(np.random.PCG64(104))
    Np = (N + P - 1) // P
    cap = 90
    idx = np.full((B, Hq, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, Hq, Np), dtype=np.int32)
    for h in range(Hq):
        for i in range(Np):
            c = int(r.integers(0, cap + 1))
            idx[0, h, i, :c] = np.sort(r.choice(N, size=c, replace=False))
            cnt[0, h, i] = c
    o, lse = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
    o2, lse2 = oracle.sparse_attn_online(q, k, v, idx, cnt, P, causal, bk)
    np.testing.assert_allclose(o2, o, rtol=0, atol=1e-12)
    fin = np.isfinite(lse)
    assert np.array_equal(fin, np.isfinite(lse2))
    np.testing.assert_allclose(lse2[fin], lse[fin], rtol=0, atol=1e-12)


def test_gqa_equals_replicated_kv():
    B, Hq, Hkv, N, D, P = 1, 6, 2, 64, 16, 16
    q = synth.random_bits(111, (B, Hq, N, D))
    k = synth.random_bits(112, (B, Hkv, N, D))
    v = synth.random_bits(113, (B, Hkv, N, D))
    kr, vr = np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1)   # contiguous grouping
    for mode, par in ((oracle.TOPK, 0.3), (oracle.TOPP, 0.7)):
        a = oracle.select(q, k, P, mode, par, True, N)
        b = oracle.select(q, kr, P, mode, par, True, N)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    idx, cnt, _ = oracle.select(q, k, P, oracle.TOPK, 0.3, False, N)
    o1, _ = oracle.sparse_attn(q, k, v, idx, cnt, P, False)
    o2, _ = oracle.sparse_attn(q, kr, vr, idx, cnt, P, False)
    np.testing.assert_array_equal(o1, o2)


def test_plumbing_workload_recovers_planted_columns():
    layer = synth.make_layer(1)
    w = layer.w
    idx, cnt, _ = oracle.select(layer.q, layer.k, w.block, oracle.TOPK, w.param, w.causal, 128)
    assert np.all(cnt == 128)
    recall = []
    for h in range(w.Hq):
        planted = set(layer.planted[h].tolist())
        for i in range(w.num_blocks):
            recall.append(len(planted & set(idx[0, h, i].tolist())) / len(planted))
    # the planted boost is 0.5 logit against a score spread of ~0.2, so most
    # (not all) planted columns land in every block's top 12.5%
    assert np.mean(recall) > 0.85


def test_compact_row_layout_matches_full_layout():
    """The compact layout (sampled rows only) is an indexing change: the same
    lists, counts, outputs and LSE as the full layout, row for row."""
    q = synth.random_bits(1, (1, 2, 300, 64))
    k = synth.random_bits(2, (1, 2, 300, 64))
    v = synth.random_bits(3, (1, 2, 300, 64))
    rows = [1, 4, 7, 9]
    Np = 5
    for mode, param in ((oracle.TOPK, 0.2), (oracle.TOPP, 0.9)):
        i1, c1, n1 = oracle.select(q, k, 64, mode, param, True, 300, rows=rows)
        i2, c2, n2 = oracle.select(q, k, 64, mode, param, True, 300, rows=rows, compact=True)
        assert n1 == n2
        for t, r in enumerate(rows):
            assert np.array_equal(i1.reshape(-1, 300)[r], i2[t])
            assert c1.reshape(-1)[r] == c2[t]
        o1, l1 = oracle.sparse_attn(q, k, v, i1, c1, 64, True, blocks=rows)
        o2, l2 = oracle.sparse_attn(q, k, v, i2, c2, 64, True, blocks=rows, compact=True)
        for t, r in enumerate(rows):
            i, h = r % Np, r // Np
            n = min(300, (i + 1) * 64) - i * 64
            assert np.array_equal(o1[0, h, i * 64:i * 64 + n], o2[t, :n])
            assert np.array_equal(l1[0, h, i * 64:i * 64 + n], l2[t, :n])
            assert np.isnan(o2[t, n:]).all()


def test_keep_diagonal_variant():
    # topK k = 1 with the block's own rows kept: the argmax plus the diagonal range
    q, k = _tiny_layer(81, 200, D=32)
    idx, cnt, _ = oracle.select(q, k, 64, oracle.TOPK, 1e-6, True, 200, keep_diag=True)
    for i in range(4):
        s = oracle.pooled_scores(q, k, 64, True, 0, 0, i)
        diag = set(range(64 * i, min(200, 64 * (i + 1))))
        want = sorted(diag | {int(np.argmax(s))})
        assert list(idx[0, 0, i, :cnt[0, 0, i]]) == want
    # keeping everything already keeps the diagonal
    a, ca, _ = oracle.select(q, k, 64, oracle.TOPK, 1.0, True, 200, keep_diag=True)
    b, cb, _ = oracle.select(q, k, 64, oracle.TOPK, 1.0, True, 200)
    assert np.array_equal(a, b) and np.array_equal(ca, cb)
    with pytest.raises(ValueError):   # lists must fit: 64 + k keys in 65 slots fails for k > 1
        oracle.select(q, k, 64, oracle.TOPK, 0.1, False, 65, keep_diag=True)


def _numpy_scores(q, k, P, causal, h, i, group):
    """Scaled pooled scores of block i from numpy: the pooled queries (pinned
    above against numpy means) times K, divided by sqrt(D)."""
    N, D = q.shape[2], q.shape[3]
    qp = oracle.bf16_to_f64(oracle.pool(q, P))[0, h, i]
    L = min(N, (i + 1) * P) if causal else N
    return (oracle.bf16_to_f64(k)[0, h // group, :L] @ qp) / math.sqrt(D)


@pytest.mark.parametrize("causal", [False, True])
def test_mins_select_is_numpy_threshold(causal):
    # Eq. 3 by its definition: every eligible key whose scaled pooled score is
    # >= the block's largest score minus alpha (alpha in scaled-score units;
    # an alpha scaled by sqrt(D), a > for >= or a threshold from another row
    # fails here).  Keys within 1e-9 of a threshold would make the comparison
    # depend on summation order; the data is checked to have none.
    N, P, D, Hq, Hkv = 300, 64, 32, 4, 2
    q = synth.random_bits(141, (1, Hq, N, D), scale=4.0)
    k = synth.random_bits(142, (1, Hkv, N, D))
    Np = (N + P - 1) // P
    partial = 0
    for alpha in (0.1, 0.5, 2.0):
        idx, cnt, ncl = oracle.select(q, k, P, oracle.MINS, alpha, causal, N)
        assert ncl == 0
        for h in range(Hq):
            for i in range(Np):
                s = _numpy_scores(q, k, P, causal, h, i, Hq // Hkv)
                thr = s.max() - alpha
                assert np.abs(s - thr).min() > 1e-9
                want = np.nonzero(s >= thr)[0]
                c = cnt[0, h, i]
                assert np.array_equal(idx[0, h, i, :c], want), (alpha, h, i)
                assert np.all(idx[0, h, i, c:] == -1)
                partial += 1 < c < len(s)
    assert partial > 10   # the thresholds cut inside most rows, not at an end


@pytest.mark.parametrize("causal", [False, True])
def test_mins_cap_keeps_first_of_total_order(causal):
    # A block whose minS set exceeds cap keeps the first cap keys of the set in
    # the total order (score descending, index ascending) -- numpy's lexsort of
    # (index, -score) -- listed ascending, and is counted once.  Duplicate key
    # rows put exact ties at the cap boundary (the lower index must win).
    N, P, D = 256, 32, 32
    q = synth.random_bits(151, (1, 1, N, D), scale=4.0)
    k = synth.random_bits(152, (1, 1, N, D))
    k[0, 0, 40::7] = k[0, 0, 3]
    for alpha, cap in ((0.4, 9), (1.0, 25), (3.0, 60)):
        idx, cnt, ncl = oracle.select(q, k, P, oracle.MINS, alpha, causal, cap)
        clamped = 0
        for i in range(N // P):
            s = _numpy_scores(q, k, P, causal, 0, i, 1)
            thr = s.max() - alpha
            assert np.abs(s - thr).min() > 1e-9
            full = set(np.nonzero(s >= thr)[0].tolist())
            order = np.lexsort((np.arange(len(s)), -s))
            kept = [int(j) for j in order if int(j) in full][:cap]
            clamped += len(full) > cap
            c = cnt[0, 0, i]
            assert c == min(cap, len(full))
            assert list(idx[0, 0, i, :c]) == sorted(kept), (alpha, i)
        assert ncl == clamped and clamped > 0


def test_oracle_plan_worked_examples():
    # Eq. 5 worked by hand (the same tables the library's test uses):
    #   head 0: (sparsity, perf) = (0.1, 1.0) (0.5, 0.8) (0.9, 0.2)
    #   head 1:                    (0.2, 1.0) (0.6, 0.9) (0.8, 0.5)
    # Mean sparsity >= 0.5 needs a summed sparsity >= 1.0.  The feasible
    # choices (summed sparsity -> summed perf): (1,1) 1.1 -> 1.7, (1,2) 1.3 ->
    # 1.3, (2,0) 1.1 -> 1.2, (2,1) 1.5 -> 1.1, (2,2) 1.7 -> 0.7; the others
    # fall short (e.g. (0,2) 0.9).  So 1.7 at (1,1) is the only optimum.
    # >= 0.85 (sum >= 1.7) leaves (2,2): 0.7; target 0 takes each head's best
    # perf, (0,0): 2.0; 0.9 (sum >= 1.8) is out of reach.
    sp = np.array([[0.1, 0.5, 0.9], [0.2, 0.6, 0.8]])
    pf = np.array([[1.0, 0.8, 0.2], [1.0, 0.9, 0.5]])
    best, optima = oracle.plan_filter_ratios(sp, pf, 0.5)
    assert best == pytest.approx(1.7) and optima == [(1, 1)]
    best, optima = oracle.plan_filter_ratios(sp, pf, 0.85)
    assert best == pytest.approx(0.7) and optima == [(2, 2)]
    best, optima = oracle.plan_filter_ratios(sp, pf, 0.0)
    assert best == pytest.approx(2.0) and optima == [(0, 0)]
    assert oracle.plan_filter_ratios(sp, pf, 0.9) == (None, [])
    # Tied optima: two identical heads with (0.2, 1.0) (0.4, 0.5); mean >= 0.3
    # needs one head at 0.4: (0,1) and (1,0) both give 1.5, (1,1) gives 1.0.
    sp2 = np.array([[0.2, 0.4], [0.2, 0.4]])
    pf2 = np.array([[1.0, 0.5], [1.0, 0.5]])
    best, optima = oracle.plan_filter_ratios(sp2, pf2, 0.3)
    assert best == pytest.approx(1.5) and sorted(optima) == [(0, 1), (1, 0)]
    # "at least": a mean exactly at the target is feasible
    best, optima = oracle.plan_filter_ratios(np.array([[0.5], [0.5]]), np.array([[0.3], [0.4]]), 0.5)
    assert best == pytest.approx(0.7) and optima == [(0, 0)]


def _random_lists(seed, B, H, Np, N, P, causal, cap):
    r = np.random.Generator(np.random.PCG64(seed))
    idx = np.full((B, H, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, H, Np), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            for i in range(Np):
                L = min(N, (i + 1) * P) if causal else N
                c = int(r.integers(0, min(cap, L) + 1))
                idx[b, h, i, :c] = np.sort(r.choice(L, size=c, replace=False))
                cnt[b, h, i] = c
    return idx, cnt


@pytest.mark.parametrize("causal", [False, True])
def test_kept_mass_matches_torch_softmax(causal):
    # Sec. 2.2's recall per row: torch's softmax (fp64, library routine) of the
    # row's scaled scores over the keys it sees, summed over its block's listed
    # keys; GQA through K rows shared by two query heads.
    B, Hq, Hkv, N, D, P = 1, 4, 2, 70, 16, 16
    q = synth.random_bits(161, (B, Hq, N, D), scale=2.0)
    k = synth.random_bits(162, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    idx, cnt = _random_lists(163, B, Hq, Np, N, P, causal, 30)
    kept = oracle.kept_mass(q, k, idx, cnt, P, causal)
    qf = torch.from_numpy(oracle.bf16_to_f64(q))
    kf = torch.from_numpy(oracle.bf16_to_f64(k))
    for h in range(Hq):
        for r in range(N):
            n = r + 1 if causal else N
            p = torch.softmax((kf[0, h // 2, :n] @ qf[0, h, r]) / math.sqrt(D), 0).numpy()
            listed = [j for j in idx[0, h, r // P, :cnt[0, h, r // P]] if j < n]
            assert abs(kept[0, h, r] - p[listed].sum()) <= 1e-12


def test_kept_mass_closed_forms():
    B, H, N, D, P = 1, 2, 96, 16, 32
    q = synth.random_bits(171, (B, H, N, D))
    k = synth.random_bits(172, (B, H, N, D))
    v = synth.random_bits(173, (B, H, N, D))
    Np = N // P
    for causal in (False, True):
        full_i, full_c = _all_keys(N, P, causal, Np, B, H)
        assert np.all(oracle.kept_mass(q, k, full_i, full_c, P, causal) == 1.0)   # every key
        empty_c = np.zeros_like(full_c)
        assert np.all(oracle.kept_mass(q, k, full_i, empty_c, P, causal) == 0.0)  # no key
        # Q = 0: uniform rows, so the recall is the share of visible keys listed
        idx, cnt = _random_lists(174, B, H, Np, N, P, causal, 40)
        kz = oracle.kept_mass(np.zeros_like(q), k, idx, cnt, P, causal)
        for h in range(H):
            for r in range(N):
                n = r + 1 if causal else N
                seen = sum(1 for j in idx[0, h, r // P, :cnt[0, h, r // P]] if j < n)
                assert abs(kz[0, h, r] - seen / n) <= 1e-15
        # the kept share is exp(LSE over the visible listed keys - LSE over all
        # visible keys), from the sparse and dense attention routines
        kept = oracle.kept_mass(q, k, idx, cnt, P, causal)
        _, lse_s = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
        _, lse_d = oracle.dense_attn(q, k, v, causal)
        np.testing.assert_allclose(kept, np.exp(lse_s - lse_d), rtol=1e-12, atol=1e-300)


def test_head_sparsity_definition():
    # Eq. 5's sp_h by hand: 2 heads, N = 10, P = 4 (blocks of 4, 4, 2 rows).
    # Non-causal: each block has 10 eligible keys (30 per head); causal: 4, 8,
    # 10 (22 per head).
    cnt = np.array([[[4, 2, 3], [10, 10, 10]]], dtype=np.int32)
    np.testing.assert_array_equal(oracle.head_sparsity(cnt, 10, 4, False),
                                  [1 - 9 / 30, 0.0])
    cc = np.array([[[4, 2, 3], [4, 8, 10]]], dtype=np.int32)
    np.testing.assert_array_equal(oracle.head_sparsity(cc, 10, 4, True), [1 - 9 / 22, 0.0])
    # the batch averages: two copies of the same head give the same sparsity
    two = np.concatenate([cnt, cnt], axis=0)
    np.testing.assert_array_equal(oracle.head_sparsity(two, 10, 4, False),
                                  oracle.head_sparsity(cnt, 10, 4, False))
