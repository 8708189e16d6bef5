"""GPU parity of important-vector selection (Sec. 3.1: pooled-query scores,
row-wise topK / topP, minS of Eq. 3 and Algorithm 1's cross-tile minS) against
the oracle, through the C ABI.  The index-set rule is in selection_parity.py."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_29494_amd as va
from paper_2603_29494_amd import synth

from selection_parity import check_rows, check_rows_keep_diag, check_rows_tiled

pytestmark = pytest.mark.gpu


def dev(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def run(q, k, block, mode, param, causal, cap=None):
    N = q.shape[2]
    if cap is None:
        cap = va.max_count(N, block, causal, "topk" if mode == oracle.TOPK else "topp", param)
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cnt = va.select(dev(q), dev(k), block, mode, param, causal, cap=cap, n_clamped=ncl)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), cnt.cpu().numpy(), cap, int(ncl.item())


def all_rows(q, block):
    B, H, N, _ = q.shape
    return list(range(B * H * ((N + block - 1) // block)))


CASES = [
    # B, Hq, Hkv, N, D, block, causal, mode, param
    (1, 2, 2, 300, 128, 64, False, oracle.TOPK, 0.15),
    (1, 4, 2, 333, 128, 64, True, oracle.TOPK, 0.1),
    (2, 2, 1, 257, 64, 64, False, oracle.TOPK, 0.5),
    (1, 3, 3, 520, 64, 16, True, oracle.TOPK, 0.3),
    (1, 2, 2, 700, 128, 128, False, oracle.TOPP, 0.9),
    (1, 4, 1, 450, 128, 64, True, oracle.TOPP, 0.95),
    (1, 2, 2, 1000, 64, 48, False, oracle.TOPP, 0.5),
    (1, 1, 1, 5000, 128, 64, False, oracle.TOPK, 0.15),
    (1, 1, 1, 5000, 128, 64, True, oracle.TOPP, 0.9),
]


@pytest.mark.parametrize("case", CASES)
def test_select_matches_oracle(gpu, case):
    B, Hq, Hkv, N, D, block, causal, mode, param = case
    q, k, _ = synth.planted_case(hash(case) % 10000, B, Hq, Hkv, N, D)
    idx, cnt, cap, _ = run(q, k, block, mode, param, causal)
    rows = all_rows(q, block)
    mism = check_rows(q, k, block, mode, param, causal, cap, idx, cnt, rows)
    assert mism <= max(1, len(rows) // 20)


@pytest.mark.parametrize("mode,param", [(oracle.TOPK, 0.125), (oracle.TOPP, 0.9)])
def test_plumbing_workload(gpu, mode, param):
    layer = synth.make_layer(1)
    w = layer.w
    idx, cnt, cap, _ = run(layer.q, layer.k, w.block, mode, param, w.causal)
    check_rows(layer.q, layer.k, w.block, mode, param, w.causal, cap, idx, cnt,
               all_rows(layer.q, w.block))


@pytest.mark.parametrize("mode,param", [(oracle.TOPK, 0.3), (oracle.TOPP, 0.5), (oracle.TOPP, 0.999)])
def test_tie_storm_zero_queries(gpu, mode, param):
    # Q = 0: every score is exactly 0; the kept keys are the lowest indices.
    N, block = 3000, 64
    q = np.zeros((1, 2, N, 128), dtype=np.uint16)
    k = synth.random_bits(5, (1, 2, N, 128))
    idx, cnt, cap, _ = run(q, k, block, mode, param, False)
    idx_o, cnt_o, _ = oracle.select(q, k, block, mode, param, False, cap)
    assert np.array_equal(cnt, cnt_o)
    assert np.array_equal(idx, idx_o)


def test_partial_ties_from_duplicate_keys(gpu):
    # many identical key rows: ties at the cut, broken toward lower indices
    N, block = 2048, 64
    k = synth.random_bits(6, (1, 1, N, 128))
    k[0, 0, 1::3] = k[0, 0, 0]
    q = synth.random_bits(7, (1, 1, N, 128))
    for mode, param in ((oracle.TOPK, 0.2), (oracle.TOPK, 0.4), (oracle.TOPP, 0.7)):
        idx, cnt, cap, _ = run(q, k, block, mode, param, False)
        check_rows(q, k, block, mode, param, False, cap, idx, cnt, all_rows(q, block))


def test_threshold_clamped_to_cap(gpu):
    q, k, _ = synth.planted_case(8, 1, 2, 2, 1500, 128, frac=0.02, logits=1.0)
    cap = 200
    idx, cnt, _, ncl = run(q, k, 64, oracle.TOPP, 0.95, False, cap=cap)
    _, cnt_o, ncl_o = oracle.select(q, k, 64, oracle.TOPP, 0.95, False, cap)
    assert ncl == ncl_o and ncl > 0
    check_rows(q, k, 64, oracle.TOPP, 0.95, False, cap, idx, cnt, all_rows(q, 64))


def test_full_keep(gpu):
    q, k, _ = synth.planted_case(9, 1, 2, 1, 400, 64)
    idx, cnt, cap, _ = run(q, k, 64, oracle.TOPK, 1.0, True)
    for i in range(7):
        L = min(400, (i + 1) * 64)
        assert cnt[0, 0, i] == L and list(idx[0, 0, i, :L]) == list(range(L))


def test_selection_then_attention_end_to_end(gpu):
    q, k, v = synth.planted_case(10, 1, 4, 2, 640, 128)
    idx, cnt, cap, _ = run(q, k, 64, oracle.TOPK, 0.2, True)
    o = va.sparse_attn(dev(q), dev(k), dev(v), torch.from_numpy(idx).cuda(),
                       torch.from_numpy(cnt).cuda(), 64, True)
    torch.cuda.synchronize()
    o_ref, _ = oracle.sparse_attn(q, k, v, idx, cnt, 64, True)
    err = np.abs(o.float().cpu().numpy() - o_ref)
    assert err.max() <= 2e-2 and err.mean() <= 2e-3


@pytest.mark.parametrize("sampled_high", [False, True])
def test_level0_interval_from_misleading_sample(gpu, sampled_high):
    # The first interval of a topK row is estimated from every 16th 32-key
    # block.  Shifting only the unsampled blocks' keys (or only the sampled
    # ones) toward the queries' direction puts the true cut above (or below)
    # that estimate; the refinement must still find the exact set.
    rng = np.random.default_rng(11 + int(sampled_high))
    N, D, block = 8192, 128, 64
    u = rng.standard_normal(D).astype(np.float32)
    u /= np.linalg.norm(u)
    q = rng.standard_normal((1, 2, N, D)).astype(np.float32) + 2.0 * u
    k = rng.standard_normal((1, 2, N, D)).astype(np.float32)
    sampled = ((np.arange(N) // 32) % 16) == 0
    shifted = sampled if sampled_high else ~sampled
    k[:, :, shifted] += 3.0 * u
    qb, kb = synth.to_bf16_bits(q), synth.to_bf16_bits(k)
    idx, cnt, cap, _ = run(qb, kb, block, oracle.TOPK, 0.1, False)
    check_rows(qb, kb, block, oracle.TOPK, 0.1, False, cap, idx, cnt, all_rows(qb, block))


MINS_CASES = [
    # B, Hq, Hkv, N, D, block, causal, alpha
    (1, 2, 2, 700, 128, 64, False, 0.0),
    (1, 2, 2, 700, 128, 64, False, 0.5),
    (1, 4, 2, 1000, 128, 64, True, 1.0),
    (2, 2, 1, 513, 64, 32, False, 2.0),
    (1, 2, 2, 600, 64, 64, True, float("inf")),
    (1, 1, 1, 6000, 128, 64, False, 1.5),
]


@pytest.mark.parametrize("case", MINS_CASES)
def test_mins_matches_oracle(gpu, case):
    # Eq. 3: every eligible key within alpha (in units of the scaled score) of
    # the block's largest score.
    B, Hq, Hkv, N, D, block, causal, alpha = case
    q, k, _ = synth.planted_case(hash(case) % 10000 + 100, B, Hq, Hkv, N, D)
    cap = va.max_count(N, block, causal, "mins", alpha)
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cnt = va.select(dev(q), dev(k), block, "mins", alpha, causal, cap=cap, n_clamped=ncl)
    torch.cuda.synchronize()
    assert int(ncl.item()) == 0
    rows = all_rows(q, block)
    mism = check_rows(q, k, block, oracle.MINS, alpha, causal, cap, idx.cpu().numpy(),
                      cnt.cpu().numpy(), rows)
    assert mism <= max(1, len(rows) // 20)


def test_mins_clamped_to_cap(gpu):
    # A wide alpha selects more than cap keys: each such block keeps its cap
    # best (counted in n_clamped), the others their full minS set.
    q, k, _ = synth.planted_case(12, 1, 2, 2, 2000, 128)
    cap = 150
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cnt = va.select(dev(q), dev(k), 64, "mins", 3.0, False, cap=cap, n_clamped=ncl)
    torch.cuda.synchronize()
    _, cnt_o, ncl_o = oracle.select(q, k, 64, oracle.MINS, 3.0, False, cap)
    assert int(ncl.item()) == ncl_o and ncl_o > 0
    check_rows(q, k, 64, oracle.MINS, 3.0, False, cap, idx.cpu().numpy(), cnt.cpu().numpy(),
               all_rows(q, 64))


TILED_CASES = [
    # B, Hq, Hkv, N, D, block, causal, alpha, tile (B_K), group_tiles (G_K)
    (1, 2, 2, 700, 128, 64, False, 0.0, 16, 16),
    (1, 2, 2, 700, 128, 64, False, 0.3, 16, 1),       # every 16-key tile its own group
    (1, 4, 2, 1000, 128, 64, True, 0.5, 32, 4),
    (2, 2, 1, 513, 64, 32, False, 1.0, 16, 16),
    (1, 2, 2, 600, 64, 64, True, float("inf"), 16, 16),
    (1, 2, 2, 300, 128, 64, False, 0.2, 16, 16),       # groups inside one short split
    (1, 2, 2, 300, 128, 64, False, 0.2, 16, 32),       # a group longer than the split
    (1, 1, 1, 6000, 128, 64, False, 0.4, 16, 16),
    (1, 1, 1, 6000, 128, 64, True, 0.4, 16, 8192),     # one group per row, across splits
    (1, 1, 1, 9000, 64, 16, False, 0.6, 32, 256),      # 8192-key groups: a reset mid-row
]


@pytest.mark.parametrize("case", TILED_CASES)
def test_mins_tiled_matches_oracle(gpu, case):
    B, Hq, Hkv, N, D, block, causal, alpha, bk, gk = case
    q, k, _ = synth.planted_case(hash(case) % 10000 + 200, B, Hq, Hkv, N, D)
    cap = va.max_count(N, block, causal, "mins_tiled", alpha)
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cnt = va.select(dev(q), dev(k), block, "mins_tiled", alpha, causal, cap=cap,
                         n_clamped=ncl, tile=bk, group_tiles=gk)
    torch.cuda.synchronize()
    assert int(ncl.item()) == 0
    rows = all_rows(q, block)
    mism = check_rows_tiled(q, k, block, alpha, causal, bk, gk, idx.cpu().numpy(),
                            cnt.cpu().numpy(), rows)
    assert mism <= max(1, len(rows) // 20)


def test_mins_tiled_default_tiling_and_clamp(gpu):
    # mode "mins_tiled" without tiling arguments is B_K = G_K = 16; a block
    # selecting more than cap keys keeps its first cap keys and is counted.
    q, k, _ = synth.planted_case(14, 1, 2, 2, 2000, 128)
    full = va.max_count(2000, 64, False, "mins_tiled", 1.0)
    a_idx, a_cnt = va.select(dev(q), dev(k), 64, "mins_tiled", 1.0, False, cap=full)
    b_idx, b_cnt = va.select(dev(q), dev(k), 64, va.SEL_MINS_TILED, 1.0, False, cap=full,
                             tile=16, group_tiles=16)
    cap = 120
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    c_idx, c_cnt = va.select(dev(q), dev(k), 64, "mins_tiled", 1.0, False, cap=cap, n_clamped=ncl)
    torch.cuda.synchronize()
    assert torch.equal(a_idx, b_idx) and torch.equal(a_cnt, b_cnt)
    a_cnt, a_idx = a_cnt.cpu().numpy(), a_idx.cpu().numpy()
    c_cnt, c_idx = c_cnt.cpu().numpy(), c_idx.cpu().numpy()
    assert int(ncl.item()) == int(np.sum(a_cnt > cap)) > 0
    assert np.array_equal(c_cnt, np.minimum(a_cnt, cap))
    assert np.array_equal(c_idx, a_idx[..., :cap])
    check_rows_tiled(q, k, 64, 1.0, False, 16, 16, a_idx, a_cnt, all_rows(q, 64))


PER_HEAD = [
    ("topk", oracle.TOPK, [0.05, 0.1, 0.2, 0.4]),
    ("topp", oracle.TOPP, [0.5, 0.8, 0.9, 0.99]),
    ("mins", oracle.MINS, [0.0, 0.5, 1.0, 2.0]),
    ("mins_tiled", oracle.MINS_TILED, [0.1, 0.3, 0.6, 1.0]),
]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("name,omode,params", PER_HEAD)
def test_per_head_parameters(gpu, name, omode, params, causal):
    # One call with a parameter per query head equals, head by head, the
    # oracle's selection of that head with its own parameter.
    B, Hq, Hkv, N, D, block = 1, 4, 2, 700, 128, 64
    q, k, _ = synth.planted_case(300 + len(name) + int(causal), B, Hq, Hkv, N, D)
    cap = va.max_count(N, block, causal, name, params)
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cnt = va.select(dev(q), dev(k), block, name, params, causal, cap=cap, n_clamped=ncl)
    torch.cuda.synchronize()
    assert int(ncl.item()) == 0
    idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
    for h in range(Hq):
        qh = np.ascontiguousarray(q[:, h:h + 1])
        kh = np.ascontiguousarray(k[:, h // (Hq // Hkv):h // (Hq // Hkv) + 1])
        ih, ch = np.ascontiguousarray(idx[:, h:h + 1]), np.ascontiguousarray(cnt[:, h:h + 1])
        rows = all_rows(qh, block)
        if omode == oracle.MINS_TILED:
            mism = check_rows_tiled(qh, kh, block, params[h], causal, 16, 16, ih, ch, rows)
        else:
            mism = check_rows(qh, kh, block, omode, params[h], causal, cap, ih, ch, rows)
        assert mism <= max(1, len(rows) // 20), (name, h)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("name,param", [("topk", 0.1), ("topp", 0.8), ("mins", 0.5),
                                        ("mins_tiled", 0.3)])
def test_keep_diagonal(gpu, name, param, causal):
    # With the diagonal kept, every list is the selection united with the keys
    # of the block's own rows: against the oracle's selection united with them
    # (near-tie differences allowed only outside the block's rows), and
    # against the same call without the flag united with them (bit-exact: the
    # selection is deterministic).
    B, Hq, Hkv, N, D, block = 1, 2, 2, 777, 128, 64
    q, k, _ = synth.planted_case(400 + len(name) + int(causal), B, Hq, Hkv, N, D)
    cap = va.max_count(N, block, causal, name, param, keep_diag=True)
    a_idx, a_cnt = va.select(dev(q), dev(k), block, name, param, causal, cap=cap, keep_diag=True)
    b_idx, b_cnt = va.select(dev(q), dev(k), block, name, param, causal, cap=cap)
    torch.cuda.synchronize()
    a_idx, a_cnt = a_idx.cpu().numpy(), a_cnt.cpu().numpy()
    omode = {"topk": oracle.TOPK, "topp": oracle.TOPP, "mins": oracle.MINS,
             "mins_tiled": oracle.MINS_TILED}[name]
    rows = all_rows(q, block)
    mism = check_rows_keep_diag(q, k, block, omode, param, causal, cap, a_idx, a_cnt, rows)
    assert mism <= max(1, len(rows) // 20)
    want_idx, want_cnt = oracle.with_diagonal(b_idx.cpu().numpy(), b_cnt.cpu().numpy(), N, block,
                                              cap)
    assert np.array_equal(a_cnt, want_cnt)
    assert np.array_equal(a_idx, want_idx)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("mode,param", [("topk", 0.2), ("topp", 0.9), ("mins", 0.5)])
def test_varlen_batch(gpu, causal, mode, param):
    # Packed sequences (one empty) in one call: each sequence's lists against
    # the oracle's selection on that sequence's rows, and equal to a separate
    # call on those rows; attention on the packed lists matches the oracle.
    lens = [300, 0, 777, 64, 129]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    Hq, Hkv, D, block = 4, 2, 128, 64
    q, k, v = synth.planted_case(500 + int(causal), 1, Hq, Hkv, int(cu[-1]), D)
    tq, tk, tv = dev(q), dev(k), dev(v)
    cap = max(va.max_count(n, block, causal, mode, param) for n in lens if n)
    idx, cnt = va.select_varlen(tq, tk, cu, block, mode, param, causal, cap=cap)
    out, lse = va.sparse_attn_varlen(tq, tk, tv, cu, idx, cnt, cap, block, causal, return_lse=True)
    torch.cuda.synchronize()
    nb, first, total = va.varlen_blocks(cu, block)
    idx = idx.view(-1).cpu().numpy()
    cnt = cnt.view(-1).cpu().numpy()
    for s, n in enumerate(lens):
        if n == 0:
            continue
        r0, r1 = int(cu[s]), int(cu[s + 1])
        i_s, c_s = va.select(tq[:, :, r0:r1], tk[:, :, r0:r1], block, mode, param, causal, cap=cap)
        torch.cuda.synchronize()
        got_i = idx[first[s] * Hq * cap:(first[s] + nb[s]) * Hq * cap].reshape(1, Hq, nb[s], cap)
        got_c = cnt[first[s] * Hq:(first[s] + nb[s]) * Hq].reshape(1, Hq, nb[s])
        qs, ks, vs = (np.ascontiguousarray(a[:, :, r0:r1]) for a in (q, k, v))
        omode = {"topk": oracle.TOPK, "topp": oracle.TOPP, "mins": oracle.MINS}[mode]
        mism = check_rows(qs, ks, block, omode, param, causal, cap, got_i, got_c, all_rows(qs, block))
        assert mism <= max(1, Hq * nb[s] // 20), s
        assert np.array_equal(got_i, i_s.cpu().numpy()) and np.array_equal(got_c, c_s.cpu().numpy())
        o_ref, lse_ref = oracle.sparse_attn(qs, ks, vs, got_i, got_c, block, causal)
        o = out[:, :, r0:r1].float().cpu().numpy()
        err = np.abs(o - o_ref)
        assert err.max() <= 2e-2 and err.mean() <= 2e-3, (s, err.max())
        l = lse[Hq * r0:Hq * r1].view(1, Hq, n).cpu().numpy()
        ok = np.isfinite(lse_ref)
        assert np.array_equal(np.isfinite(l), ok)
        assert np.abs(l[ok] - lse_ref[ok]).max() <= 1e-4  # fp32 normaliser (see test_attn_gpu)


@pytest.mark.parametrize("mode,param", [("topk", 0.1), ("topp", 0.9), ("mins", 0.7)])
def test_list_writer_alignment_paths(gpu, mode, param):
    # Lists of rows that start on 16 bytes are stored four entries at a time,
    # others one at a time: both give the same lists and -1 padding.
    q, k, _ = synth.planted_case(600 + len(mode), 1, 3, 3, 1337, 128)
    need = va.max_count(1337, 64, True, mode, param)
    caps = [need + (-need) % 4, need + (-need) % 4 + 1]       # a multiple of 4, and not
    res = []
    for cap in caps:
        idx, cnt = va.select(dev(q), dev(k), 64, mode, param, True, cap=cap)
        torch.cuda.synchronize()
        res.append((idx.cpu().numpy(), cnt.cpu().numpy()))
    (i0, c0), (i1, c1) = res
    assert np.array_equal(c0, c1)
    assert np.array_equal(i0, i1[..., :caps[0]]) and np.all(i1[..., caps[0]:] == -1)
    check_rows(q, k, 64, {"topk": oracle.TOPK, "topp": oracle.TOPP, "mins": oracle.MINS}[mode],
               param, True, caps[0], i0, c0, all_rows(q, 64))


@pytest.mark.parametrize("mode,param", [("topk", 0.15), ("topp", 0.9), ("mins", 0.5),
                                        ("mins_tiled", 0.3)])
def test_selection_is_deterministic(gpu, mode, param):
    # Two identical calls give bit-identical lists and counts (the scores,
    # histograms and candidate ranks do not depend on scheduling).
    q, k, _ = synth.planted_case(700 + len(mode), 1, 4, 2, 5000, 128)
    tq, tk = dev(q), dev(k)
    cap = va.max_count(5000, 64, False, mode, param)
    ws = torch.empty(va.workspace_bytes(tq, tk, 64, False, mode, cap), dtype=torch.uint8,
                     device="cuda")
    runs = []
    for _ in range(3):
        idx, cnt = va.select(tq, tk, 64, mode, param, False, cap=cap, workspace=ws)
        torch.cuda.synchronize()
        runs.append((idx.cpu().numpy(), cnt.cpu().numpy()))
    for idx, cnt in runs[1:]:
        assert np.array_equal(idx, runs[0][0]) and np.array_equal(cnt, runs[0][1])


def test_topp_mass_beyond_fp32_exponent_range(gpu):
    # Scores spread over ~100 nats: the softmax weights of the low keys are
    # below fp32's range (exp(-100) ~ 4e-44), so their topP masses take the
    # exact power-of-two rescale branch; the lists still follow the rule.
    N, block, D = 3000, 64, 128
    q, k, _ = synth.planted_case(750, 1, 2, 2, N, D, frac=0.05, logits=3.0)
    kf = synth.bits_to_f32(k)
    r = np.random.Generator(np.random.PCG64(751))
    kf *= np.float32(12.0)                               # widen every score ~12x
    kf[0, :, r.choice(N, 40, replace=False)] *= np.float32(3.0)
    k = synth.to_bf16_bits(kf)
    spread = []
    for h in range(2):
        s = oracle.pooled_scores(q, k, block, False, 0, h, 3)
        spread.append(s.max() - s.min())
    assert min(spread) > 90.0, spread
    for p in (0.5, 0.99, 0.999999):
        idx, cnt, cap, _ = run(q, k, block, oracle.TOPP, p, False)
        check_rows(q, k, block, oracle.TOPP, p, False, cap, idx, cnt, all_rows(q, block))


@pytest.mark.parametrize("mode,param", [("topk", 0.2), ("topp", 0.9), ("mins", 0.5),
                                        ("mins_tiled", 0.3)])
def test_unpadded_lists(gpu, mode, param):
    # VECATTN_UNPADDED: the first C entries of each list are those of the padded
    # call, the entries past C keep what the caller left there.
    q, k, _ = synth.planted_case(770 + len(mode), 1, 3, 3, 1500, 128)
    tq, tk = dev(q), dev(k)
    cap = va.max_count(1500, 64, True, mode, param)
    a_idx, a_cnt = va.select(tq, tk, 64, mode, param, True, cap=cap)
    Np = (1500 + 63) // 64
    b_idx = torch.full((1, 3, Np, cap), 0x7FFF7FFF, dtype=torch.int32, device="cuda")
    b_cnt = torch.empty((1, 3, Np), dtype=torch.int32, device="cuda")
    va.select(tq, tk, 64, mode, param, True, cap=cap, idx=b_idx, counts=b_cnt, unpadded=True)
    torch.cuda.synchronize()
    assert torch.equal(a_cnt, b_cnt)
    live = torch.arange(cap, device="cuda").view(1, 1, 1, -1) < a_cnt.unsqueeze(-1)
    assert torch.equal(torch.where(live, a_idx, 0), torch.where(live, b_idx, 0))
    assert bool((b_idx[~live] == 0x7FFF7FFF).all())
    assert va.check_lists(b_idx, b_cnt, 1500) == 0
