"""GPU parity of query pooling (Eq. 2) and vector-sparse attention (Eq. 4,
Algorithm 2) against the CPU oracle, called through the C ABI.

Tolerances: pooling is bit-exact (both sides round the exact block mean to
bf16 once); attention output within max-abs 2e-2 and mean-abs 2e-3 of the fp64
oracle on identical indices, LSE within 1e-4 absolute, empty rows exactly 0.
The LSE bound follows from the arithmetic: the kernel's normaliser is the fp32
sum of the fp32 softmax weights (each exp2 within a few ulp), a tree of four adds
per lane and tile and one add per tile, so for T tiles log of the sum is within
about (T + 8) 2^-23 of the exact one (under 3e-6 for the <= 16 tiles of these
lists), plus the fp32 rounding of the scaled maximum (|m| <= 100: 4e-6).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2603_29494_amd as va
from paper_2603_29494_amd import synth

pytestmark = pytest.mark.gpu

ATOL_MAX, ATOL_MEAN, LSE_TOL = 2e-2, 2e-3, 1e-4


def dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def random_lists(seed, B, H, Np, N, P, causal, max_count, cap, min_count=0):
    r = np.random.Generator(np.random.PCG64(seed))
    idx = np.full((B, H, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, H, Np), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            for i in range(Np):
                L = min(N, (i + 1) * P) if causal else N
                c = int(r.integers(min(min_count, L), min(max_count, L) + 1))
                idx[b, h, i, :c] = np.sort(r.choice(L, size=c, replace=False))
                cnt[b, h, i] = c
    return idx, cnt


def check_attn(o_gpu, lse_gpu, o_ref, lse_ref, label=""):
    o = o_gpu.float().cpu().numpy().astype(np.float64)
    err = np.abs(o - o_ref)
    assert np.isfinite(o).all(), label
    assert err.max() <= ATOL_MAX, f"{label} max abs err {err.max()}"
    assert err.mean() <= ATOL_MEAN, f"{label} mean abs err {err.mean()}"
    lg = lse_gpu.cpu().numpy().astype(np.float64)
    empty = np.isneginf(lse_ref)
    assert np.array_equal(np.isneginf(lg), empty), label
    if empty.any():
        assert np.all(o[empty] == 0.0), label
    if (~empty).any():
        assert np.abs(lg[~empty] - lse_ref[~empty]).max() <= LSE_TOL, label


@pytest.mark.parametrize("N,P,D", [(200, 64, 128), (77, 1, 64), (130, 128, 64), (64, 48, 128)])
def test_pool_bit_exact(gpu, N, P, D):
    q = synth.random_bits(1000 + N, (2, 3, N, D), scale=2.0)
    got = host_bits(va.pool(dev(q), P))
    assert np.array_equal(got, oracle.pool(q, P))


def test_pool_strided_input(gpu):
    q = synth.random_bits(7, (1, 100, 4, 64))        # [B, N, H, D] storage
    tq = dev(q).permute(0, 2, 1, 3)                    # logical [B, H, N, D]
    ref = oracle.pool(np.ascontiguousarray(q.transpose(0, 2, 1, 3)), 16)
    assert np.array_equal(host_bits(va.pool(tq, 16)), ref)


CASES = [
    # B, Hq, Hkv, N, D, P, causal, max_count, cap
    (1, 2, 2, 300, 128, 64, False, 200, 200),
    (1, 4, 2, 333, 128, 64, True, 333, 333),
    (2, 2, 1, 257, 64, 64, False, 257, 260),
    (1, 3, 3, 400, 64, 16, True, 150, 150),
    (1, 2, 1, 500, 128, 128, False, 300, 320),
    (1, 2, 2, 190, 128, 48, True, 190, 190),
    # 128-row workgroups (8 waves): causal with D = 64, and two per 256-row block
    (1, 2, 2, 300, 64, 128, True, 300, 300),
    (1, 2, 1, 600, 128, 256, True, 600, 600),
    # 12 heads over the XCD groups: whole heads per group and heads shared by all
    (3, 4, 2, 200, 64, 64, False, 150, 150),
    (3, 4, 1, 264, 128, 64, True, 264, 264),
]


@pytest.mark.parametrize("case", CASES)
def test_sparse_attn_matches_oracle(gpu, case):
    B, Hq, Hkv, N, D, P, causal, mx, cap = case
    seed = hash(case) % 10000
    q = synth.random_bits(seed + 1, (B, Hq, N, D))
    k = synth.random_bits(seed + 2, (B, Hkv, N, D))
    v = synth.random_bits(seed + 3, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    idx, cnt = random_lists(seed + 4, B, Hq, Np, N, P, causal, mx, cap)
    cnt[0, 0, 0] = 0                                  # an empty block
    idx[0, 0, 0, :] = -1
    o_ref, lse_ref = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
    o, lse = va.sparse_attn(dev(q), dev(k), dev(v), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(cnt).cuda(), P, causal, return_lse=True)
    torch.cuda.synchronize()
    check_attn(o, lse, o_ref, lse_ref, str(case))


@pytest.mark.parametrize("causal", [False, True])
def test_full_keep_equals_dense(gpu, causal):
    B, Hq, Hkv, N, D, P = 1, 4, 1, 320, 128, 64
    q, k, v = (synth.random_bits(s, (B, h, N, D)) for s, h in ((11, Hq), (12, Hkv), (13, Hkv)))
    Np = N // P
    idx = np.full((B, Hq, Np, N), -1, dtype=np.int32)
    cnt = np.zeros((B, Hq, Np), dtype=np.int32)
    for i in range(Np):
        L = (i + 1) * P if causal else N
        idx[:, :, i, :L] = np.arange(L)
        cnt[:, :, i] = L
    o_ref, lse_ref = oracle.dense_attn(q, k, v, causal)
    o, lse = va.sparse_attn(dev(q), dev(k), dev(v), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(cnt).cuda(), P, causal, return_lse=True)
    torch.cuda.synchronize()
    check_attn(o, lse, o_ref, lse_ref, f"dense causal={causal}")


def test_causal_rows_without_visible_keys(gpu):
    B, H, N, D, P = 1, 1, 128, 64, 64
    q, k, v = (synth.random_bits(s, (B, H, N, D)) for s in (21, 22, 23))
    idx = np.full((1, 1, 2, 8), -1, dtype=np.int32)
    idx[0, 0, 0, :3] = [40, 50, 63]
    idx[0, 0, 1, :2] = [0, 127]
    cnt = np.array([[[3, 2]]], dtype=np.int32)
    o_ref, lse_ref = oracle.sparse_attn(q, k, v, idx, cnt, P, True)
    o, lse = va.sparse_attn(dev(q), dev(k), dev(v), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(cnt).cuda(), P, True, return_lse=True)
    torch.cuda.synchronize()
    assert torch.all(o[0, 0, :40] == 0)
    check_attn(o, lse, o_ref, lse_ref, "empty rows")


def test_strided_q_and_out(gpu):
    B, Hq, Hkv, N, D, P = 1, 4, 2, 256, 128, 64
    q = synth.random_bits(31, (B, N, Hq, D))
    k = synth.random_bits(32, (B, Hkv, N, D))
    v = synth.random_bits(33, (B, Hkv, N, D))
    qc = np.ascontiguousarray(q.transpose(0, 2, 1, 3))
    Np = N // P
    idx, cnt = random_lists(34, B, Hq, Np, N, P, False, 200, 200, min_count=1)
    o_ref, _ = oracle.sparse_attn(qc, k, v, idx, cnt, P, False)
    tq = dev(q).permute(0, 2, 1, 3)
    out = torch.empty((B, N, Hq, D), dtype=torch.bfloat16, device="cuda").permute(0, 2, 1, 3)
    va.sparse_attn(tq, dev(k), dev(v), torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(),
                   P, False, out=out)
    torch.cuda.synchronize()
    err = np.abs(out.float().cpu().numpy() - o_ref)
    assert err.max() <= ATOL_MAX and err.mean() <= ATOL_MEAN


def test_plumbing_workload_with_oracle_indices(gpu):
    layer = synth.make_layer(1)
    w = layer.w
    idx, cnt, _ = oracle.select(layer.q, layer.k, w.block, oracle.TOPK, w.param, w.causal, 128)
    o_ref, lse_ref = oracle.sparse_attn(layer.q, layer.k, layer.v, idx, cnt, w.block, w.causal)
    o, lse = va.sparse_attn(dev(layer.q), dev(layer.k), dev(layer.v), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(cnt).cuda(), w.block, w.causal, return_lse=True)
    torch.cuda.synchronize()
    check_attn(o, lse, o_ref, lse_ref, "plumbing_1k")


@pytest.mark.parametrize("D", [64, 128])
def test_k_and_v_with_different_row_strides(gpu, D):
    # V stored [B, N, Hkv, D] (row stride Hkv * D) and K [B, Hkv, N, D]: the
    # gathers then need separate K and V offsets.
    B, Hq, Hkv, N, P = 1, 4, 2, 300, 64
    q = synth.random_bits(41, (B, Hq, N, D))
    k = synth.random_bits(42, (B, Hkv, N, D))
    v = synth.random_bits(43, (B, N, Hkv, D))
    vc = np.ascontiguousarray(v.transpose(0, 2, 1, 3))
    Np = (N + P - 1) // P
    idx, cnt = random_lists(44, B, Hq, Np, N, P, True, N, N, min_count=1)
    o_ref, lse_ref = oracle.sparse_attn(q, k, vc, idx, cnt, P, True)
    o, lse = va.sparse_attn(dev(q), dev(k), dev(v).permute(0, 2, 1, 3),
                            torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), P, True,
                            return_lse=True)
    torch.cuda.synchronize()
    check_attn(o, lse, o_ref, lse_ref, f"kv strides D={D}")


def sparse_lists(seed, B, H, Np, N, P, causal, max_count):
    """Short random ascending lists (1 .. max_count keys per block) for long
    sequences, drawn without a pass over all N keys per block."""
    r = np.random.Generator(np.random.PCG64(seed))
    idx = np.full((B * H * Np, max_count), -1, dtype=np.int32)
    cnt = np.zeros(B * H * Np, dtype=np.int32)
    for row in range(B * H * Np):
        i = row % Np
        L = min(N, (i + 1) * P) if causal else N
        want = int(r.integers(1, min(max_count, L) + 1))
        uniq = np.unique(r.integers(0, L, size=2 * want + 8))
        keys = np.sort(r.choice(uniq, size=min(want, uniq.size), replace=False))
        idx[row, :keys.size] = keys
        cnt[row] = keys.size
    return idx.reshape(B, H, Np, max_count), cnt.reshape(B, H, Np)


# Long sequences whose K/V sizes make the kernel deal blocks to groups of 2, 4
# and 8 XCDs (K and V rows of one KV head: N * D * 4 bytes, half when causal;
# the group is the smallest whose concurrently swept heads fit ~160 MB):
# 30.7 MB x 8 heads -> 2, with two 64-row chunks per 128-row block; the same
# causal; 46 MB x 8 (B = 2) -> 4; one 205 MB KV head shared by 2 query heads -> 8.
XCD_CASES = [(1, 8, 8, 60000, 128, False), (1, 8, 8, 120000, 64, True),
             (2, 4, 4, 90000, 64, False), (1, 2, 1, 400000, 64, False)]


@pytest.mark.parametrize("case", XCD_CASES, ids=["g2_chunked", "g2_causal", "g4_batch2", "g8_gqa"])
def test_long_sequences_sampled(gpu, case):
    B, Hq, Hkv, N, P, causal = case
    D = 128
    print(f"long sequence {case}", flush=True)
    q = synth.random_bits(61, (B, Hq, N, D))
    k = synth.random_bits(62, (B, Hkv, N, D))
    v = synth.random_bits(63, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    idx, cnt = sparse_lists(64, B, Hq, Np, N, P, causal, 96)
    o, lse = va.sparse_attn(dev(q), dev(k), dev(v), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(cnt).cuda(), P, causal, return_lse=True)
    torch.cuda.synchronize()
    # Causal rows can see no listed key: O = 0 and LSE = -inf there, finite elsewhere.
    assert bool(torch.isfinite(o.float()).all())
    assert bool((torch.isfinite(lse) | torch.isneginf(lse)).all())
    rng = np.random.Generator(np.random.PCG64(65))
    total = B * Hq * Np
    rows = np.unique(np.concatenate([[0, Np - 1, total - 1],
                                     rng.choice(total, size=9, replace=False)]))
    flat_i, flat_c = idx.reshape(total, -1), cnt.reshape(total)
    o_ref, lse_ref = oracle.sparse_attn(q, k, v, flat_i[rows], flat_c[rows], P, causal,
                                        blocks=rows, compact=True, nthreads=8)
    for t, r in enumerate(rows):
        i, h, b = r % Np, (r // Np) % Hq, r // (Np * Hq)
        n = min(N, (i + 1) * P) - i * P
        got = o[b, h, i * P:i * P + n].float().cpu().numpy().astype(np.float64)
        err = np.abs(got - o_ref[t, :n])
        assert err.max() <= ATOL_MAX and err.mean() <= ATOL_MEAN, (case, int(r), err.max())
        lg = lse[b, h, i * P:i * P + n].cpu().numpy().astype(np.float64)
        empty = np.isneginf(lse_ref[t, :n])
        assert np.array_equal(np.isneginf(lg), empty) and np.all(got[empty] == 0.0), (case, int(r))
        if (~empty).any():
            assert np.abs(lg[~empty] - lse_ref[t, :n][~empty]).max() <= LSE_TOL, (case, int(r))


@pytest.mark.parametrize("causal", [False, True])
def test_extreme_logits_move_the_softmax_reference(gpu, causal):
    # Scores with a spread of tens of nats, the largest keys toward the end of
    # every (ascending) list: tiles keep bringing maxima far above the running
    # reference (weights beyond 2^8), so the kernel must move its reference,
    # rescale O and the normaliser and recompute the weights, over and over.
    B, Hq, Hkv, N, D, P = 1, 2, 1, 1200, 128, 64
    q = synth.random_bits(91, (B, Hq, N, D), scale=6.0)
    kf = synth.bits_to_f32(synth.random_bits(92, (B, Hkv, N, D), scale=5.0))
    kf *= np.linspace(0.3, 1.5, N, dtype=np.float32).reshape(1, 1, N, 1)   # later keys larger
    k = synth.to_bf16_bits(kf)
    v = synth.random_bits(93, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    idx, cnt = random_lists(94, B, Hq, Np, N, P, causal, 900, 900, min_count=1)
    o_ref, lse_ref = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
    fin = np.isfinite(lse_ref)
    qf, kk = oracle.bf16_to_f64(q), oracle.bf16_to_f64(k)
    s = (qf[0, 0, :64] @ kk[0, 0].T) / math.sqrt(D)
    assert s.max() - s.min() > 150.0                   # tens of log2 units between tiles
    o, lse = va.sparse_attn(dev(q), dev(k), dev(v), torch.from_numpy(idx).cuda(),
                            torch.from_numpy(cnt).cuda(), P, causal, return_lse=True)
    torch.cuda.synchronize()
    check_attn(o, lse, o_ref, lse_ref, f"extreme logits causal={causal}")
    assert np.abs(lse_ref[fin]).max() > 100.0


def test_causal_attention_is_deterministic(gpu):
    """Causal lists are walked from their first tile, so the summation order and
    O are the same on every call (with and without a block order)."""
    B, Hq, Hkv, N, D, P = 1, 4, 2, 700, 128, 64
    q, k, v = (dev(synth.random_bits(900 + j, (B, h, N, D))) for j, h in enumerate((Hq, Hkv, Hkv)))
    Np = (N + P - 1) // P
    idx, cnt = random_lists(77, B, Hq, Np, N, P, True, N, N)
    ti, tc = torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda()
    order = va.attn_order(ti, tc, N, P)
    first, lse1 = va.sparse_attn(q, k, v, ti, tc, P, True, return_lse=True)
    for o in (None, order, None):
        again, lse2 = va.sparse_attn(q, k, v, ti, tc, P, True, return_lse=True, order=o)
        assert torch.equal(again.view(torch.int16), first.view(torch.int16))
        assert torch.equal(lse1, lse2)
