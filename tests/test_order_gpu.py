"""Block order for the sparse attention (vecattn_attn_order) and the attention
taken in that order (vecattn_sparse_attn_ordered), through the C ABI.

The order is integer work, compared bit for bit with its definition written
out in numpy (count descending, then the sampled mean key, then the block
index).  The ordered attention must meet the attention bar of test_attn_gpu
(max-abs 2e-2, mean-abs 2e-3 and LSE 1e-4 against the fp64 oracle) whatever
the order, since Eq. 4 treats the query blocks independently."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_29494_amd as va
from paper_2603_29494_amd import synth

pytestmark = pytest.mark.gpu

ATOL_MAX, ATOL_MEAN, LSE_TOL = 2e-2, 2e-3, 1e-4


def lists(seed, B, H, Np, N, P, causal, counts_from, cap):
    """Random ascending lists; counts_from(r, L) draws a block's count."""
    r = np.random.Generator(np.random.PCG64(seed))
    idx = np.full((B, H, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, H, Np), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            for i in range(Np):
                L = min(N, (i + 1) * P) if causal else N
                c = min(int(counts_from(r, L)), L, cap)
                idx[b, h, i, :c] = np.sort(r.choice(L, size=c, replace=False))
                cnt[b, h, i] = c
    return idx, cnt


def order_ref(idx, cnt, N, cap):
    """The documented order, written out: per (b, h), sort by
    (2^30 - C) << 33 | sig << 24 | i, with sig = min(511, floor(64 * sum / N))
    over the entries at floor((2j + 1) C / 16), j < 8."""
    B, H, Np = cnt.shape
    out = np.empty((B, H, Np), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            for s0 in range(0, Np, 16384):  # heads of more blocks: segment by segment
                keys = []
                for i in range(s0, min(Np, s0 + 16384)):
                    c = min(max(int(cnt[b, h, i]), 0), cap)
                    s = 0
                    if c > 0:
                        for j in range(8):
                            e = int(idx[b, h, i, ((2 * j + 1) * c) // 16])
                            s += min(max(e, 0), N - 1)
                    sig = min((s * 64) // N, 511)
                    keys.append(((2 ** 30 - c) << 33) | (sig << 24) | (i - s0))
                seg = np.argsort(np.array(keys, dtype=np.uint64), kind="stable")
                out[b, h, s0:s0 + len(seg)] = s0 + seg
    return out


def cuda_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("N,P,cap,kind", [
    (1000, 16, 200, "varied"),     # 63 blocks: not a power of two
    (1000, 16, 40, "equal"),       # every count equal: the signature and index decide
    (64, 64, 64, "varied"),        # one block
    (5000, 8, 16, "tied"),         # 625 blocks, counts from {0, 8, 16}: many full ties
])
def test_order_matches_definition(gpu, N, P, cap, kind):
    Np = (N + P - 1) // P
    draw = {"varied": lambda r, L: r.integers(0, cap + 1),
            "equal": lambda r, L: cap,
            "tied": lambda r, L: 8 * r.integers(0, 3)}[kind]
    idx, cnt = lists(11 + N + cap, 2, 3, Np, N, P, False, draw, cap)
    got = va.attn_order(cuda_i32(idx), cuda_i32(cnt), N, P).cpu().numpy()
    assert np.array_equal(got, order_ref(idx, cnt, N, cap))


@pytest.mark.parametrize("Np", [16384, 16385, 40000])
def test_order_segments(gpu, Np):
    """Up to 16384 blocks per head are sorted at once; longer heads segment by
    segment (a one-block tail, and two whole segments and a partial one)."""
    r = np.random.Generator(np.random.PCG64(Np))
    N, P, cap = Np, 1, 2
    cnt = r.integers(0, 3, size=(1, 1, Np)).astype(np.int32)
    idx = np.sort(r.integers(0, N, size=(1, 1, Np, cap)), axis=-1).astype(np.int32)
    idx = np.where(np.arange(cap)[None, None, None, :] < cnt[..., None], idx, -1).astype(np.int32)
    got = va.attn_order(cuda_i32(idx), cuda_i32(cnt), N, P).cpu().numpy()
    assert np.array_equal(got, order_ref(idx, cnt, N, cap))
    for s0 in range(0, Np, 16384):  # each segment a permutation of its own blocks
        seg = got[0, 0, s0:s0 + 16384]
        assert np.array_equal(np.sort(seg), np.arange(s0, s0 + len(seg)))


def check_attn(o_gpu, lse_gpu, o_ref, lse_ref, label):
    o = o_gpu.float().cpu().numpy().astype(np.float64)
    err = np.abs(o - o_ref)
    assert np.isfinite(o).all(), label
    assert err.max() <= ATOL_MAX and err.mean() <= ATOL_MEAN, (label, err.max(), err.mean())
    lg = lse_gpu.cpu().numpy().astype(np.float64)
    empty = np.isneginf(lse_ref)
    assert np.array_equal(np.isneginf(lg), empty), label
    if (~empty).any():
        assert np.abs(lg[~empty] - lse_ref[~empty]).max() <= LSE_TOL, label


@pytest.mark.parametrize("B,Hq,Hkv,N,D,P,causal", [
    (1, 4, 2, 600, 128, 64, True),     # GQA, causal, ragged last block
    (2, 2, 2, 520, 64, 128, False),    # 128-row blocks (8-wave workgroups), ragged
])
def test_ordered_attention_parity(gpu, B, Hq, Hkv, N, D, P, causal):
    q = synth.random_bits(100 + N, (B, Hq, N, D))
    k = synth.random_bits(200 + N, (B, Hkv, N, D))
    v = synth.random_bits(300 + N, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    cap = N
    # counts spread from empty to every eligible key, as topP lists are
    idx, cnt = lists(400 + N, B, Hq, Np, N, P, causal, lambda r, L: r.integers(0, L + 1), cap)
    o_ref, lse_ref = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
    tq, tk, tv = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda() for x in (q, k, v))
    ti, tc = cuda_i32(idx), cuda_i32(cnt)
    order = va.attn_order(ti, tc, N, P)
    assert np.array_equal(order.cpu().numpy(), order_ref(idx, cnt, N, cap))
    for name, o in (("attn_order", order), ("reversed", torch.flip(order, dims=[-1]).contiguous()),
                    ("ascending", torch.arange(Np, dtype=torch.int32, device="cuda")
                     .expand(B, Hq, Np).contiguous())):
        out, lse = va.sparse_attn(tq, tk, tv, ti, tc, P, causal, return_lse=True, order=o)
        check_attn(out, lse, o_ref, lse_ref, name)


def test_order_not_a_permutation(gpu):
    """Entries are clamped to [0, N_p); blocks an order row misses are left
    unwritten, blocks it repeats are computed again (same result)."""
    B, Hq, Hkv, N, D, P, causal = 1, 2, 1, 300, 64, 64, False
    q = synth.random_bits(31, (B, Hq, N, D))
    k = synth.random_bits(32, (B, Hkv, N, D))
    v = synth.random_bits(33, (B, Hkv, N, D))
    Np = (N + P - 1) // P  # 5, the last block 44 rows
    cap = N
    idx, cnt = lists(34, B, Hq, Np, N, P, causal, lambda r, L: r.integers(1, L + 1), cap)
    o_ref, _ = oracle.sparse_attn(q, k, v, idx, cnt, P, causal)
    tq, tk, tv = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda() for x in (q, k, v))
    rows = np.array([[0, 0, 7, -1, 2],   # clamped: 0, 0, 4, 0, 2 -> blocks 1 and 3 missed
                     [3, 1, 3, 1, 3]])   # blocks 0, 2 and 4 missed
    order = cuda_i32(rows.reshape(B, Hq, Np).astype(np.int32))
    sentinel = 123.0
    out = torch.full((B, Hq, N, D), sentinel, dtype=torch.bfloat16, device="cuda")
    va.sparse_attn(tq, tk, tv, cuda_i32(idx), cuda_i32(cnt), P, causal, out=out, order=order)
    o = out.float().cpu().numpy().astype(np.float64)
    for h, taken in ((0, {0, 2, 4}), (1, {1, 3})):
        for i in range(Np):
            r0, r1 = i * P, min(N, (i + 1) * P)
            blk = o[0, h, r0:r1]
            if i in taken:
                assert np.abs(blk - o_ref[0, h, r0:r1]).max() <= ATOL_MAX, (h, i)
            else:
                assert (blk == sentinel).all(), (h, i)
