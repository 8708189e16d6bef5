"""GPU parity of the selection statistics against the oracle, through the C ABI:
the recall of a selected pattern (the attention mass its lists keep, Sec. 2.2)
and Eq. 5's per-head sparsity sp_h (Sec. 3.1.2).

Recall tolerance: the kernel scores in fp32 from exact bf16 products and sums
the softmax weights in fp32 (each lane over ~N/4 keys, then 4 partial sums).
A score error of a few 1e-6 relative moves a weight by about that much, and a
sequential fp32 sum of n terms is within n * 2^-24 relative; for the rows here
(n <= ~1300 per lane) that bounds |kept_gpu - kept_oracle| by ~1e-4, so max-abs
2e-4 and mean-abs 2e-5 are the bars.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_29494_amd as va
from paper_2603_29494_amd import synth

pytestmark = pytest.mark.gpu

KEPT_MAX, KEPT_MEAN = 2e-4, 2e-5


def dev(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def random_lists(seed, B, H, Np, N, P, causal, max_count, cap):
    r = np.random.Generator(np.random.PCG64(seed))
    idx = np.full((B, H, Np, cap), -1, dtype=np.int32)
    cnt = np.zeros((B, H, Np), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            for i in range(Np):
                L = min(N, (i + 1) * P) if causal else N
                c = int(r.integers(0, min(max_count, L) + 1))
                idx[b, h, i, :c] = np.sort(r.choice(L, size=c, replace=False))
                cnt[b, h, i] = c
    return idx, cnt


RECALL_CASES = [
    # B, Hq, Hkv, N, D, P, causal
    (1, 2, 2, 300, 128, 64, False),
    (1, 4, 2, 333, 128, 64, True),
    (2, 2, 1, 257, 64, 64, False),
    (1, 3, 3, 400, 64, 16, True),
    (1, 2, 1, 500, 128, 128, False),      # two 64-row chunks per block
    (1, 2, 2, 190, 128, 48, True),
    (1, 1, 1, 5000, 128, 64, False),
]


@pytest.mark.parametrize("case", RECALL_CASES)
def test_recall_matches_oracle(gpu, case):
    B, Hq, Hkv, N, D, P, causal = case
    seed = sum(case) + 17 * int(causal)
    q = synth.random_bits(seed + 1, (B, Hq, N, D), scale=2.0)
    k = synth.random_bits(seed + 2, (B, Hkv, N, D))
    Np = (N + P - 1) // P
    idx, cnt = random_lists(seed + 3, B, Hq, Np, N, P, causal, N // 3, N // 3 + 5)
    cnt[0, 0, 0] = 0                    # an empty list keeps nothing
    idx[0, 0, 0, :] = -1
    ref = oracle.kept_mass(q, k, idx, cnt, P, causal)
    got = va.recall(dev(q), dev(k), torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), P,
                    causal).cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    assert np.isfinite(got).all()
    assert err.max() <= KEPT_MAX and err.mean() <= KEPT_MEAN, (case, err.max(), err.mean())
    assert np.all(got[0, 0, :min(N, P)] == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_recall_of_full_and_planted_selection(gpu, causal):
    # Every eligible key listed keeps the whole row (1 up to fp32 rounding);
    # the GPU's own topK lists on a planted layer keep what the oracle says
    # they keep, and more than their share of the keys.
    B, Hq, Hkv, N, D, P = 1, 2, 1, 640, 128, 64
    q, k, _ = synth.planted_case(33 + int(causal), B, Hq, Hkv, N, D)
    Np = N // P
    idx = np.full((B, Hq, Np, N), -1, dtype=np.int32)
    cnt = np.zeros((B, Hq, Np), dtype=np.int32)
    for i in range(Np):
        L = (i + 1) * P if causal else N
        idx[:, :, i, :L] = np.arange(L)
        cnt[:, :, i] = L
    full = va.recall(dev(q), dev(k), torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda(), P,
                     causal)
    assert float((full - 1.0).abs().max()) <= 1e-5
    ti, tc = va.select(dev(q), dev(k), P, "topk", 0.15, causal)
    got = va.recall(dev(q), dev(k), ti, tc, P, causal).cpu().numpy().astype(np.float64)
    ref = oracle.kept_mass(q, k, ti.cpu().numpy(), tc.cpu().numpy(), P, causal)
    err = np.abs(got - ref)
    assert err.max() <= KEPT_MAX and err.mean() <= KEPT_MEAN, (err.max(), err.mean())
    assert got.mean() > 0.3


def test_recall_full_size_sampled(gpu):
    # The 75k-token DiT layer (8 of its 40 heads) with the selection's own
    # lists: sampled blocks against the oracle.
    layer = synth.make_layer(4, heads=range(8))
    w = layer.w
    q, k = dev(layer.q), dev(layer.k)
    print("recall: 75k DiT layer, 8 heads", flush=True)
    idx, cnt = va.select(q, k, w.block, w.mode, w.param, w.causal)
    kept = va.recall(q, k, idx, cnt, w.block, w.causal)
    torch.cuda.synchronize()
    B, Hq, N, _ = q.shape
    Np = w.num_blocks
    rng = np.random.Generator(np.random.PCG64(4343))
    rows = np.sort(rng.choice(B * Hq * Np, size=16, replace=False))
    cap = idx.shape[-1]
    flat_i = idx.view(-1, cap)[torch.from_numpy(rows).cuda()].cpu().numpy()
    flat_c = cnt.view(-1)[torch.from_numpy(rows).cuda()].cpu().numpy()
    # the oracle reads lists by flat block id: place the sampled rows there
    full_i = np.zeros((B * Hq * Np, cap), dtype=np.int32)
    full_c = np.zeros(B * Hq * Np, dtype=np.int32)
    full_i[rows], full_c[rows] = flat_i, flat_c
    ref = oracle.kept_mass(layer.q, layer.k, full_i.reshape(B, Hq, Np, cap),
                           full_c.reshape(B, Hq, Np), w.block, w.causal, blocks=rows, nthreads=16)
    got = kept.cpu().numpy().astype(np.float64)
    errs = []
    for r in rows:
        i, h = r % Np, (r // Np) % Hq
        sl = slice(i * w.block, min(N, (i + 1) * w.block))
        errs.append(np.abs(got[0, h, sl] - ref[0, h, sl]))
    err = np.concatenate(errs)
    # ~19k keys per lane here: the fp32 sums are within ~1e-3 relative at worst
    assert err.max() <= 1e-3 and err.mean() <= 1e-4, (err.max(), err.mean())
    print(f"recall 75k: mean kept {got.mean():.4f}, max|d| {err.max():.2e}", flush=True)


@pytest.mark.parametrize("causal", [False, True])
def test_head_sparsity_is_bit_exact(gpu, causal):
    # Integer sums and one fp64 division on both sides: identical doubles.
    r = np.random.Generator(np.random.PCG64(55 + int(causal)))
    B, Hq, N, P = 2, 5, 1000, 64
    Np = (N + P - 1) // P
    L = np.array([min(N, (i + 1) * P) if causal else N for i in range(Np)])
    cnt = (r.uniform(0, 1, size=(B, Hq, Np)) * L).astype(np.int32)
    got = va.head_sparsity_of(torch.from_numpy(cnt).cuda(), N, P, causal).cpu().numpy()
    assert np.array_equal(got, oracle.head_sparsity(cnt, N, P, causal))
