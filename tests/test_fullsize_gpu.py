"""The five synthetic workloads at full size, in the launch configuration the
benchmark times (selection with the library's default cap and workspace,
the block order, then sparse attention on its lists in that order), checked against the CPU oracle on a
random sample of query blocks: the selection rule of selection_parity and
the attention bar of test_attn_gpu (max-abs 2e-2, mean-abs 2e-3 against the
fp64 oracle on the GPU's own lists).  Plus properties that hold for every
block: lists ascending and in range, counts within [1, cap], and for topK the
exact budget.  Algorithm 1's cross-tile minS runs on the 75k DiT layer's
full sequence length (8 of its heads, so that cap = N lists stay small)."""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2603_29494_amd as va
from paper_2603_29494_amd import synth
from selection_parity import check_rows, check_rows_tiled

pytestmark = pytest.mark.gpu

# Sampled blocks per head checked against the oracle: the selection rule, and
# (a subset, as the fp64 attention oracle is slower) the attention bar.
SELECT_PER_HEAD = {1: 16, 2: 8, 3: 64, 4: 8, 5: 64}
ATTN_PER_HEAD = {1: 16, 2: 8, 3: 8, 4: 8, 5: 8}
NTHREADS = min(16, os.cpu_count() or 1)


def sample_per_head(rng, B, Hq, Np, per_head):
    rows = []
    for bh in range(B * Hq):
        rows.append(bh * Np + np.sort(rng.choice(Np, size=min(per_head, Np), replace=False)))
    return np.concatenate(rows)


def dev(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_workload_full_size(gpu, cid):
    layer = synth.make_layer(cid)
    w = layer.w
    q, k, v = dev(layer.q), dev(layer.k), dev(layer.v)
    B, Hq, N, D = q.shape
    P = w.block
    Np = (N + P - 1) // P
    print(f"workload {cid} {w.name}: select + attention", flush=True)
    idx, cnt = va.select(q, k, P, w.mode, w.param, w.causal)
    order = va.attn_order(idx, cnt, N, P)
    out = va.sparse_attn(q, k, v, idx, cnt, P, w.causal, order=order)
    torch.cuda.synchronize()
    cap = idx.shape[-1]
    # The block order: a permutation of each head's blocks, counts non-increasing.
    ar = torch.arange(Np, device="cuda", dtype=torch.int32)
    assert bool((torch.sort(order, dim=-1).values == ar).all())
    oc = torch.gather(cnt, 2, order.long())
    assert bool((oc[..., 1:] <= oc[..., :-1]).all())

    # Every block: counts, order, range (on the GPU, without copying the lists).
    L = torch.tensor([min(N, (i + 1) * P) if w.causal else N for i in range(Np)], device="cuda")
    c = cnt.long()
    assert bool((c >= 1).all()) and bool((c <= cap).all())
    if w.mode == "topk":
        kt = torch.tensor([min(max(math.ceil(w.param * int(l) - 1e-9), 1), int(l)) for l in L.tolist()],
                          device="cuda")
        assert bool((c == kt.view(1, 1, Np)).all()), "topK budget"
    flat = idx.view(-1, cap)
    cflat = c.view(-1)
    col = torch.arange(cap, device="cuda")
    chunk = max(1, (1 << 24) // cap)  # rows per check: the lists of a long layer are large
    for s in range(0, flat.shape[0], chunk):
        f, cf = flat[s:s + chunk], cflat[s:s + chunk]
        live = col.view(1, -1) < cf.view(-1, 1)
        assert bool(((f >= 0) | ~live).all()) and bool(((f == -1) | live).all())
        asc = (f[:, 1:] > f[:, :-1]) | ~live[:, 1:]
        assert bool(asc.all()), "lists ascending"
        Lrow = L[(torch.arange(s, s + f.shape[0], device="cuda") % Np)]
        assert bool(((f < Lrow.view(-1, 1)) | ~live).all()), "keys eligible"

    # Sampled blocks against the oracle: the selection rule on every sampled
    # block, the attention bar on a subset of them.
    rng = np.random.Generator(np.random.PCG64(4242 + cid))
    rows = sample_per_head(rng, B, Hq, Np, SELECT_PER_HEAD[cid])
    rsel = torch.from_numpy(rows).cuda()
    idx_s = flat[rsel].cpu().numpy()
    cnt_s = cflat[rsel].int().cpu().numpy()
    mode = oracle.TOPK if w.mode == "topk" else oracle.TOPP
    print(f"workload {cid}: selection rule on {len(rows)} sampled blocks", flush=True)
    mism = check_rows(layer.q, layer.k, P, mode, w.param, w.causal, cap, idx_s, cnt_s, rows,
                      compact=True)
    assert mism <= max(1, len(rows) // 20), mism
    keep = np.concatenate([np.arange(bh * SELECT_PER_HEAD[cid],
                                     bh * SELECT_PER_HEAD[cid] + ATTN_PER_HEAD[cid])
                           for bh in range(B * Hq)])
    keep = keep[keep < len(rows)]
    rows, idx_s, cnt_s = rows[keep], idx_s[keep], cnt_s[keep]
    print(f"workload {cid}: attention on {len(rows)} sampled blocks", flush=True)
    o_ref, _ = oracle.sparse_attn(layer.q, layer.k, layer.v, idx_s, cnt_s, P, w.causal,
                                  blocks=rows, compact=True, nthreads=NTHREADS)
    o_gpu = out.view(B, Hq, N, D)
    errs = []
    for t, r in enumerate(rows):
        i, h, b = r % Np, (r // Np) % Hq, r // (Np * Hq)
        n = min(N, (i + 1) * P) - i * P
        got = o_gpu[b, h, i * P:i * P + n].float().cpu().numpy()
        errs.append(np.abs(got - o_ref[t, :n]))
    err = np.concatenate([e.ravel() for e in errs])
    assert np.isfinite(err).all()
    assert err.max() <= 2e-2 and err.mean() <= 2e-3, (err.max(), err.mean())
    print(f"workload {cid}: {len(rows)} sampled blocks, max|dO| {err.max():.2e}, "
          f"mean|dO| {err.mean():.2e}", flush=True)


@pytest.mark.parametrize("group_tiles", [16, 8192])
def test_mins_tiled_full_length(gpu, group_tiles):
    layer = synth.make_layer(4, heads=range(8))
    w = layer.w
    q, k = dev(layer.q), dev(layer.k)
    B, Hq, N, D = q.shape
    P = w.block
    Np = (N + P - 1) // P
    alpha = 0.5
    print(f"cross-tile minS, N {N}, G_K {group_tiles}", flush=True)
    ncl = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cnt = va.select(q, k, P, "mins_tiled", alpha, False, cap=N, n_clamped=ncl, tile=16,
                         group_tiles=group_tiles)
    torch.cuda.synchronize()
    assert int(ncl.item()) == 0
    c = cnt.long().view(-1)
    assert bool((c >= 1).all()) and bool((c <= N).all())
    flat = idx.view(-1, N)
    col = torch.arange(N, device="cuda")
    for s in range(0, flat.shape[0], 256):
        f, cf = flat[s:s + 256], c[s:s + 256]
        live = col.view(1, -1) < cf.view(-1, 1)
        assert bool(((f >= 0) & (f < N) | ~live).all()) and bool(((f == -1) | live).all())
        assert bool(((f[:, 1:] > f[:, :-1]) | ~live[:, 1:]).all()), "lists ascending"
    rng = np.random.Generator(np.random.PCG64(5151 + group_tiles))
    rows = sample_per_head(rng, B, Hq, Np, 8)
    rsel = torch.from_numpy(rows).cuda()
    check_rows_tiled(layer.q, layer.k, P, alpha, False, 16, group_tiles,
                     flat[rsel].cpu().numpy(), c[rsel].int().cpu().numpy(), rows, compact=True)
    print(f"cross-tile minS G_K {group_tiles}: mean keep {float(c.double().mean()) / N:.3f}",
          flush=True)
