"""The selection entry point without a caller workspace (vecattn_select_noalloc,
for callers that cannot allocate device memory), through the C ABI: its lists
and counts equal vecattn_select's on the same inputs (the same kernels on a
workspace the library holds), also on a second, smaller call right after the
first (the workspace keeps the first call's contents), and follow the oracle's
selection rule; shapes whose workspace exceeds the library's 64 MiB are
rejected."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_29494_amd import _lib, synth
from selection_parity import check_rows

pytestmark = pytest.mark.gpu


def dev(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


CASES = [  # seed, B, Hq, Hkv, N, D, block, causal, mode, param
    (1, 1, 4, 2, 3000, 128, 64, True, "topk", 0.15),
    (2, 1, 2, 2, 1000, 64, 64, False, "topk", 0.25),
    (3, 1, 4, 1, 2500, 128, 64, False, "topp", 0.9),
    (4, 1, 2, 2, 700, 128, 48, True, "topp", 0.8),
    (5, 1, 3, 3, 2000, 128, 64, False, "mins", 0.5),
    (6, 2, 2, 1, 900, 64, 32, True, "mins", 0.3),
]


@pytest.mark.parametrize("pair", [(0, 1), (2, 3), (4, 5)])
def test_noalloc_matches_select_twice_in_a_row(gpu, pair):
    for n in pair:                       # the second call is the smaller one
        seed, B, Hq, Hkv, N, D, block, causal, mode, param = CASES[n]
        q, k, _ = synth.planted_case(800 + seed, B, Hq, Hkv, N, D)
        tq, tk = dev(q), dev(k)
        cap = _lib.max_count(N, block, causal, mode, param)
        ws = _lib.workspace_bytes(tq, tk, block, causal, mode, cap)
        assert ws <= _lib.STATIC_WORKSPACE_BYTES
        Np = (N + block - 1) // block
        idx = torch.full((B, Hq, Np, cap), 7, dtype=torch.int32, device="cuda")
        cnt = torch.full((B, Hq, Np), 7, dtype=torch.int32, device="cuda")
        _lib.select_noalloc(tq, tk, block, mode, param, causal, cap, idx, cnt)
        ref_i, ref_c = _lib.select(tq, tk, block, mode, param, causal, cap=cap)
        torch.cuda.synchronize()
        assert torch.equal(cnt, ref_c) and torch.equal(idx, ref_i), CASES[n]
        omode = {"topk": oracle.TOPK, "topp": oracle.TOPP, "mins": oracle.MINS}[mode]
        rows = list(range(B * Hq * Np))
        mism = check_rows(q, k, block, omode, param, causal, cap, idx.cpu().numpy(),
                          cnt.cpu().numpy(), rows)
        assert mism <= max(1, len(rows) // 20)


def test_noalloc_rejects_workspace_beyond_limit(gpu):
    # 40 heads x 75600 keys need far more than 64 MiB: CAPACITY, no launch.
    q = torch.empty((1, 40, 75600, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.empty((1, 40, 75600, 128), dtype=torch.bfloat16, device="cuda")
    assert _lib.workspace_bytes(q, k, 64, False, "topk", 11340) > _lib.STATIC_WORKSPACE_BYTES
    idx = torch.empty((1, 40, 1182, 11340), dtype=torch.int32, device="cuda")
    cnt = torch.empty((1, 40, 1182), dtype=torch.int32, device="cuda")
    with pytest.raises(_lib.VecattnError) as e:
        _lib.select_noalloc(q, k, 64, "topk", 0.15, False, 11340, idx, cnt)
    assert e.value.status == _lib.ERR_CAPACITY
