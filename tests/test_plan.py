"""Per-head filter ratios (Eq. 5, Sec. 3.1.2): the library's dynamic programme
(host code behind the C ABI) against the oracle's exhaustive search of the
same objective -- the largest summed per-head performance whose mean
sparsity reaches the target.  Several choices can be optimal, so the optimum
value is compared and the returned choice is checked to attain it."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2603_29494_amd as va
from paper_2603_29494_amd import _lib


def test_worked_example():
    # Two heads, three candidates each (sparsity, perf):
    #   head 0: (0.1, 1.0) (0.5, 0.8) (0.9, 0.2);  head 1: (0.2, 1.0) (0.6, 0.9) (0.8, 0.5)
    # mean sparsity >= 0.5 needs a sparsity sum >= 1.0: the best is (0.5 + 0.6,
    # 0.8 + 0.9 = 1.7); >= 0.85 leaves only (0.9, 0.8): 0.7; target 0: 2.0.
    sp = np.array([[0.1, 0.5, 0.9], [0.2, 0.6, 0.8]])
    pf = np.array([[1.0, 0.8, 0.2], [1.0, 0.9, 0.5]])
    assert va.plan_filter_ratios(sp, pf, 0.5)[0].tolist() == [1, 1]
    assert va.plan_filter_ratios(sp, pf, 0.5)[1] == pytest.approx(1.7)
    assert va.plan_filter_ratios(sp, pf, 0.85)[0].tolist() == [2, 2]
    assert va.plan_filter_ratios(sp, pf, 0.0)[0].tolist() == [0, 0]
    with pytest.raises(va.VecattnError):
        va.plan_filter_ratios(sp, pf, 0.9)


@pytest.mark.parametrize("seed", range(40))
def test_matches_exhaustive_search(seed):
    r = np.random.Generator(np.random.PCG64(900 + seed))
    H, C = int(r.integers(1, 6)), int(r.integers(1, 6))
    sp = r.integers(0, 21, size=(H, C)) / 20.0      # multiples of 1/grid: no rounding
    pf = r.standard_normal((H, C))
    for target in (0.0, float(r.uniform(0, 1)), float(r.choice(sp.ravel())), 1.0):
        best, optima = oracle.plan_filter_ratios(sp, pf, target)
        if best is None:
            with pytest.raises(va.VecattnError):
                va.plan_filter_ratios(sp, pf, target)
            continue
        choice, val = va.plan_filter_ratios(sp, pf, target)
        assert val == pytest.approx(best, abs=1e-9)
        assert tuple(choice.tolist()) in optima
        assert sp[np.arange(H), choice].mean() >= target - 1e-12


def test_tied_optima_return_one_of_them():
    # two identical heads (0.2, 1.0) (0.4, 0.5), mean >= 0.3: (0,1) and (1,0)
    # both reach 1.5 (hand-worked; the oracle's pin lists both)
    sp = np.array([[0.2, 0.4], [0.2, 0.4]])
    pf = np.array([[1.0, 0.5], [1.0, 0.5]])
    choice, val = va.plan_filter_ratios(sp, pf, 0.3)
    assert val == pytest.approx(1.5) and tuple(choice.tolist()) in ((0, 1), (1, 0))


def test_target_zero_takes_each_heads_best_and_lower_index_on_ties():
    sp = np.array([[0.0, 0.3, 0.6], [0.1, 0.2, 0.3]])
    pf = np.array([[0.5, 0.9, 0.9], [0.7, 0.1, 0.7]])
    choice, val = va.plan_filter_ratios(sp, pf, 0.0)
    assert choice.tolist() == [1, 0] and val == pytest.approx(1.6)


def test_forty_heads_monotone_and_feasible():
    r = np.random.Generator(np.random.PCG64(77))
    H, C = 40, 16
    sp = np.sort(r.uniform(0, 1, size=(H, C)), axis=1)
    pf = 1.0 - sp ** r.uniform(1, 4, size=(H, 1))   # performance falls as sparsity rises
    prev = np.inf
    for target in np.linspace(0.0, 0.9, 10):
        choice, val = va.plan_filter_ratios(sp, pf, target, grid=2000)
        assert sp[np.arange(H), choice].mean() >= target - 0.5 / 2000
        assert val <= prev + 1e-9
        prev = val
        uni = [pf[:, c].sum() for c in range(C) if sp[:, c].mean() >= target + 0.5 / 2000]
        if uni:
            assert val >= max(uni) - 1e-9    # never worse than one candidate for all heads


def test_rejects_bad_arguments():
    lib = _lib.load()
    sp = np.array([[0.5]])
    pf = np.array([[1.0]])
    ch = np.zeros(1, dtype=np.int32)
    best = ctypes.c_double()
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    call = lambda H=1, C=1, s=sp, p=pf, t=0.5, g=100, c=ch: lib.vecattn_plan_filter_ratios(
        H, C, None if s is None else P(s), None if p is None else P(p), t, g,
        None if c is None else P(c), ctypes.byref(best))
    assert call() == 0
    assert call(H=0) == 1 and call(C=0) == 1
    assert call(s=None) == 1 and call(p=None) == 1 and call(c=None) == 1
    assert call(t=-0.1) == 1 and call(t=1.5) == 1 and call(t=float("nan")) == 1
    assert call(g=0) == 1
    assert call(s=np.array([[1.5]])) == 1
    assert call(p=np.array([[np.inf]])) == 1
    assert call(t=0.6) == 3                     # out of reach


@pytest.mark.gpu
def test_head_sparsity_table_and_plan_on_gpu(gpu):
    # sp_h(alpha) measured by the GPU selection equals the oracle's; Perf_h is
    # the oracle's recall of each head's pooled softmax mass (a synthetic
    # stand-in for the paper's model-level performance); the plan reaches the
    # target and beats using one alpha for every head.
    import torch
    from paper_2603_29494_amd import synth
    q, k, _ = synth.planted_case(31, 1, 6, 6, 1024, 128)
    # heads differ: scale the queries of head h by (1 + h / 2) (sharper maps)
    qf = synth.bits_to_f32(q) * (1.0 + 0.5 * np.arange(6)).reshape(1, 6, 1, 1).astype(np.float32)
    q = synth.to_bf16_bits(qf)
    dev = lambda b: torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).cuda()
    alphas = [0.25, 0.5, 1.0, 2.0, 4.0]
    sp_gpu = va.head_sparsity(dev(q), dev(k), 64, "mins", alphas, False).numpy()
    Np, N = 16, 1024
    sp_ora = np.zeros_like(sp_gpu)
    perf = np.zeros_like(sp_gpu)
    for c, a in enumerate(alphas):
        idx, cnt, _ = oracle.select(q, k, 64, oracle.MINS, a, False, N)
        for h in range(6):
            sp_ora[h, c] = 1.0 - cnt[0, h].sum() / (Np * N)
            rec = []
            for i in range(Np):
                s = oracle.pooled_scores(q, k, 64, False, 0, h, i)
                e = np.exp(s - s.max())
                rec.append(e[idx[0, h, i, :cnt[0, h, i]]].sum() / e.sum())
            perf[h, c] = np.mean(rec)
    assert np.abs(sp_gpu - sp_ora).max() <= 2e-3
    target = float(np.median(sp_ora))
    choice, val = va.plan_filter_ratios(sp_ora, perf, target)
    assert sp_ora[np.arange(6), choice].mean() >= target - 1e-3
    uni = [perf[:, c].sum() for c in range(len(alphas)) if sp_ora[:, c].mean() >= target]
    assert val >= max(uni) - 1e-9
    # the plan applied in one selection call (one alpha per head)
    per_head = [alphas[c] for c in choice]
    _, cnt = va.select(dev(q), dev(k), 64, "mins", per_head, False, cap=N)
    got = 1.0 - cnt[0].double().sum(dim=1).cpu().numpy() / (Np * N)
    assert np.abs(got - sp_ora[np.arange(6), choice]).max() <= 2e-3
