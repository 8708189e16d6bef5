"""The sparse-pattern statistics tool (Sec. 2.2): curve invariants that hold
for any attention map, and the vertical-vector structure of the planted
synthetic workload (CPU, small maps)."""
import numpy as np
import pytest
import torch

from paper_2603_29494_amd import patterns, synth


def _map(seed, n=256, d=32, causal=False):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(n, d, generator=g) * 1.5
    k = torch.randn(n, d, generator=g)
    return patterns.attention_map(q, k, causal)


@pytest.mark.parametrize("causal", [False, True])
def test_oracle_dominates_and_curves_are_monotone(causal):
    a = _map(1, causal=causal)
    oracle = patterns.sparsity_recall(a, "oracle", 1, causal)
    for p in ("block", "vertical_vector", "horizontal_vector", "line"):
        sp, rc = patterns.sparsity_recall(a, p, 16, causal)
        assert np.all(np.diff(sp) <= 1e-12) and np.all(np.diff(rc) >= -1e-12), p
        assert sp[0] == 1.0 and rc[0] == 0.0
        assert abs(rc[-1] - 1.0) < 1e-9 and abs(sp[-1]) < 1e-9, p
        for s, r in zip(sp, rc):    # no mask of that size keeps more mass than the top entries
            assert patterns.recall_at(oracle, s) >= r - 1e-9, (p, s)


def test_unit_regions_are_the_oracle():
    a = _map(2)
    o = patterns.sparsity_recall(a, "oracle", 1, False)
    for p in ("block", "vertical_vector", "horizontal_vector"):
        c = patterns.sparsity_recall(a, p, 1, False)
        assert np.allclose(c[0], o[0]) and np.allclose(c[1], o[1]), p


def test_line_steps_count_overlaps_once():
    a = _map(3, n=64)
    sp, rc = patterns.sparsity_recall(a, "line", 1, True)
    assert len(sp) == 64 + 64 + 1              # causal: 64 columns, 64 lower diagonals
    assert abs(rc[-1] - 1.0) < 1e-9 and abs(sp[-1]) < 1e-9
    # each step's increments never exceed the line's own entries
    assert np.all(np.diff(1.0 - sp) * 64 * 65 / 2 <= 64 + 1e-6)


def test_planted_workload_has_vertical_vector_structure():
    # The plumbing workload plants key columns that every query favours: at
    # 90% sparsity vertical vectors (P = 64 queries x 1 key) keep more of the
    # attention mass than horizontal vectors or 64 x 64 blocks.
    layer = synth.make_layer(1)
    q = torch.from_numpy(synth.bits_to_f32(layer.q[0, 0]))
    k = torch.from_numpy(synth.bits_to_f32(layer.k[0, 0]))
    r = patterns.compare(q, k, 64, False, sparsities=(0.9,), max_lines=0)
    v, h, b = r["vertical_vector"][0.9], r["horizontal_vector"][0.9], r["block"][0.9]
    assert v > h and v > b, r
    assert r["oracle"][0.9] >= v
