"""Seeded synthetic attention-layer inputs with vertical-vector structure.

This module only draws random tensors; it holds none of the method's
arithmetic (no pooling, scoring, selection or attention).  Both the GPU path
and the CPU oracle take their inputs from here.

Every stream is ``numpy.random.Generator(PCG64(SeedSequence([seed, tag, head])))``
so a subset of heads can be regenerated without drawing the others.  Values are
drawn in fp32, structure is added in fp32, and the result is rounded once to
bf16 (round to nearest even, through ``torch``'s fp32 -> bf16 conversion).
Tensors are returned as bf16 bit patterns (``numpy.uint16``), contiguous
``[B, H, N, D]``.

The five workloads stand in for the paper's video-understanding (causal VLM
prefill) and video-generation (non-causal DiT) attention layers; the paper's
datasets and model activations are not available, so the vertical structure is
planted: a set of key columns is shifted along a per-head direction that the
queries share, which makes those columns score high for every query block.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, Iterable, Optional

import numpy as np

TAG_Q, TAG_K, TAG_V, TAG_DIR, TAG_PLANT, TAG_FRAME, TAG_RFF, TAG_MISC = range(8)


@dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    B: int
    Hq: int
    Hkv: int
    N: int
    D: int
    causal: bool
    block: int
    mode: str          # "topk" (param = keep ratio) or "topp" (param = mass threshold)
    param: float
    seed: int
    gen: Dict[str, float] = field(default_factory=dict)

    @property
    def num_blocks(self) -> int:
        return (self.N + self.block - 1) // self.block


def _seed(cid: int) -> int:
    return 20260329 + 1000 * cid


# Generator constants.  Logit units: a query shift gamma*u and key shift beta*u
# (u a unit vector) add gamma*beta/sqrt(D) to the score.  mu (the planted
# columns' logit boost) of the two topP workloads was set by bisection on mu,
# measuring the mean share of eligible keys the CPU oracle's topP selection
# keeps on seeded random blocks: for the Hunyuan-shaped DiT, 64 blocks of each
# of its 24 heads, mu = 4.745 -> mean keep 0.379 (per-head means 0.14 to 0.75,
# from the heads' planted densities of 1% to 8%; 8 blocks per head had put the
# mean 0.02 low); for the long VLM prefill, 48
# blocks of 3 heads, mu = 8 -> median keep ~2%, mean ~18% (blocks whose local
# window holds most of the mass keep far more).
WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "plumbing_1k", 1, 2, 2, 1024, 64, False, 64, "topk", 0.125, _seed(1),
                dict(n_planted=32, key_shift=4.0, query_shift=1.0)),
    2: Workload(2, "vlm_prefill_32k", 1, 28, 4, 32768, 128, True, 64, "topk", 0.10, _seed(2),
                dict(planted_frac=0.03, mu=4.0, query_shift=1.0, chunk=1024,
                     chunk_sigma=128 ** -0.25)),
    3: Workload(3, "vlm_long_131k", 1, 28, 4, 131072, 128, True, 64, "topp", 0.95, _seed(3),
                dict(planted_frac=0.02, mu=8.0, query_shift=1.0, window=256.0,
                     window_logits=2.0)),
    4: Workload(4, "dit_wan_75k", 1, 40, 40, 75600, 128, False, 64, "topk", 0.15, _seed(4),
                dict(planted_frac=0.04, key_shift_sqrtd=2.0, frame=3600, frame_sigma=0.5)),
    5: Workload(5, "dit_hunyuan_119k", 1, 24, 24, 118800, 128, False, 128, "topp", 0.9, _seed(5),
                dict(dens_lo=0.01, dens_hi=0.08, mu=4.745, query_shift=1.0)),
}


def _rng(seed: int, tag: int, h: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag, h])))


def _normal(seed: int, tag: int, h: int, shape) -> np.ndarray:
    return _rng(seed, tag, h).standard_normal(size=shape, dtype=np.float32)


def _unit(seed: int, tag: int, h: int, D: int) -> np.ndarray:
    u = _normal(seed, tag, h, (D,)).astype(np.float64)
    return (u / np.linalg.norm(u)).astype(np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 (round to nearest even) bit patterns as uint16."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


@dataclass
class Layer:
    w: Workload
    q: np.ndarray   # uint16 bf16 bits [B, Hq, N, D]
    k: np.ndarray   # uint16 bf16 bits [B, Hkv, N, D]
    v: np.ndarray   # uint16 bf16 bits [B, Hkv, N, D]
    planted: Dict[int, np.ndarray]  # kv head -> planted key rows


def _planted_rows(seed: int, h: int, N: int, n: int) -> np.ndarray:
    return np.sort(_rng(seed, TAG_PLANT, h).choice(N, size=n, replace=False))


def _rff(seed: int, N: int, D: int, length: float) -> np.ndarray:
    """Random Fourier features phi(t) = sqrt(2/D) cos(w t + b) with w ~ N(0, 1/length^2):
    phi(t).phi(t') approximates exp(-(t-t')^2 / (2 length^2)) (Rahimi & Recht, 2007)."""
    r = _rng(seed, TAG_RFF, 0)
    w = r.standard_normal(D) / length
    b = r.uniform(0.0, 2.0 * math.pi, D)
    t = np.arange(N, dtype=np.float64)[:, None]
    return (math.sqrt(2.0 / D) * np.cos(t * w[None, :] + b[None, :])).astype(np.float32)


def make_layer(cid: int, heads: Optional[Iterable[int]] = None, mu: Optional[float] = None) -> Layer:
    """Inputs of workload ``cid``.  ``heads`` restricts Q to those query heads
    (K/V then hold only the kv heads they use, in order); ``mu`` overrides the
    planted-column logit boost (used when calibrating)."""
    w = WORKLOADS[cid]
    g = w.gen
    B, Hq, Hkv, N, D, s = w.B, w.Hq, w.Hkv, w.N, w.D, w.seed
    grp = Hq // Hkv
    qheads = list(range(Hq)) if heads is None else sorted(set(int(h) for h in heads))
    kvheads = sorted(set(h // grp for h in qheads))
    q = np.empty((B, len(qheads), N, D), dtype=np.uint16)
    k = np.empty((B, len(kvheads), N, D), dtype=np.uint16)
    v = np.empty((B, len(kvheads), N, D), dtype=np.uint16)
    planted: Dict[int, np.ndarray] = {}
    rff = None
    if cid == 3:
        rff = _rff(s, N, D, g["window"])
        a = math.sqrt(g["window_logits"] * math.sqrt(D))
    if cid == 5:
        order = _rng(s, TAG_MISC, 0).permutation(Hq)
        dens = np.linspace(g["dens_lo"], g["dens_hi"], Hq)[np.argsort(order)]
    for b in range(B):
        for kk, hk in enumerate(kvheads):
            tag = b * 4096 + hk
            K = _normal(s, TAG_K, tag, (N, D))
            V = _normal(s, TAG_V, tag, (N, D))
            if cid == 1:
                u = _unit(s, TAG_DIR, 0, D)
                rows = _planted_rows(s, tag, N, int(g["n_planted"]))
                K[rows] += g["key_shift"] * u
            elif cid in (2, 3):
                u = _unit(s, TAG_DIR, tag, D)
                rows = _planted_rows(s, tag, N, int(round(g["planted_frac"] * N)))
                beta = (g["mu"] if mu is None else mu) * math.sqrt(D) / g["query_shift"]
                K[rows] += beta * u
                if cid == 2:
                    nch = (N + g["chunk"] - 1) // int(g["chunk"])
                    off = _normal(s, TAG_FRAME, tag, (nch, D)) * g["chunk_sigma"]
                    K += np.repeat(off, int(g["chunk"]), axis=0)[:N]
                else:
                    K += a * rff
            elif cid == 4:
                u = _unit(s, TAG_DIR, tag, D)
                rows = _planted_rows(s, tag, N, int(round(g["planted_frac"] * N)))
                K[rows] += g["key_shift_sqrtd"] * math.sqrt(D) * u
                nfr = (N + int(g["frame"]) - 1) // int(g["frame"])
                off = _normal(s, TAG_FRAME, tag, (nfr, D)) * g["frame_sigma"]
                K += np.repeat(off, int(g["frame"]), axis=0)[:N]
            elif cid == 5:
                u = _unit(s, TAG_DIR, tag, D)
                rows = _planted_rows(s, tag, N, max(1, int(round(dens[hk] * N))))
                beta = (g["mu"] if mu is None else mu) * math.sqrt(D) / g["query_shift"]
                K[rows] += beta * u
            planted[hk] = rows
            k[b, kk] = to_bf16_bits(K)
            v[b, kk] = to_bf16_bits(V)
            del K, V
        for qq, h in enumerate(qheads):
            hk = h // grp
            tag = b * 4096 + h
            Q = _normal(s, TAG_Q, tag, (N, D))
            if cid == 1:
                Q += g["query_shift"] * _unit(s, TAG_DIR, 0, D)
            elif cid in (2, 3, 5):
                Q += g["query_shift"] * _unit(s, TAG_DIR, b * 4096 + hk, D)
                if cid == 2:
                    nch = (N + g["chunk"] - 1) // int(g["chunk"])
                    off = _normal(s, TAG_FRAME, b * 4096 + hk, (nch, D)) * g["chunk_sigma"]
                    Q += np.repeat(off, int(g["chunk"]), axis=0)[:N]
                if cid == 3:
                    Q += a * rff
            q[b, qq] = to_bf16_bits(Q)
            del Q
    return Layer(w, q, k, v, planted)


def random_bits(seed: int, shape, scale: float = 1.0) -> np.ndarray:
    """i.i.d. N(0, scale^2) tensor rounded to bf16 bits (test inputs)."""
    x = np.random.Generator(np.random.PCG64(seed)).standard_normal(size=shape, dtype=np.float32)
    return to_bf16_bits(x * np.float32(scale))


def planted_case(seed: int, B: int, Hq: int, Hkv: int, N: int, D: int, frac: float = 0.05,
                 logits: float = 3.0):
    """Small random layer with planted heavy key columns (test inputs): returns
    (q, k, v) bf16 bits."""
    r = np.random.Generator(np.random.PCG64(seed))
    q = r.standard_normal((B, Hq, N, D), dtype=np.float32)
    k = r.standard_normal((B, Hkv, N, D), dtype=np.float32)
    v = r.standard_normal((B, Hkv, N, D), dtype=np.float32)
    g = Hq // Hkv
    for b in range(B):
        for hk in range(Hkv):
            u = r.standard_normal(D).astype(np.float32)
            u /= np.linalg.norm(u)
            n = max(1, int(round(frac * N)))
            rows = r.choice(N, size=n, replace=False)
            k[b, hk, rows] += np.float32(logits * math.sqrt(D)) * u
            q[b, hk * g:(hk + 1) * g] += u
    return to_bf16_bits(q), to_bf16_bits(k), to_bf16_bits(v)
