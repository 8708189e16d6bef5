"""Keep ratio of the topP synthetic workloads (3: long VLM prefill, 5:
Hunyuan-shaped DiT) under the CPU oracle, for choosing their planted-column
boost mu.  Not a test; run by hand:

    python tests/calibrate_topp_workloads.py 5 4.35
    python tests/calibrate_topp_workloads.py 3 8.0

Prints the mean / median / min / max fraction of eligible keys that the
oracle's topP selection keeps on 48 random blocks of a few query heads.
"""
import os
import sys
import time

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
from paper_2603_29494_amd import synth  # noqa: E402


def keep_stats(cid: int, mu: float, nblocks: int = 48, seed: int = 1):
    heads = [0, 9, 17] if cid == 3 else [0, 5, 11, 23]
    layer = synth.make_layer(cid, heads=heads, mu=mu)
    w = layer.w
    B, Hq, N, _ = layer.q.shape
    Np = (N + w.block - 1) // w.block
    rows = np.sort(np.random.default_rng(seed).choice(B * Hq * Np, size=nblocks, replace=False))
    mode = oracle.TOPP if w.mode == "topp" else oracle.TOPK
    _, cnt, _ = oracle.select(layer.q, layer.k, w.block, mode, w.param, w.causal, N, rows=rows,
                              nthreads=os.cpu_count() or 1)
    cnt = cnt.reshape(-1)[rows]
    L = np.array([min(N, (r % Np + 1) * w.block) if w.causal else N for r in rows])
    return cnt / L


if __name__ == "__main__":
    cid = int(sys.argv[1])
    mu = float(sys.argv[2]) if len(sys.argv) > 2 else None
    t0 = time.time()
    k = keep_stats(cid, mu)
    print(f"workload {cid} mu {mu}: keep mean {k.mean():.4f} median {np.median(k):.4f} "
          f"min {k.min():.4f} max {k.max():.4f} ({time.time() - t0:.0f} s)")
