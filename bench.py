"""Benchmark: one vertical-vector sparse attention layer (selection + sparse
attention) on one MI355X at the 75k-token DiT shape.

Workload (Wan-style 720p video DiT self-attention): latent grid 21x45x80 =
75600 tokens, 40 heads, head_dim 128, bf16, non-causal, query block 64,
topK keep ratio 15% (11340 keys per block).  Inputs are seeded synthetic
tensors with planted vertical structure (paper_2603_29494_amd.synth, workload
4); the paper's model activations are not available.

A step = vecattn_select (pooling, scoring, topK; lists without the -1 padding
past each count, which the attention never reads) + vecattn_attn_order (the
order in which the attention takes each head's blocks) +
vecattn_sparse_attn_ordered over all heads, inputs resident in HBM.  Timing: HIP events on the launch stream around
each call.  The W warm-up steps run back to back (their last ones give the
warm-cache figures); each of the K timed steps starts cold: a 1 GiB scratch
buffer is written just before it (outside its events), evicting the 256 MB
last-level cache and the L2s.  Prints one JSON line:
  value  = dense-equivalent TFLOP/s = 4 * Hq * N^2 * D / (median cold ms per layer)
  ms_per_step = median cold ms per layer (min / max and the warm figures beside)
  roofline   = the sparse-attention kernel (the dominant one): algorithmic
               MFMA FLOPs on the gathered tiles per launch / its mean duration
               over the timed steps, against 2516.6 TFLOP/s
  cpu_baseline = the CPU oracle on a bounded sample of the same layer,
               extrapolated to the layer
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
PEAK_HBM_GBS = 8000.0
TRAFFIC_RECORD = os.path.join(HERE, "profiles", "hbm_traffic_dit_wan_75k.md")
ATTN_SOURCE = os.path.join(HERE, "paper_2603_29494_amd", "csrc", "sparse_attn.hip")


def recorded_traffic(workload: str):
    """Bytes per launch of the attention kernel from the committed counter
    record (FETCH_SIZE + WRITE_SIZE, calibrated against a copy kernel), or
    None when the record is for another workload or another kernel source."""
    import hashlib
    try:
        sha = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
        for line in open(TRAFFIC_RECORD):
            f = dict(t.split("=", 1) for t in line.split() if "=" in t)
            if line.strip().startswith("traffic ") and f.get("workload") == workload \
                    and f.get("source_sha256") == sha:
                return float(f["bytes_per_launch"])
    except (OSError, ValueError, KeyError):
        pass
    return None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", type=int, default=4, help="synthetic workload id (1-5)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-blocks", type=int, default=0,
                    help="query blocks in the CPU-oracle sample (0: sized for ~15 s)")
    return ap.parse_args()


def cpu_baseline(layer, sample_blocks):
    """The oracle (selection + Eq. 4 attention, fp64) on a sample of query
    blocks, all host threads.  Scaled to dense-equivalent TFLOP/s of the
    sampled blocks."""
    import oracle
    w = layer.w
    q, k, v = layer.q, layer.k, layer.v
    B, Hq, N, D = q.shape
    Np = w.num_blocks
    nthreads = os.cpu_count() or 1
    rng = np.random.Generator(np.random.PCG64(12345))
    if sample_blocks <= 0:  # ~1/3 s per block and thread on the 75k layer: ~15 s in all
        sample_blocks = max(8, min(48 * nthreads, 2048))
    rows = np.sort(rng.choice(B * Hq * Np, size=sample_blocks, replace=False)).astype(np.int64)
    mode = oracle.TOPK if w.mode == "topk" else oracle.TOPP
    cap = oracle.topk_count(w.param, N) if w.mode == "topk" else N
    t0 = time.perf_counter()
    idx, cnt, _ = oracle.select(q, k, w.block, mode, w.param, w.causal, cap, rows=rows,
                                nthreads=nthreads)
    t1 = time.perf_counter()
    oracle.sparse_attn(q, k, v, idx, cnt, w.block, w.causal, blocks=rows, nthreads=nthreads)
    t2 = time.perf_counter()
    nrows = 0
    dense = 0.0
    for r in rows:
        i = int(r % Np)
        n_i = min(N, (i + 1) * w.block) - i * w.block
        keys = N if not w.causal else min(N, (i + 1) * w.block)
        dense += 4.0 * n_i * keys * D
        nrows += n_i
    secs = t2 - t0
    total_rows = B * Hq * N
    return {"value": dense / secs / 1e12, "unit": "TFLOP/s (dense-equivalent)", "cores": nthreads,
            "kind": "oracle", "extrapolated": True,
            "sample": f"{sample_blocks} random query blocks of the same layer ({nrows} of its "
                      f"{total_rows} query rows), select {t1 - t0:.2f} s + attention {t2 - t1:.2f} s; "
                      f"value = the sample's dense-equivalent FLOPs over its time, so the whole "
                      f"layer would take ~{secs * total_rows / nrows:.0f} s on these cores",
            "seconds": secs}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the sparse-attention layer is sharded by head "
              "across GPUs only by design (no multi-GPU path is built)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2603_29494_amd as va
    from paper_2603_29494_amd import synth

    va.load()  # fail loudly if the HIP library is missing
    if not torch.cuda.is_available():
        print("no GPU available", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    layer = synth.make_layer(args.workload)
    w = layer.w
    t_gen = time.perf_counter() - t_gen

    def to_dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)

    q, k, v = to_dev(layer.q), to_dev(layer.k), to_dev(layer.v)
    B, Hq, N, D = q.shape
    P = w.block
    Np = (N + P - 1) // P
    mode = w.mode
    cap = va.max_count(N, P, w.causal, mode, w.param)
    idx = torch.empty((B, Hq, Np, cap), dtype=torch.int32, device=dev)
    counts = torch.empty((B, Hq, Np), dtype=torch.int32, device=dev)
    ws = torch.empty(va.workspace_bytes(q, k, P, w.causal, mode, cap), dtype=torch.uint8, device=dev)
    out = torch.empty_like(q)
    order = torch.empty((B, Hq, Np), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev)   # cache eviction

    def step(ev):
        ev[0].record(stream)
        va.select(q, k, P, mode, w.param, w.causal, cap=cap, idx=idx, counts=counts, workspace=ws,
                  unpadded=True)
        ev[1].record(stream)
        va.attn_order(idx, counts, N, P, out=order)
        ev[2].record(stream)
        va.sparse_attn(q, k, v, idx, counts, P, w.causal, out=out, order=order)
        ev[3].record(stream)

    def new_events(n):
        return [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n)]

    warm_ev = new_events(args.warmup)
    for s in range(args.warmup):          # back to back: warm caches
        step(warm_ev[s])
    torch.cuda.synchronize()
    events = new_events(args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):           # timed: each step after a 1 GiB write
        scratch.fill_(s & 0xFF)
        step(events[s])
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps

    def stats(evs):
        sel = np.array([e[0].elapsed_time(e[1]) for e in evs])
        odr = np.array([e[1].elapsed_time(e[2]) for e in evs])
        att = np.array([e[2].elapsed_time(e[3]) for e in evs])
        lay = np.array([e[0].elapsed_time(e[3]) for e in evs])
        return sel, odr, att, lay

    sel_all, order_all, attn_all, layer_all = stats(events)
    sel_ms = float(np.median(sel_all))
    attn_ms = float(np.median(attn_all))
    layer_ms = float(np.median(layer_all))
    attn_mean_ms = float(np.mean(attn_all))    # the roofline's launch average
    warm = None
    if args.warmup >= 3:                  # the warm-up steps after the first two
        ws_, _, wa_, wl_ = stats(warm_ev[2:])
        warm = {"ms_per_step_median": round(float(np.median(wl_)), 4),
                "ms_select_median": round(float(np.median(ws_)), 4),
                "ms_attention_median": round(float(np.median(wa_)), 4), "steps": len(wl_)}

    cnt = counts.cpu().numpy().astype(np.int64)
    rows_per_block = np.minimum(N, (np.arange(Np) + 1) * P) - np.arange(Np) * P
    pairs = float((cnt * rows_per_block[None, None, :]).sum())   # query rows x selected keys
    f_alg = 4.0 * D * pairs                                        # QK^T + PV on gathered tiles
    if w.causal:
        f_dense = 2.0 * B * Hq * D * N * (N + 1)
        L = np.minimum(N, (np.arange(Np) + 1) * P)
    else:
        f_dense = 4.0 * B * Hq * N * N * D
        L = np.full(Np, N)
    keep = float(cnt.sum()) / float(B * Hq * L.sum())
    bytes_sel = 2.0 * B * N * D * (Hq + k.shape[1]) + 4.0 * cnt.sum() + 4.0 * B * Hq * Np
    dense_tflops = f_dense / (layer_ms * 1e-3) / 1e12
    attn_tflops = f_alg / (attn_mean_ms * 1e-3) / 1e12

    result = {
        "metric": "ms/layer + dense-equiv TFLOP/s (MFMA-peak %) at 75k-token DiT shape",
        "value": round(dense_tflops, 2),
        "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(layer_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": B, "q_heads": Hq, "kv_heads": int(k.shape[1]),
                   "seq_len": N, "head_dim": D, "causal": bool(w.causal), "query_block": P,
                   "selection": f"{mode} {w.param}"},
        "timing": "cold cache (1 GiB written before each timed step); median of the steps",
        "ms_per_step_min": round(float(layer_all.min()), 4),
        "ms_per_step_max": round(float(layer_all.max()), 4),
        "ms_select": round(sel_ms, 4),
        "ms_select_min_max": [round(float(sel_all.min()), 4), round(float(sel_all.max()), 4)],
        "ms_order": round(float(np.median(order_all)), 4),
        "ms_attention": round(attn_ms, 4),
        "ms_attention_min_max": [round(float(attn_all.min()), 4), round(float(attn_all.max()), 4)],
        "selection_pct": round(100.0 * sel_ms / layer_ms, 2),
        "warm": warm,
        "wall_ms_per_step": round(wall_ms, 4),
        "attention_mfma_pct": round(100.0 * attn_tflops / PEAK_BF16_TFLOPS, 2),
        "selection_hbm_pct": round(100.0 * bytes_sel / (sel_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 2),
        "achieved_keep": round(keep, 6),
        "roofline": {"bound": "mfma",
                     "kernel": f"k_sparse_attn<{D}, {'true' if k.stride() == v.stride() else 'false'}, "
                               f"{128 if w.block % 128 == 0 else 64}>",
                     "achieved": round(attn_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": recorded_traffic(w.name)},
        # K and V rows (2 x D bf16 each) gathered per selected key, per 64-row chunk
        "attention_gathered_bytes": 4.0 * D * float(cnt.sum()) * ((P + 63) // 64),
        "input_generation_s": round(t_gen, 1),
    }
    if not args.no_cpu_baseline:
        cb = cpu_baseline(layer, args.cpu_sample_blocks)
        result["cpu_baseline"] = {k2: (round(v2, 6) if isinstance(v2, float) else v2)
                                  for k2, v2 in cb.items()}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
