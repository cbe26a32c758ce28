#!/usr/bin/env python3
"""Benchmark of the selective-replay hot path on one MI355X.

One step = restore by crop (Algorithm 1, restore step) + one replay prefill of
the sanitized suffix (Algorithm 1, replay loop, prefill form), on the 8B
attention geometry: 32 query / 8 KV heads, d = 128, bf16, a contaminated cache
of 10240 tokens cropped to 8189 (unaligned to the 16-token block) and a
2048-token suffix replayed against it.  Inputs are seeded synthetic tensors
resident in HBM before timing starts.

A crop is destructive, so before every step the pre-crop block table, lengths
and free list (a few KB) are copied back outside the timed region; each step
is then bracketed by synchronisations and timed with HIP events on the stream
the library launches on.  The library's own event hook times the attention
kernel inside every timed step (the roofline figure).  The CPU baseline runs
the fp64 oracle on a bounded sample of the same workload's query rows.

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "suffix replay prefill tokens/s + attention TFLOP/s (% of bf16 MFMA peak)"
PEAK_BF16_TFLOPS = 2500.0       # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0


def attention_flops(P: int, S: int, hq: int, d: int) -> float:
    """Algorithmic FLOPs of prefix+causal attention: QK^T and PV over keys <= p."""
    return 4.0 * hq * d * (S * P + S * (S + 1) / 2.0)


def to_dev(arr, torch):
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()


def cpu_baseline(ep, w, budget_s: float):
    """fp64 oracle on a bounded, evenly spaced sample of suffix tokens (all heads)."""
    import oracle
    import workloads as W

    P, S = ep.prefix, ep.suffix
    hq, d = w.geometry.n_q_heads, w.geometry.head_dim
    f64 = lambda a: W.bf16_bits_to_f32(a).astype(np.float64)
    q, k, v = f64(ep.q[P:]), f64(ep.k), f64(ep.v)

    def run(n_tok):
        toks = np.linspace(0, S - 1, n_tok).round().astype(np.int64)
        rows = (toks[:, None] * hq + np.arange(hq)[None, :]).reshape(-1)
        pool = oracle.PoolModel(2 * (ep.t_contaminated // w.block_size + 2), 1,
                                ep.t_contaminated // w.block_size + 2, w.block_size)
        pool.reserve([0], [ep.t_contaminated]); pool.commit([0], [ep.t_contaminated])
        t0 = time.perf_counter()
        pool.crop([0], [P])
        pool.reserve([0], [S]); pool.commit([0], [S])
        oracle.attention(q, k, v, P, w.scale, rows=rows)
        return time.perf_counter() - t0

    dt = run(4)
    n_tok = int(max(4, min(S, 4 * budget_s / max(dt, 1e-6))))
    dt = run(n_tok)
    return {"value": n_tok / dt, "unit": "tokens/s", "cores": oracle.threads(), "kind": "oracle",
            "sample": f"{n_tok} of {S} suffix tokens (evenly spaced, all {hq} heads), "
                      f"fp64, {dt:.1f} s incl. crop + reserve on the oracle pool"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this hot path runs on one GPU; multi-GPU runs are not built "
                                   "(--gpus must be 1)", "n_gpus": args.gpus}), flush=True)
        return 2

    import torch

    import workloads as W
    from paper_2609_04875_amd import BF16, KVPool

    w = W.workload("llama8b_p8189_s2048_bf16")
    g = w.geometry
    ep = W.single_episode(w)
    P, S, Tc = ep.prefix, ep.suffix, ep.t_contaminated
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    nb = -(-Tc // w.block_size) + -(-(P + S) // w.block_size) + 8
    pool = KVPool(1, g.n_q_heads, g.n_kv_heads, g.head_dim, nb, 1, -(-Tc // w.block_size) + 4, BF16,
                  w.block_size)
    cq, ck, cv = (to_dev(ep.contaminated(x), torch) for x in ("q", "k", "v"))
    assert pool.replay(0, [0], [Tc], cq, ck, cv, torch.empty_like(cq), w.scale) == 0
    torch.cuda.synchronize()
    contaminated = pool.save_meta()
    q, k, v = (to_dev(getattr(ep, x)[P:], torch) for x in ("q", "k", "v"))
    o = torch.empty_like(q)
    del cq, ck, cv
    pool.enable_timing(True)

    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    step_ms, crop_ms, attn_ms, append_ms = [], [], [], []
    for i in range(args.warmup + args.steps):
        pool.load_meta(contaminated)          # outside the timed region
        torch.cuda.synchronize()
        ev[0].record(stream)
        rc1 = pool.crop([0], [P])
        ev[1].record(stream)
        rc2 = pool.replay(0, [0], [S], q, k, v, o, w.scale)
        ev[2].record(stream)
        torch.cuda.synchronize()
        if rc1 or rc2:
            raise RuntimeError(f"crop/replay failed: {rc1} {rc2}")
        if i >= args.warmup:
            step_ms.append(ev[0].elapsed_time(ev[2]))
            crop_ms.append(ev[0].elapsed_time(ev[1]))
            a_ms, t_ms = pool.last_times()
            append_ms.append(a_ms)
            attn_ms.append(t_ms)
    total_s = sum(step_ms) / 1e3
    tokens = S * args.steps
    flops = attention_flops(P, S, g.n_q_heads, g.head_dim)
    attn_mean = float(np.mean(attn_ms))
    achieved = flops / (attn_mean * 1e-3) / 1e12
    result = {
        "metric": METRIC,
        "value": tokens / total_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_s * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "prefix": P, "suffix": S, "contaminated": Tc,
                   "n_q_heads": g.n_q_heads, "n_kv_heads": g.n_kv_heads, "head_dim": g.head_dim,
                   "block_size": w.block_size, "episodes": 1, "recomputed_tokens": S},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "kernel": "attn_bf16_kernel<128,4>", "flops_per_launch": flops,
                     "kernel_ms": attn_mean},
        "breakdown_ms": {"crop": float(np.mean(crop_ms)), "append": float(np.mean(append_ms)),
                         "attention": attn_mean, "step": total_s * 1e3 / args.steps,
                         "step_min": float(np.min(step_ms))},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(ep, w, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
