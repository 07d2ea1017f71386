"""Benchmark of the PSA block-sparse attention forward on one MI355X.

A step is one psa_attention_fwd call over one batch of the workload (stripe-parameter upload,
kept-block counting, load-balanced scheduling and the persistent sparse attention kernel),
with Q/K/V already resident in HBM.  The library's own dense kernel is timed on the same
tensors for the speedup.  One JSON line goes to stdout; details go to stderr.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wan14b|wan1_3b|hunyuan|sweep]
                    [--target 0.3] [--no-dense] [--no-cpu-baseline]
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA peak (published)
WORKLOAD_TEXT = {
    "wan14b": "Wan 2.1 14B 720p attention layer: B=1, 40 heads, d=128, grid 21x45x80 (N=75600), "
              "block 128, seeded per-head stripes (kept-tile density 10-40%)",
    "wan1_3b": "Wan 2.1 1.3B 480p attention layer: B=1, 12 heads, d=128, grid 21x30x52 (N=32760), "
               "block 128, seeded per-head stripes (kept-tile density 15-40%)",
    "hunyuan": "HunyuanVideo 720p joint attention: B=1, 24 heads, d=128, grid 33x45x80 + 256 text "
               "(N=119056), block 128, seeded per-head stripes (kept-tile density 10-35%)",
    "sweep": "Wan 2.1 14B shape (B=1, 40 heads, d=128, N=75600), every head forced to one kept-tile "
             "density",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="wan14b", choices=sorted(WORKLOAD_TEXT))
    p.add_argument("--target", type=float, default=0.3, help="sweep density")
    p.add_argument("--dense-steps", type=int, default=None)
    p.add_argument("--no-dense", action="store_true")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--copy-mb", type=int, default=0,
                   help="run one plain device copy of this many MiB first (counter calibration)")
    return p.parse_args()


def time_calls(fn, steps, warmup, torch):
    """Mean ms per call over `steps` calls after `warmup`, HIP events on the current stream."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def computed_flops(psa, cfg, params, torch):
    """4 d sum over kept tiles of (valid query rows x valid key rows), from the library's map."""
    bm, _, per_head = psa.build_blockmap(params, (cfg.frames, cfg.height, cfg.width, cfg.n_text), cfg.block)
    nb = cfg.n_blocks
    lens = torch.full((nb,), float(cfg.block), dtype=torch.float64, device=bm.device)
    lens[-1] = cfg.n_tokens - (nb - 1) * cfg.block
    pairs = (bm.to(torch.float64) * lens[None, :, None] * lens[None, None, :]).sum().item()
    density = per_head.double().sum().item() / (len(params) * nb * nb)
    return 4.0 * cfg.head_dim * cfg.batch * pairs, density


def cpu_baseline(cfg, params, seconds):
    """The oracle on the host cores, on a seeded sample of query blocks of the same workload."""
    import oracle
    from threadpoolctl import threadpool_info
    from workloads.inputs import make_head_qkv, rope_tables
    bmap = oracle.blockmap(params, cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)
    rows_kept = oracle.kept_per_row(bmap)
    nb = cfg.n_blocks
    lens = np.full(nb, cfg.block, dtype=np.float64)
    lens[-1] = cfg.n_tokens - (nb - 1) * cfg.block
    rng = np.random.default_rng(12345)
    heads = rng.choice(cfg.heads, size=min(4, cfg.heads), replace=False)
    tables = rope_tables(cfg)
    data = {int(h): make_head_qkv(cfg, 0, int(h), tables) for h in heads}
    flops = 0.0
    n_blocks = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds and n_blocks < 400:
        h = int(heads[n_blocks % len(heads)])
        qb = int(rng.integers(nb))
        q, k, v = data[h]
        rows = np.arange(qb * cfg.block, min(cfg.n_tokens, (qb + 1) * cfg.block))
        oracle.masked_attention(q, k, v, bmap[h], cfg.block, cfg.scale, rows)
        flops += 4.0 * cfg.head_dim * lens[qb] * float((bmap[h, qb] * lens).sum())
        n_blocks += 1
    elapsed = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {
        "value": flops / elapsed / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": "%d query blocks of 128 rows from heads %s of the same workload (float64 numpy "
                  "oracle, %.1f s, %d host cores visible); %.3g TFLOP computed, mean %.1f kept "
                  "blocks per sampled row" % (n_blocks, sorted(int(x) for x in heads), elapsed,
                                              os.cpu_count() or 0, flops / 1e12,
                                              float(rows_kept[heads].mean())),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (the attention "
              "kernel shards over heads; see DESIGN.md). Run with --gpus 1.", file=sys.stderr)
        return 2
    import torch
    import paper_2609_37001_amd as psa
    from workloads import get_config, make_qkv, stripe_params

    name = args.workload
    cfg = get_config(name)
    params = stripe_params(name, args.target if name == "sweep" else None)
    grid = (cfg.frames, cfg.height, cfg.width, cfg.n_text)
    log("workload %s: generating inputs" % name)
    t0 = time.perf_counter()
    q, k, v = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to("cuda:0")
               for x in make_qkv(cfg, workers=16))
    log("inputs ready in %.1f s" % (time.perf_counter() - t0))
    if args.copy_mb:
        src = torch.ones(args.copy_mb << 18, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: %d MiB read, %d MiB written" % (args.copy_mb, args.copy_mb))
        del src, dst
    o = torch.empty_like(q)
    ws = psa.Workspace(cfg.batch, cfg.heads, grid, cfg.block, q.device)
    flops, density = computed_flops(psa, cfg, params, torch)

    def sparse():
        psa.attention_fwd(q, k, v, grid, cfg.block, params, cfg.scale, out=o, workspace=ws)

    ms = time_calls(sparse, args.steps, args.warmup, torch)
    tflops = flops / (ms * 1e-3) / 1e12
    dense_flops = cfg.dense_flops
    result = {
        "metric": "sparse-attn fwd computed TFLOP/s & MFU; speedup vs own dense at Wan-14B shape",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[name] + (" (target %.2f)" % args.target if name == "sweep" else ""),
                   "kept_tile_density": round(density, 5), "computed_tflop": round(flops / 1e12, 4),
                   "dense_tflop": round(dense_flops / 1e12, 4)},
        "mfu": round(tflops / PEAK_BF16_TFLOPS, 4),
        "dense_equiv_tflops": round(dense_flops / (ms * 1e-3) / 1e12, 2),
    }
    log("sparse: %.3f ms/step, %.1f TFLOP/s computed, MFU %.3f, density %.4f" % (ms, tflops, tflops / PEAK_BF16_TFLOPS, density))
    if not args.no_dense:
        def dense():
            psa.dense_fwd(q, k, v, cfg.block, cfg.scale, out=o)
        dsteps = args.dense_steps or max(3, args.steps // 2)
        dms = time_calls(dense, dsteps, 1, torch)
        dtf = dense_flops / (dms * 1e-3) / 1e12
        speedup = dms / ms
        result.update({
            "dense_ms": round(dms, 4),
            "dense_tflops": round(dtf, 2),
            "dense_mfu": round(dtf / PEAK_BF16_TFLOPS, 4),
            "speedup_vs_dense": round(speedup, 3),
            "mfu_ratio_sparse_over_dense": round((tflops / dtf), 4),
            "speedup_over_inverse_density": round(speedup * density, 4),
        })
        log("dense: %.3f ms, %.1f TFLOP/s, speedup %.3f (x density %.3f)" % (dms, dtf, speedup, speedup * density))
    result["roofline"] = {
        "bound": "mfma",
        "achieved": round(tflops, 2),
        "peak": PEAK_BF16_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
        "traffic": None,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline: timing the oracle for about %.0f s" % args.cpu_seconds)
        result["cpu_baseline"] = cpu_baseline(cfg, params, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
