"""Benchmark of the PSA block-sparse attention forward on one MI355X.

A step is one psa_attention_fwd call over one batch of the workload (stripe-parameter upload,
kept-block counting, load-balanced scheduling and the persistent sparse attention kernel),
with Q/K/V already resident in HBM.  The library's own dense kernel is timed on the same
tensors for the speedup.  One JSON line goes to stdout; details go to stderr.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wan14b|wan1_3b|hunyuan|sweep]
                    [--target 0.3] [--no-dense] [--no-cpu-baseline]

The roofline figure is that of the persistent sparse kernel alone (psa_attention_run over a
planned workspace, timed with HIP events on the launch stream).  Its HBM traffic comes from two
rocprofv3 counter runs summarised by

    python bench.py --counters <FETCH_SIZE run dir> <WRITE_SIZE run dir>

into profiles/; the figure is reported only while the kernel sources hash to the ones profiled.
"""
import argparse
import csv
import glob
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA peak (published)
HBM_PEAK = 8.0e12             # MI355X HBM3E bandwidth, bytes/s (published)
KERNEL = "psa_pair_kernel<128, 128, true, false>"       # the sparse attention at block 128
KERNEL_3D = "psa_pair_kernel<128, 128, true, true>"     # ... with the 3D-padding masks
ATTN_PREFIXES = ("psa_sparse_kernel", "psa_dense_kernel", "psa_pair_kernel")  # attention kernels
COUNTERS_MD = os.path.join(ROOT, "profiles", "psa_pair_kernel_wan14b_counters.md")
SOURCES = ("paper_2609_37001_amd/csrc/psa_kernels.hip", "paper_2609_37001_amd/csrc/psa_launch.h",
           "paper_2609_37001_amd/csrc/psa_api.hip", "paper_2609_37001_amd/build.py", "include/psa.h")
WORKLOAD_TEXT = {
    "tiny": "tiny layer: B=1, 2 heads, d=64, grid 4x16x16 (N=1024), block 64, stripes drawn uniformly "
            "from the paper's candidate ranges",
    "wan14b": "Wan 2.1 14B 720p attention layer: B=1, 40 heads, d=128, grid 21x45x80 (N=75600), "
              "block 128, seeded per-head stripes (kept-tile density 10-40%)",
    "wan1_3b": "Wan 2.1 1.3B 480p attention layer: B=1, 12 heads, d=128, grid 21x30x52 (N=32760), "
               "block 128, seeded per-head stripes (kept-tile density 15-40%)",
    "hunyuan": "HunyuanVideo 720p joint attention: B=1, 24 heads, d=128, grid 33x45x80 + 256 text "
               "(N=119056), block 128, seeded per-head stripes (kept-tile density 10-35%)",
    "sweep": "Wan 2.1 14B shape (B=1, 40 heads, d=128, N=75600), every head forced to one kept-tile "
             "density",
    "wan14b_3d": "Wan 2.1 14B 720p attention layer in the PSABlock-centric layout: B=1, 40 heads, "
                 "d=128, grid 21x45x80 3D-padded to 21x48x80, 3x8x16 PSABlocks, tiles of 128, "
                 "seeded per-head stripes in PSABlock units (PSABlock-pair density 10-40%)",
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
    p.add_argument("--waits", metavar="PMC_DIR",
                   help="wave-cycle breakdown of the attention kernels from a rocprofv3 --pmc run of "
                        "SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY "
                        "SQ_ACTIVE_INST_MISC SQ_ACTIVE_INST_SCA GRBM_GUI_ACTIVE, and exit")
    p.add_argument("--hbm", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "TRACE_DIR"),
                   help="HBM bytes and bandwidth of the sparse and dense kernels of --workload from "
                        "two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) and a kernel trace, and exit")
    p.add_argument("--counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="summarise two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) and exit")
    p.add_argument("--sweep-all", action="store_true",
                   help="sparse at every forced density of the sweep workload against one dense run")
    p.add_argument("--search", type=int, default=0, metavar="K",
                   help="time PSA-Search scoring of K candidates per head (all heads per call)")
    p.add_argument("--gemm-reference", action="store_true",
                   help="time a plain bf16 16384^3 torch.matmul (hipBLASLt): the chip's sustained "
                        "bf16 MFMA rate under its power limit, for comparison")
    p.add_argument("--kernel-stats", metavar="TRACE_DIR",
                   help="print the kernel table of a rocprofv3 --kernel-trace --stats csv run and exit")
    p.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "BENCH_OUT"),
                   help="summarise a rocprofv3 --kernel-trace run of this script (same --steps, "
                        "--warmup, --dense-steps): per-launch durations of the timed legs only, "
                        "and the roofline fraction against the JSON line the run printed to BENCH_OUT; "
                        "then exit")
    p.add_argument("--utilisation", nargs=3, metavar=("SQ_DIR", "TCC_DIR", "TRACE_DIR"),
                   help="print utilisation figures of the attention kernels from two rocprofv3 "
                        "--pmc runs and a kernel trace, and exit")
    p.add_argument("--copy-calibration-mb", type=int, default=1024,
                   help="size of the --copy-mb copy in the profiled runs (for --counters)")
    return p.parse_args()


def source_hash():
    """Hash of the code that builds and launches the kernels: C and C++ sources with their
    comments and whitespace removed (a documentation change keeps the recorded counters), the
    build script as it is."""
    h = hashlib.sha256()
    for rel in SOURCES:
        with open(os.path.join(ROOT, rel)) as f:
            text = f.read()
        if not rel.endswith(".py"):
            text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
            text = re.sub(r"//[^\n]*", " ", text)
            text = " ".join(text.split())
        h.update(text.encode())
    return h.hexdigest()[:16]


def time_calls(fn, steps, warmup, torch):
    """Per-call ms of `steps` back-to-back calls after `warmup`: HIP events recorded on the
    current stream (the stream every library call launches on) between consecutive calls."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return {"mean": ev[0].elapsed_time(ev[-1]) / steps, "median": float(np.median(per)),
            "min": float(min(per))}


def counter_rows(run_dir, counter):
    """{kernel name: [per-dispatch values]} of one counter in a rocprofv3 csv run directory."""
    out = {}
    for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter:
                    out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return out


def summarise_counters(fetch_dir, write_dir, copy_mb):
    """Markdown summary of the two counter runs; HBM bytes of the sparse kernel per launch,
    each counter scaled by what it reads for the plain 'copy_mb' MiB device copy."""
    fetch, write = counter_rows(fetch_dir, "FETCH_SIZE"), counter_rows(write_dir, "WRITE_SIZE")

    def pick(rows, key):
        hits = [v for k, v in rows.items() if key in k]
        if not hits:
            raise SystemExit("no dispatch of %s in the counter runs" % key)
        return hits[0]

    copy_bytes = copy_mb * 1048576.0
    f_copy, w_copy = max(pick(fetch, "copyBuffer")), max(pick(write, "copyBuffer"))
    f_scale, w_scale = copy_bytes / (f_copy * 1024.0), copy_bytes / (w_copy * 1024.0)
    f_k, w_k = pick(fetch, KERNEL), pick(write, KERNEL)
    f_mean, w_mean = sum(f_k) / len(f_k), sum(w_k) / len(w_k)
    traffic = f_mean * 1024.0 * f_scale + w_mean * 1024.0 * w_scale
    lines = [
        "# HBM traffic counters: %s, Wan 2.1 14B shape" % KERNEL,
        "",
        "Workload: B=1, 40 heads, N=75600 (21x45x80), d=128, block 128, seeded stripes "
        "(kept-tile density 0.238).",
        "",
        "Commands (repository root, MI355X; one counter pass per run):",
        "",
        "    cd /tmp && export TMPDIR=/tmp && cd -",
        "    rocprofv3 --pmc FETCH_SIZE --output-format csv -d %s -o run -- "
        "python3 bench.py --steps 2 --warmup 1 --no-dense --no-cpu-baseline --copy-mb %d" % (fetch_dir, copy_mb),
        "    rocprofv3 --pmc WRITE_SIZE --output-format csv -d %s -o run -- "
        "python3 bench.py --steps 2 --warmup 1 --no-dense --no-cpu-baseline --copy-mb %d" % (write_dir, copy_mb),
        "    python3 bench.py --counters %s %s" % (fetch_dir, write_dir),
        "",
        "| quantity | value |",
        "|---|---|",
        "| copy calibration: %d MiB device copy, FETCH_SIZE | %.0f KiB (scale %.4f) |" % (copy_mb, f_copy, f_scale),
        "| copy calibration: %d MiB device copy, WRITE_SIZE | %.0f KiB (scale %.4f) |" % (copy_mb, w_copy, w_scale),
        "| sparse kernel dispatches | %d |" % len(f_k),
        "| FETCH_SIZE per dispatch (raw) | %.0f KiB |" % f_mean,
        "| WRITE_SIZE per dispatch (raw) | %.0f KiB |" % w_mean,
        "| read bytes per launch (scaled) | %.4g |" % (f_mean * 1024.0 * f_scale),
        "| written bytes per launch (scaled) | %.4g |" % (w_mean * 1024.0 * w_scale),
        "",
        "traffic_bytes_per_launch: %.6g" % traffic,
        "source_hash: %s" % source_hash(),
        "",
        "Algorithmic bytes per launch: Q, K, V read once and O written once, "
        "4 x 40 x 75600 x 128 x 2 B = 3.097e9 B.  Traffic above that is K/V tiles that missed "
        "the L2 (each kept tile is streamed once per pair of query blocks).",
    ]
    return "\n".join(lines) + "\n"


def kernel_stats_table(trace_dir):
    """Markdown table of rocprofv3's kernel_stats.csv (durations in microseconds)."""
    paths = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not paths:
        raise SystemExit("no kernel_stats.csv under %s" % trace_dir)
    lines = ["| kernel | calls | total us | average us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    with open(paths[0]) as f:
        for r in csv.DictReader(f):
            name = r["Name"].split("(")[0].replace("void ", "")
            lines.append("| %s | %s | %.1f | %.1f | %.1f | %.1f | %.2f |" % (
                name, r["Calls"], float(r["TotalDurationNs"]) / 1e3, float(r["AverageNs"]) / 1e3,
                float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    return "\n".join(lines) + "\n"


def trace_dispatches(trace_dir):
    """{kernel name: [duration ns in dispatch order]} from rocprofv3's kernel_trace.csv."""
    paths = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not paths:
        raise SystemExit("no kernel_trace.csv under %s" % trace_dir)
    rows = []
    with open(paths[0]) as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"].split("(")[0].replace("void ", "").replace("psa::", "")
            rows.append((int(r["Dispatch_Id"]), name, int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    out = {}
    for _, name, ns in sorted(rows):
        out.setdefault(name, []).append(ns)
    return out


def trace_summary(trace_dir, bench_out, steps, warmup, dense_steps):
    """The kernel launches of each timed leg of a profiled `bench.py` run (the order of main()):
    `warmup` + `steps` psa_attention_fwd calls, then 1 + `steps` psa_attention_run calls, then
    1 + `dense_steps` dense calls; warm-up launches are dropped.  The roofline fraction from the
    trace's mean of the timed run-alone launches is set beside the one the run's JSON line
    reports (HIP events around the same launches)."""
    disp = trace_dispatches(trace_dir)
    sparse = disp.get(KERNEL.replace("psa::", ""), [])
    dense = disp.get(KERNEL.replace("true, false", "false, false"), [])
    expect = warmup + steps + 1 + steps
    if len(sparse) != expect:
        raise SystemExit("%d sparse launches in the trace, %d expected from --steps %d --warmup %d"
                         % (len(sparse), expect, steps, warmup))
    step_leg = sparse[warmup:warmup + steps]
    run_leg = sparse[warmup + steps + 1:]
    dense_leg = dense[1:1 + dense_steps] if len(dense) == 1 + dense_steps else []
    line = None
    with open(bench_out) as f:
        for l in f:
            if l.startswith("{") and '"roofline"' in l:
                line = json.loads(l)
    if line is None:
        raise SystemExit("no JSON line in %s" % bench_out)
    flops = line["config"]["computed_tflop"] * 1e12
    stat = lambda v: (sum(v) / len(v) / 1e6, float(np.median(v)) / 1e6, min(v) / 1e6) if v else (0, 0, 0)
    s_mean, s_med, s_min = stat(step_leg)
    r_mean, r_med, r_min = stat(run_leg)
    d_mean, d_med, d_min = stat(dense_leg)
    frac_trace = flops / (r_mean * 1e-3) / (PEAK_BF16_TFLOPS * 1e12)
    frac_line = line["roofline"]["frac"]
    rows = [
        "| leg | launches | mean ms | median ms | min ms |",
        "|---|---|---|---|---|",
        "| %s in the timed psa_attention_fwd steps | %d | %.3f | %.3f | %.3f |" % (KERNEL, len(step_leg), s_mean, s_med, s_min),
        "| %s in the timed psa_attention_run calls (roofline) | %d | %.3f | %.3f | %.3f |" % (KERNEL, len(run_leg), r_mean, r_med, r_min),
    ]
    if dense_leg:
        rows.append("| %s, timed dense calls | %d | %.3f | %.3f | %.3f |"
                    % (KERNEL.replace("true, false", "false, false"), len(dense_leg), d_mean, d_med, d_min))
    text = "\n".join(rows) + "\n\n"
    text += ("Warm-up launches dropped: %d + 1 sparse, 1 dense.  The same run's JSON line: ms_per_step %.4f, "
             "kernel_ms mean %.4f, roofline frac %.4f.  From the trace: %.4f TFLOP / %.4f ms / %.0f TFLOP/s "
             "= frac %.4f (%+.2f %% against the line).\n"
             % (warmup, line["ms_per_step"], line["kernel_ms"]["mean"], frac_line, flops / 1e12, r_mean,
                PEAK_BF16_TFLOPS, frac_trace, 100.0 * (frac_trace / frac_line - 1.0)))
    return text


def utilisation_rows(sq_dir, tcc_dir, trace_dir, label):
    """Clock, MFMA busy, VALU, LDS and L2 figures of the attention kernels (MI355X: 8 XCDs,
    1024 SIMDs; GRBM_GUI_ACTIVE sums the XCDs)."""
    def per_kernel(run_dir):
        out = {}
        for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                for r in csv.DictReader(f):
                    name = r["Kernel_Name"].split("(")[0].replace("void ", "").replace("psa::", "")
                    if name.startswith(ATTN_PREFIXES):
                        out.setdefault(name, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        return {k: {c: sum(v) / len(v) for c, v in d.items()} for k, d in out.items()}
    sq, tcc = per_kernel(sq_dir), per_kernel(tcc_dir)
    dur = {}
    for path in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                dur[r["Name"].split("(")[0].replace("void ", "").replace("psa::", "")] = float(r["AverageNs"]) * 1e-9
    rows = []
    for k in sorted(sq):
        a, b, t = sq[k], tcc[k], dur[k]
        cyc = a["GRBM_GUI_ACTIVE"] / 8.0
        rows.append("| %s | %s | %.2f | %.2f | %.3f | %.1f | %.2f | %.3f | %.0f | %.3f |" % (
            label, k, t * 1e3, cyc / t / 1e9, a["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * 1024),
            a["SQ_VALU_MFMA_BUSY_CYCLES"] / a["SQ_INSTS_MFMA"],
            (a["SQ_INSTS_VALU"] - a["SQ_INSTS_MFMA"]) / a["SQ_INSTS_MFMA"],   # SQ_INSTS_VALU counts MFMAs
            a["SQ_ACTIVE_INST_VALU"] * 4 / (cyc * 1024), a["SQ_LDS_BANK_CONFLICT"],
            b["TCC_HIT_sum"] / (b["TCC_HIT_sum"] + b["TCC_MISS_sum"])))
    return rows


def hbm_rows(fetch_dir, write_dir, trace_dir, cfg, copy_mb):
    """HBM-side bytes and bandwidth of the attention kernels: FETCH_SIZE and WRITE_SIZE per
    dispatch, each scaled by what it reads for the plain 'copy_mb' MiB device copy of the same
    run, over the kernel's average duration in the trace."""
    fetch, write = counter_rows(fetch_dir, "FETCH_SIZE"), counter_rows(write_dir, "WRITE_SIZE")
    copy_bytes = copy_mb * 1048576.0

    def scale(rows):
        copies = [max(v) for k, v in rows.items() if "copyBuffer" in k]
        if not copies:
            raise SystemExit("no copy dispatch in %s: profile it with --copy-mb" % rows)
        return copy_bytes / (copies[0] * 1024.0)

    f_scale, w_scale = scale(fetch), scale(write)
    dur = {}
    for path in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                dur[r["Name"].split("(")[0].replace("void ", "").replace("psa::", "")] = float(r["AverageNs"]) * 1e-9
    algo = 8.0 * cfg.batch * cfg.heads * cfg.n_tokens * cfg.head_dim
    rows = []
    for full, vals in sorted(fetch.items()):
        k = full.split("(")[0].replace("void ", "").replace("psa::", "")
        if not k.startswith(ATTN_PREFIXES):
            continue
        wv = [v for kk, v in write.items() if kk.split("(")[0].replace("void ", "").replace("psa::", "") == k][0]
        rd = sum(vals) / len(vals) * 1024.0 * f_scale
        wr = sum(wv) / len(wv) * 1024.0 * w_scale
        t = dur[k]
        rows.append("| %s | %s | %.2f | %.1f | %.3f | %.3f | %.0f | %.3f |" % (
            cfg.name, k, t * 1e3, rd / 1e9, wr / 1e9, algo / 1e9, (rd + wr) / t / 1e9, (rd + wr) / t / HBM_PEAK))
    return rows


HBM_HEADER = ("| workload | kernel | ms (trace) | read GB | written GB | algorithmic GB | achieved GB/s | "
              "fraction of 8 TB/s |\n|---|---|---|---|---|---|---|---|")


def wait_rows(run_dir, label):
    """Where the waves of the attention kernels spend their cycles: executing, waiting for a
    dependency (data, waitcnt, barrier), or ready but waiting for the issue port (per-wave
    quad-cycle counters over SQ_WAVE_CYCLES)."""
    out = {}
    for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                name = r["Kernel_Name"].split("(")[0].replace("void ", "").replace("psa::", "")
                if name.startswith(ATTN_PREFIXES):
                    out.setdefault(name, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    rows = []
    for k in sorted(out):
        m = {c: sum(v) / len(v) for c, v in out[k].items()}
        wave = m["SQ_WAVE_CYCLES"]
        rows.append("| %s | %s | %.2f | %.3f | %.3f | %.3f | %.3f | %.3f |" % (
            label, k, wave * 4 / (m["GRBM_GUI_ACTIVE"] / 8.0 * 1024), m["SQ_ACTIVE_INST_ANY"] / wave,
            m["SQ_WAIT_ANY"] / wave, m["SQ_WAIT_INST_ANY"] / wave, m["SQ_ACTIVE_INST_SCA"] / wave,
            m["SQ_ACTIVE_INST_MISC"] / wave))
    return rows


WAIT_HEADER = ("| workload | kernel | waves per SIMD | executing | waiting for a dependency | "
               "waiting for issue | scalar | branch |\n|---|---|---|---|---|---|---|---|")


UTIL_HEADER = ("| workload | kernel | ms (trace) | clock GHz | MFMA busy | MFMA cycles per MFMA | "
               "other VALU insts per MFMA | VALU active | LDS bank-conflict cycles | L2 hit |\n"
               "|---|---|---|---|---|---|---|---|---|---|")


def recorded_traffic():
    """Bytes per launch of the sparse kernel from the committed counter summary, or None when
    the summary is missing or the kernel sources changed since it was taken."""
    try:
        text = open(COUNTERS_MD).read()
    except OSError:
        return None
    vals = dict(l.split(": ", 1) for l in text.splitlines() if l.startswith(("traffic_bytes", "source_hash")))
    if vals.get("source_hash", "").strip() != source_hash():
        return None
    return float(vals["traffic_bytes_per_launch"])


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
    """The oracle on the host cores, on a seeded, stratified sample of (head, query block) rows of
    the same workload: the longest row, the shortest non-empty row, the partial last block, a text
    block if there is one, then seeded random rows until `seconds` have passed (at most 400)."""
    import oracle
    from threadpoolctl import threadpool_info
    from workloads.inputs import make_head_qkv, rope_tables
    bmap = oracle.blockmap(params, cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)
    rows_kept = oracle.kept_per_row(bmap)
    nb = cfg.n_blocks
    lens = np.full(nb, cfg.block, dtype=np.float64)
    lens[-1] = cfg.n_tokens - (nb - 1) * cfg.block
    picks = [tuple(int(x) for x in np.unravel_index(np.argmax(rows_kept), rows_kept.shape))]
    masked = np.where(rows_kept > 0, rows_kept, np.iinfo(np.int32).max)
    picks.append(tuple(int(x) for x in np.unravel_index(np.argmin(masked), rows_kept.shape)))
    picks.append((cfg.heads - 1, nb - 1))
    _, _, _, glob_blk = oracle.block_coordinates(cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)
    if glob_blk.any():
        picks.append((0, int(np.nonzero(glob_blk)[0][0])))
    rng = np.random.default_rng(12345)
    heads = sorted({h for h, _ in picks} | {int(x) for x in rng.choice(cfg.heads, size=min(4, cfg.heads),
                                                                       replace=False)})
    tables = rope_tables(cfg)
    data = {h: make_head_qkv(cfg, 0, h, tables) for h in heads}        # inputs, not timed
    flops = 0.0
    done = []
    t0 = time.perf_counter()
    while len(done) < 400 and (len(done) < len(picks) or time.perf_counter() - t0 < seconds):
        h, qb = picks[len(done)] if len(done) < len(picks) else (heads[int(rng.integers(len(heads)))],
                                                                 int(rng.integers(nb)))
        q, k, v = data[h]
        rows = np.arange(qb * cfg.block, min(cfg.n_tokens, (qb + 1) * cfg.block))
        oracle.masked_attention(q, k, v, bmap[h], cfg.block, cfg.scale, rows)
        flops += 4.0 * cfg.head_dim * lens[qb] * float((bmap[h, qb] * lens).sum())
        done.append((h, qb))
    elapsed = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    full = 4.0 * cfg.head_dim * cfg.batch * float((bmap * lens[None, :, None] * lens[None, None, :]).sum())
    return {
        "value": flops / elapsed / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "extrapolated_full_step_s": round(full / (flops / elapsed), 1),
        "sample": "%d (head, query block) rows of %d tokens of the same workload, stratified (longest row, "
                  "shortest non-empty row, partial last block%s, then seeded random rows), each computed in "
                  "full by the float64 numpy oracle in %.1f s with %d BLAS threads (%d host cores visible); "
                  "%.3g TFLOP, mean %.1f kept blocks per sampled row; random rows from heads %s"
                  % (len(done), cfg.block, ", a text block" if glob_blk.any() else "", elapsed, threads,
                     os.cpu_count() or 0, flops / 1e12, float(np.mean([rows_kept[h, qb] for h, qb in done])),
                     heads),
    }


def group_tokens(cfg):
    """Tokens of every PSABlock (and of the text group) of a 3D workload, host arithmetic."""
    bt, bh, bw = cfg.psablock
    tp, hp, wp = cfg.coarse_grid
    ext = lambda full, b, n: np.minimum(b, full - b * np.arange(n))
    cnt = (ext(cfg.frames, bt, tp)[:, None, None] * ext(cfg.height, bh, hp)[None, :, None]
           * ext(cfg.width, bw, wp)[None, None, :]).ravel().astype(np.float64)
    return np.append(cnt, float(cfg.n_text)) if cfg.n_text else cnt


def bench_3d(args, cfg, params, torch, psa):
    """The PSABlock-centric path: layout conversion, plan + run, conversion back."""
    name = cfg.name
    grid = (cfg.frames, cfg.height, cfg.width, cfg.n_text)
    pb, tile = cfg.psablock, cfg.block
    from workloads import make_qkv
    q, k, v = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to("cuda:0")
               for x in make_qkv(cfg, workers=16))
    qb, kb, vb = (psa.to_blocks(x, grid, pb) for x in (q, k, v))
    ob = torch.empty_like(qb)
    o = torch.empty_like(q)
    ws = psa.Workspace3d(cfg.batch, cfg.heads, grid, pb, tile, q.device)
    bm, _, _ = psa.build_blockmap_3d(params, grid, pb, device=q.device)
    cnt = torch.from_numpy(group_tokens(cfg)).to(q.device)
    flops = 4.0 * cfg.head_dim * cfg.batch * (bm.double() * cnt[None, :, None] * cnt[None, None, :]).sum().item()
    density = bm.double().mean().item()

    def step():
        psa.attention_fwd_3d(qb, kb, vb, grid, pb, params, tile, cfg.scale, out=ob, workspace=ws)

    t_step = time_calls(step, args.steps, args.warmup, torch)
    _, kept = psa.plan_3d(params, grid, pb, tile, batch=cfg.batch, workspace=ws, return_kept_per_tile=True)
    processed = 4.0 * cfg.head_dim * tile * tile * cfg.batch * kept.double().sum().item()

    def kernel_only():
        psa.run_3d(qb, kb, vb, grid, pb, tile, ws, cfg.scale, out=ob)

    t_kernel = time_calls(kernel_only, args.steps, 1, torch)

    def to_layout():
        for x, xb in ((q, qb), (k, kb), (v, vb)):
            psa.to_blocks(x, grid, pb, out=xb)

    def from_layout():
        psa.from_blocks(ob, grid, pb, out=o)

    t_to = time_calls(to_layout, args.steps, 1, torch)
    t_from = time_calls(from_layout, args.steps, 1, torch)
    elem = cfg.batch * cfg.heads * cfg.head_dim * 2.0
    to_bytes = 3 * (cfg.n_tokens + cfg.n_blocked) * elem
    from_bytes = (cfg.n_tokens + cfg.n_blocked) * elem
    ms = t_step["mean"]
    tflops = flops / (ms * 1e-3) / 1e12
    k_tflops = flops / (t_kernel["mean"] * 1e-3) / 1e12
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
        "config": {"workload": WORKLOAD_TEXT[name], "psablock_pair_density": round(density, 5),
                   "computed_tflop": round(flops / 1e12, 4), "processed_tflop": round(processed / 1e12, 4),
                   "blocked_tokens": cfg.n_blocked, "tokens": cfg.n_tokens},
        "mfu": round(tflops / PEAK_BF16_TFLOPS, 4),
        "step_ms": {key: round(val, 4) for key, val in t_step.items()},
        "kernel_ms": {key: round(val, 4) for key, val in t_kernel.items()},
        "padding_overhead": round(processed / flops - 1.0, 4),
        "padded_token_ratio": round(cfg.n_blocked / cfg.n_tokens - 1.0, 4),
        "layout": {"to_blocks_qkv_ms": round(t_to["mean"], 4), "from_blocks_o_ms": round(t_from["mean"], 4),
                   "to_blocks_gbps": round(to_bytes / (t_to["mean"] * 1e-3) / 1e9, 1),
                   "from_blocks_gbps": round(from_bytes / (t_from["mean"] * 1e-3) / 1e9, 1),
                   "hbm_peak_gbps": 8000.0},
    }
    log("3d sparse: %.3f ms/step, kernel %.3f ms, %.1f TFLOP/s computed (%.1f processed), density %.4f, "
        "padding overhead %.3f" % (ms, t_kernel["mean"], tflops, processed / (ms * 1e-3) / 1e12, density,
                                   processed / flops - 1))
    log("layout: to_blocks(q,k,v) %.3f ms (%.0f GB/s), from_blocks(o) %.3f ms (%.0f GB/s)"
        % (t_to["mean"], to_bytes / (t_to["mean"] * 1e-3) / 1e9, t_from["mean"],
           from_bytes / (t_from["mean"] * 1e-3) / 1e9))
    if not args.no_dense:
        def dense():
            psa.dense_fwd(q, k, v, 128, cfg.scale, out=o)
        dms = time_calls(dense, args.dense_steps or max(3, args.steps // 2), 1, torch)["mean"]
        result.update({"dense_ms": round(dms, 4), "speedup_vs_dense": round(dms / ms, 3),
                       "speedup_vs_dense_with_layout": round(dms / (ms + t_to["mean"] + t_from["mean"]), 3)})
        log("dense (original order, unpadded): %.3f ms, speedup %.3f (%.3f with the layout conversions)"
            % (dms, dms / ms, dms / (ms + t_to["mean"] + t_from["mean"])))
    result["roofline"] = {"kernel": KERNEL_3D, "bound": "mfma",
                          "achieved": round(k_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                          "frac": round(k_tflops / PEAK_BF16_TFLOPS, 4), "traffic": None}
    print(json.dumps(result), flush=True)
    return 0


def bench_search(args, cfg, torch, psa):
    """PSA-Search scoring: per candidate, one sparse call for all heads, the L2 reduction
    against the dense output, and the kept counts for the sparsity."""
    from paper_2609_37001_amd import search
    from workloads import make_qkv
    from workloads.candidates import candidates
    grid = (cfg.frames, cfg.height, cfg.width, cfg.n_text)
    q, k, v = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to("cuda:0")
               for x in make_qkv(cfg, workers=16))
    cands = [c[:args.search] for c in candidates(cfg.name, max(args.search, 1))]
    search.score(q, k, v, grid, cfg.block, [c[:1] for c in cands], cfg.scale)        # warm-up
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    res = search.score(q, k, v, grid, cfg.block, cands, cfg.scale)
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end)
    full = psa.dense_fwd(q, k, v, cfg.block, cfg.scale)
    o = torch.empty_like(q)
    t_l2 = time_calls(lambda: psa.l2_distance(o, full), args.steps, 2, torch)
    l2_bytes = 2.0 * q.numel() * 2
    per_cand = ms / args.search
    picks = search.select(res, 0.02)
    result = {
        "metric": "PSA-Search scoring: candidate evaluations per second (all heads per evaluation)",
        "value": round(1e3 / per_cand, 3),
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.search,
        "warmup": 1,
        "ms_per_step": round(per_cand, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[cfg.name] + "; %d candidates per head from the paper's "
                               "candidate space" % args.search,
                   "includes": "dense reference once, per candidate: plan + sparse kernel + L2 + kept counts"},
        "wall_s": round(wall, 3),
        "extrapolated_s_per_100_candidates": round(per_cand * 100 / 1e3, 2),
        "mean_candidate_sparsity": round(float(res.sparsity.mean()), 4),
        "mean_selected_sparsity_alpha_0.02": round(float(np.mean([res.sparsity[h][i] for h, i in enumerate(picks)])), 4),
        "l2_kernel": {"ms": round(t_l2["mean"], 4), "gbps": round(l2_bytes / (t_l2["mean"] * 1e-3) / 1e9, 1),
                      "hbm_peak_gbps": 8000.0},
    }
    log("search: %d candidates x %d heads in %.1f ms (%.2f ms per candidate), L2 kernel %.3f ms (%.0f GB/s)"
        % (args.search, cfg.heads, ms, per_cand, t_l2["mean"], l2_bytes / (t_l2["mean"] * 1e-3) / 1e9))
    print(json.dumps(result), flush=True)
    return 0


def bench_sweep(args, torch, psa):
    """Every density of the sweep workload (the Wan 14B shape), sparse against one dense run."""
    from workloads import get_config, make_qkv, stripe_params
    from workloads.configs import SWEEP_TARGETS
    cfg = get_config("sweep")
    grid = (cfg.frames, cfg.height, cfg.width, cfg.n_text)
    q, k, v = (torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to("cuda:0")
               for x in make_qkv(cfg, workers=16))
    o = torch.empty_like(q)
    ws = psa.Workspace(cfg.batch, cfg.heads, grid, cfg.block, q.device)
    dms = time_calls(lambda: psa.dense_fwd(q, k, v, cfg.block, cfg.scale, out=o), 4, 1, torch)["mean"]
    rows = []
    for target in SWEEP_TARGETS:
        params = stripe_params("sweep", target)
        flops, density = computed_flops(psa, cfg, params, torch)
        t = time_calls(lambda: psa.attention_fwd(q, k, v, grid, cfg.block, params, cfg.scale, out=o,
                                                 workspace=ws), args.steps, args.warmup, torch)
        tf = flops / (t["mean"] * 1e-3) / 1e12
        rows.append({"target": target, "density": round(density, 4), "ms": round(t["mean"], 3),
                     "tflops": round(tf, 1), "speedup_vs_dense": round(dms / t["mean"], 3),
                     "speedup_x_density": round(dms / t["mean"] * density, 3)})
        log("sweep %.2f: density %.4f, %.3f ms, %.1f TFLOP/s, speedup %.2f (x density %.3f)"
            % (target, density, t["mean"], tf, dms / t["mean"], dms / t["mean"] * density))
    best = max(rows, key=lambda r: r["tflops"])
    result = {
        "metric": "sparse-attn fwd computed TFLOP/s & MFU; speedup vs own dense at Wan-14B shape",
        "value": rows[3]["tflops"], "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": rows[3]["ms"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT["sweep"] + "; value is the 30 % run, every run below"},
        "dense_ms": round(dms, 3), "sweep": rows, "best_tflops": best["tflops"],
    }
    print(json.dumps(result), flush=True)
    return 0


def bench_gemm_reference(args, torch):
    """A reference point for the roofline: a plain bf16 16384^3 matrix product through torch
    (hipBLASLt) on random N(0,1) operands, the chip's sustained dense bf16 MFMA rate under the
    same power limit as the attention kernels.  Not part of the attention path."""
    n = 16384
    gen = torch.Generator(device="cuda:0").manual_seed(0)
    a = torch.randn(n, n, device="cuda:0", generator=gen).bfloat16()
    b = torch.randn(n, n, device="cuda:0", generator=gen).bfloat16()
    c = torch.empty(n, n, device="cuda:0", dtype=torch.bfloat16)
    t = time_calls(lambda: torch.matmul(a, b, out=c), args.steps, args.warmup, torch)
    tflops = 2.0 * n ** 3 / (t["mean"] * 1e-3) / 1e12
    log("gemm reference: bf16 %d^3 torch.matmul %.3f ms (median %.3f, min %.3f), %.1f TFLOP/s, %.3f of %.0f"
        % (n, t["mean"], t["median"], t["min"], tflops, tflops / PEAK_BF16_TFLOPS, PEAK_BF16_TFLOPS))
    print(json.dumps({"reference": "bf16 %d^3 torch.matmul (hipBLASLt)" % n, "ms": round(t["mean"], 4),
                      "tflops": round(tflops, 2), "frac_of_peak": round(tflops / PEAK_BF16_TFLOPS, 4)}), flush=True)
    return 0


def main():
    args = parse()
    if args.kernel_stats:
        sys.stdout.write(kernel_stats_table(args.kernel_stats))
        return 0
    if args.trace_summary:
        sys.stdout.write(trace_summary(args.trace_summary[0], args.trace_summary[1], args.steps, args.warmup,
                                       args.dense_steps or max(3, args.steps // 2)))
        return 0
    if args.utilisation:
        label = os.path.basename(os.path.normpath(args.utilisation[0]))
        print(UTIL_HEADER)
        print("\n".join(utilisation_rows(*args.utilisation, label)))
        return 0
    if args.counters:
        sys.stdout.write(summarise_counters(args.counters[0], args.counters[1], args.copy_calibration_mb))
        return 0
    if args.waits:
        print(WAIT_HEADER)
        print("\n".join(wait_rows(args.waits, os.path.basename(os.path.normpath(args.waits)))))
        return 0
    if args.hbm:
        from workloads import get_config
        print(HBM_HEADER)
        print("\n".join(hbm_rows(*args.hbm, get_config(args.workload), args.copy_calibration_mb)))
        return 0
    if args.gpus != 1:
        print("bench.py measures one GPU only: there is no multi-GPU path (the attention would "
              "shard over heads, with one all-to-all before and after). Run with --gpus 1.", file=sys.stderr)
        return 2
    import torch
    if args.gemm_reference:
        return bench_gemm_reference(args, torch)
    import paper_2609_37001_amd as psa
    from workloads import get_config, make_qkv, stripe_params

    name = args.workload
    cfg = get_config(name)
    params = stripe_params(name, args.target if name == "sweep" else None)
    if cfg.psablock is not None:
        return bench_3d(args, cfg, params, torch, psa)
    if args.search:
        return bench_search(args, cfg, torch, psa)
    if args.sweep_all:
        return bench_sweep(args, torch, psa)
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

    t_step = time_calls(sparse, args.steps, args.warmup, torch)
    ms = t_step["mean"]
    tflops = flops / (ms * 1e-3) / 1e12

    # The dominant kernel alone: psa_attention_run over the plan the step above left in ws.
    def kernel_only():
        psa.run(q, k, v, grid, cfg.block, ws, cfg.scale, out=o)

    t_kernel = time_calls(kernel_only, args.steps, 1, torch)
    k_tflops = flops / (t_kernel["mean"] * 1e-3) / 1e12
    props = torch.cuda.get_device_properties(0)
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
        "context_paper": "H100, FA3 baseline, uniform 75 % sparsity at this shape: PSA 55.12 ms, "
                         "29.26 TFLOP, 53.68 % MFU (989 TFLOP/s peak); context only, other hardware "
                         "and workload" if name == "wan14b" else None,
        "step_ms": {key: round(val, 4) for key, val in t_step.items()},
        "kernel_ms": {key: round(val, 4) for key, val in t_kernel.items()},
        "device": {"name": props.name, "arch": getattr(props, "gcnArchName", ""),
                   "compute_units": props.multi_processor_count,
                   "hbm_gib": round(props.total_memory / 2 ** 30, 1)},
        "seeds": {"qkv": 0, "stripes": "workloads/stripe_params.json (seeded density targeting)"},
    }
    log("sparse: %.3f ms/step (median %.3f, min %.3f), %.1f TFLOP/s computed, MFU %.3f, density %.4f"
        % (ms, t_step["median"], t_step["min"], tflops, tflops / PEAK_BF16_TFLOPS, density))
    log("sparse kernel alone: %.3f ms (median %.3f, min %.3f), %.1f TFLOP/s"
        % (t_kernel["mean"], t_kernel["median"], t_kernel["min"], k_tflops))
    if not args.no_dense:
        def dense():
            psa.dense_fwd(q, k, v, cfg.block, cfg.scale, out=o)
        dsteps = args.dense_steps or max(3, args.steps // 2)
        dms = time_calls(dense, dsteps, 1, torch)["mean"]
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
    traffic = recorded_traffic() if name == "wan14b" else None
    result["roofline"] = {
        "kernel": KERNEL,
        "bound": "mfma",
        "achieved": round(k_tflops, 2),
        "peak": PEAK_BF16_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(k_tflops / PEAK_BF16_TFLOPS, 4),
        "traffic": traffic,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline: timing the oracle for about %.0f s" % args.cpu_seconds)
        result["cpu_baseline"] = cpu_baseline(cfg, params, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
