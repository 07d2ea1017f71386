"""Helpers shared by the GPU parity tests: device inputs, sampled oracle comparison, metrics."""
import functools
import math

import numpy as np

import oracle
from workloads import get_config, make_head_qkv, make_qkv, stripe_params
from workloads.inputs import bf16_round, rope_tables

REL_L2_TOL = 1e-2      # relative L2 error of O against the oracle
MAX_ABS_TOL = 3e-2     # max absolute error of O against the oracle
# Absolute error of the natural-log normaliser against the oracle evaluated on the kernel's own
# operand (kernel_q): the kernel sums the bf16-rounded weights into l.  bf16 keeps 8 significant
# bits, so each weight, and hence the sum, is off by a relative 2^-8 at most:
# ln(1 + 2^-8) = 3.9e-3; 4e-3 with fp32 accumulation and the exp2/log2 approximations.
LSE_ABS_TOL = 4e-3
LN2 = math.log(2.0)


def kernel_q(q, scale):
    """The operand the kernel multiplies K by: q * (scale * log2(e)), formed in fp32 as the
    library does and rounded to bf16 (include/psa.h, Numerics).  The oracle with softmax scale
    ln 2 evaluated on it is the kernel's exp2-domain softmax of exactly these inputs."""
    c = np.float32(scale) * np.float32(1.4426950408889634)
    return bf16_round(np.asarray(q, dtype=np.float32) * c)


def torch():
    import torch as t
    return t


@functools.lru_cache(maxsize=2)
def device_qkv(name):
    """Q, K, V of workload `name` on cuda:0 as bf16 [B, H, N, d]."""
    t = torch()
    cfg = get_config(name)
    out = []
    for x in make_qkv(cfg, workers=16):
        out.append(t.from_numpy(x.view(np.int16)).view(t.bfloat16).to("cuda:0"))
        del x
    return tuple(out)


def grid_of(cfg):
    return (cfg.frames, cfg.height, cfg.width, cfg.n_text)


def oracle_map(cfg, params):
    return oracle.blockmap(params, cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)


def sample_blocks(cfg, bmap, n_random=6, seed=0):
    """(head, query block) pairs: longest and shortest non-empty rows, an empty row if any, the
    last (possibly partial) block, a text block if any, and seeded random ones."""
    rows = oracle.kept_per_row(bmap)
    nb = rows.shape[1]
    picks = []
    h, q = np.unravel_index(np.argmax(rows), rows.shape)
    picks.append((int(h), int(q)))
    masked = np.where(rows > 0, rows, np.iinfo(np.int32).max)
    h, q = np.unravel_index(np.argmin(masked), rows.shape)
    picks.append((int(h), int(q)))
    empty = np.argwhere(rows == 0)
    if len(empty):
        picks.append(tuple(int(x) for x in empty[len(empty) // 2]))
    picks.append((int(cfg.heads - 1), nb - 1))
    _, _, _, g = oracle.block_coordinates(cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)
    if g.any():
        picks.append((0, int(np.nonzero(g)[0][0])))
    rng = np.random.default_rng(seed)
    for _ in range(n_random):
        picks.append((int(rng.integers(cfg.heads)), int(rng.integers(nb))))
    return list(dict.fromkeys(picks))


def compare_rows(cfg, params, bmap, o_dev, lse_dev, picks, batch=0):
    """Oracle rows of the sampled (head, query block) pairs against the device output.

    Returns (rel_l2, max_abs, max_abs_lse) pooled over every sampled row."""
    tables = rope_tables(cfg)
    num = den = 0.0
    max_abs = max_lse = 0.0
    by_head = {}
    for h, qb in picks:
        by_head.setdefault(h, []).append(qb)
    for h, qbs in by_head.items():
        q, k, v = make_head_qkv(cfg, batch, h, tables)
        rows = np.concatenate([np.arange(qb * cfg.block, min(cfg.n_tokens, (qb + 1) * cfg.block))
                               for qb in qbs])
        o_ref, _ = oracle.masked_attention(q, k, v, bmap[h], cfg.block, cfg.scale, rows)
        o = o_dev[batch, h, rows].float().cpu().numpy().astype(np.float64)
        num += float(((o - o_ref) ** 2).sum())
        den += float((o_ref ** 2).sum())
        max_abs = max(max_abs, float(np.abs(o - o_ref).max()))
        if lse_dev is not None:
            _, lse_ref = oracle.masked_attention(kernel_q(q, cfg.scale), k, v, bmap[h], cfg.block,
                                                 LN2, rows)
            lse = lse_dev[batch, h, rows].cpu().numpy().astype(np.float64)
            fin = np.isfinite(lse_ref)
            assert (np.isneginf(lse) == ~fin).all(), "empty rows must give lse = -inf"
            if fin.any():
                max_lse = max(max_lse, float(np.abs(lse[fin] - lse_ref[fin]).max()))
            assert (o[~fin] == 0).all(), "empty rows must give o = 0"
    rel = (num / den) ** 0.5 if den > 0 else (0.0 if num == 0 else float("inf"))
    return rel, max_abs, max_lse


def params_of(name, target=None):
    return stripe_params(name, target)
