"""Per-head stripe parameters M = (T_w, T_o, T_s, S_w, S_o, S_s) for each workload.

Units: temporal parameters count frames, spatial parameters count block slots within a frame
(a frame of H*W tokens holds ceil(H*W / block) slots); for the PSABlock workload they count
PSABlocks along time and PSABlocks of the H' x W' plane.  The candidate ranges are the paper's
(appendix, "Initialization of Mask Candidates"): T_o in {0,+-1,+-2}, T_s in {1,2,3,inf},
S_o in {0,+-1}, S_s in {1,3,5,6,inf}; widths run from 1 to the extent of the axis.
An infinite stride is encoded as STRIDE_INF = 2^31 - 1.

* ``tiny``: every parameter drawn uniformly from those sets with ``default_rng([1, 0])``.
* the other workloads: density-targeted tuples stored in ``stripe_params.json``, which
  ``make_stripe_params.py`` writes (it evaluates densities with the oracle).
"""
import json
import os

import numpy as np

STRIDE_INF = 2 ** 31 - 1
T_OFFSETS = (0, 1, -1, 2, -2)
T_STRIDES = (1, 2, 3, STRIDE_INF)
S_OFFSETS = (0, 1, -1)
S_STRIDES = (1, 3, 5, 6, STRIDE_INF)

_JSON = os.path.join(os.path.dirname(os.path.abspath(__file__)), "stripe_params.json")


def coarse_extent(cfg):
    """(T', S'): frames and block slots per frame; with PSABlocks, PSABlocks along time and
    PSABlocks of the H' x W' plane."""
    if cfg.psablock is not None:
        tp, hp, wp = cfg.coarse_grid
        return tp, hp * wp
    return cfg.frames, -(-(cfg.height * cfg.width) // cfg.block)


def uniform_draw(cfg, n_heads, seed):
    """Uniform draws from the candidate sets (widths 1..extent)."""
    rng = np.random.default_rng(seed)
    tp, sp = coarse_extent(cfg)
    out = []
    for _ in range(n_heads):
        out.append((int(rng.integers(1, tp + 1)), int(rng.choice(T_OFFSETS)), int(rng.choice(T_STRIDES)),
                    int(rng.integers(1, sp + 1)), int(rng.choice(S_OFFSETS)), int(rng.choice(S_STRIDES))))
    return out


def load_json():
    with open(_JSON) as f:
        return json.load(f)


def stripe_params(name, target=None):
    """List of per-head 6-tuples for workload ``name`` (``target`` selects a sweep density)."""
    from .configs import get_config
    cfg = get_config(name)
    if name == "tiny":
        return uniform_draw(cfg, cfg.heads, [1, 0])
    data = load_json()
    if name == "sweep":
        key = "%.2f" % (1.0 if target is None else target)
        return [tuple(m) for m in data["sweep"][key]["params"]]
    return [tuple(m) for m in data[name]["params"]]
