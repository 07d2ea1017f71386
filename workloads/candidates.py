"""Candidate masks of PSA-Search: about 100 configurations per head, drawn uniformly from the
paper's candidate space (appendix "Initialization of Mask Candidates": T_o in {0,+-1,+-2},
T_s in {1,2,3,inf}, S_o in {0,+-1}, S_s in {1,3,5,6,inf}; widths 1..extent of the axis), as the
experiments sample about 100 per head (Sec. 4 setup).  Seeded per head with
``default_rng([2, config index, head])``; distinct tuples, in draw order."""
import numpy as np

from .configs import CONFIGS
from .params import S_OFFSETS, S_STRIDES, T_OFFSETS, T_STRIDES, coarse_extent


def candidates(name, n_candidates=100):
    """List over heads of lists of n_candidates distinct 6-tuples."""
    cfg = CONFIGS[name]
    index = list(CONFIGS).index(name)
    tp, sp = coarse_extent(cfg)
    space = tp * len(T_OFFSETS) * len(T_STRIDES) * sp * len(S_OFFSETS) * len(S_STRIDES)
    if n_candidates > space:
        raise ValueError("only %d distinct candidates exist" % space)
    out = []
    for h in range(cfg.heads):
        rng = np.random.default_rng([2, index, h])
        seen, head = set(), []
        while len(head) < n_candidates:
            m = (int(rng.integers(1, tp + 1)), int(rng.choice(T_OFFSETS)), int(rng.choice(T_STRIDES)),
                 int(rng.integers(1, sp + 1)), int(rng.choice(S_OFFSETS)), int(rng.choice(S_STRIDES)))
            if m not in seen:
                seen.add(m)
                head.append(m)
        out.append(head)
    return out
