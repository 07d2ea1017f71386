"""CPU oracle for PSA block-sparse attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import this package.  It shares no code with the HIP library (``paper_2609_37001_amd``) and
imports nothing from it.  Everything here is plain numpy, computed in float64:

* ``stripe``    -- the stripe-to-mask definition: Algorithm 1 (IsAttending) of the paper's
                   Sec. 3.2, evaluated on block coordinates (masking at PSABlock granularity,
                   Sec. 3.2 "Hardware-Aware Design").
* ``attention`` -- naive masked softmax attention: exact softmax attention restricted to the
                   kept blocks, with padded keys excluded (Algorithm 2's consumer body computes
                   exactly this up to rounding).
* ``psablock``  -- 3D PSABlocks with 3D padding (Sec. 3.2): the PSABlock grid, the group of
                   every original token, Algorithm 1 on the PSABlock grid, and the
                   PSABlock-centric (T', H', W', bt, bh, bw) layout.
* ``search``    -- PSA-Search (Algorithm 3) and its dual interface: per-head relative L2 loss
                   of a candidate against full attention, and the selection rules.

Every function is pinned by tests against values fixed by the paper and by mathematics
(hand-worked maps, closed-form counts, symmetry and periodicity invariants, library softmax
attention, brute force on tiny inputs); see the ``tests/test_oracle_*.py`` files.
"""
from .stripe import (STRIDE_INF, axis_condition, is_attending, block_coordinates,  # noqa: F401
                     blockmap, kept_per_row, kept_per_head)
from .attention import masked_attention  # noqa: F401
from .psablock import (psablock_grid, token_groups, group_coordinates,  # noqa: F401
                       psablock_map, to_blocks, from_blocks)
from . import search  # noqa: F401
