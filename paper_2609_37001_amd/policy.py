"""Timestep policy of the sparse attention (Sec. 4, setup: the first 20 % of the denoising steps
are exempt from sparsification, since the early steps lay out the coarse structure).

LayerAttention is the per-layer runtime piece: it plans the layer's stripes once (the plan
depends only on the sizes and the stripes, which stay fixed over the steps) and, at each step,
runs the dense kernel during the exempt steps and the planned sparse kernel afterwards.
"""
import math

from . import dense_fwd, plan, run


class TimestepPolicy:
    """Dense for the first ceil(dense_fraction * total_steps) steps (step indices from 0)."""

    def __init__(self, total_steps, dense_fraction=0.2):
        if total_steps < 1 or not 0.0 <= dense_fraction <= 1.0:
            raise ValueError("total_steps >= 1 and 0 <= dense_fraction <= 1 are required")
        self.total_steps = int(total_steps)
        self.dense_fraction = float(dense_fraction)
        # a tolerance keeps exact products such as 0.2 * 50 = 10 from rounding up to 11
        self.dense_steps = min(self.total_steps, math.ceil(self.dense_fraction * self.total_steps - 1e-9))

    def is_dense(self, step):
        if not 0 <= step < self.total_steps:
            raise ValueError("step %d outside [0, %d)" % (step, self.total_steps))
        return step < self.dense_steps


class LayerAttention:
    """One attention layer under a timestep policy: q, k, v bf16 [batch, heads, N, d]."""

    def __init__(self, params, grid, block, batch, policy, scale=None, device=None):
        self.params = [tuple(int(x) for x in m) for m in params]
        self.grid, self.block, self.batch, self.scale = grid, int(block), int(batch), scale
        self.policy = policy
        self.workspace = None
        self.device = device

    def _planned(self, device, stream):
        # The plan is enqueued on the stream of the run that first needs it, so the run follows
        # it; a later run on another stream is ordered by the caller, as for any input.
        if self.workspace is None:
            self.workspace = plan(self.params, self.grid, self.block, batch=self.batch, device=device,
                                  stream=stream)
        return self.workspace

    def __call__(self, q, k, v, step, out=None, stream=None):
        if self.policy.is_dense(step):
            return dense_fwd(q, k, v, self.block, self.scale, out=out, stream=stream)
        return run(q, k, v, self.grid, self.block, self._planned(q.device, stream), self.scale,
                   out=out, stream=stream)
