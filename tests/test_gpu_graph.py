"""HIP graph capture: the plan, the run and the dense kernel enqueue kernels only (no memset,
allocation or synchronisation), so a caller can capture them once and replay them.  Every replay,
with eager work and synchronisations between replays, matches the eager result bit for bit, and
follows new data written into the captured input buffers."""
import numpy as np
import pytest

import paper_2609_37001_amd as psa
from workloads.inputs import bf16_round

import gpu_util as gu

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def dev(x):
    t = gu.torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").bfloat16()


@pytest.mark.parametrize("block", [64, 128])
def test_graph_replays_match_eager(block):
    torch = gu.torch()
    f, hh, ww, nt, d = 3, 16, 24, 40, 128
    n = f * hh * ww + nt
    grid = (f, hh, ww, nt)
    params = [(1, 0, 2, 2, 0, 3), (2, 1, INF, 1, 0, INF), (1, 0, INF, 1, 0, INF)]
    rng = np.random.default_rng(block)
    q, k, v = (dev(bf16_round(rng.standard_normal((1, len(params), n, d)).astype(np.float32)))
               for _ in range(3))
    q_next = dev(bf16_round(rng.standard_normal((1, len(params), n, d)).astype(np.float32)))

    def eager():
        o_s = psa.attention_fwd(q, k, v, grid, block, params, 0.1)
        o_d = psa.dense_fwd(q, k, v, block, 0.1)
        torch.cuda.synchronize()
        return o_s, o_d

    ref_s, ref_d = eager()
    o_s, o_d = torch.empty_like(q), torch.empty_like(q)
    ws = psa.Workspace(1, len(params), grid, block, q.device)
    ws_run = psa.plan(params, grid, block)                      # planned eagerly, run in the graph
    o_r = torch.empty_like(q)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        psa.attention_fwd(q, k, v, grid, block, params, 0.1, out=o_s, workspace=ws)
        psa.run(q, k, v, grid, block, ws_run, 0.1, out=o_r)
        psa.dense_fwd(q, k, v, block, 0.1, out=o_d)
    for replay in range(4):
        for t in (o_s, o_r, o_d):
            t.zero_()
        psa.dense_fwd(k, q, v, block, 0.2)                      # eager library work in between
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_s, ref_s), "replay %d: plan + run differs from eager" % replay
        assert torch.equal(o_r, ref_s), "replay %d: run differs from eager" % replay
        assert torch.equal(o_d, ref_d), "replay %d: dense differs from eager" % replay
    q.copy_(q_next)
    ref_s, ref_d = eager()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(o_s, ref_s) and torch.equal(o_r, ref_s) and torch.equal(o_d, ref_d)
    assert not torch.equal(o_s, o_d)                            # the stripes are sparse
