"""psa_attention_fwd_noalloc through the C ABI against psa_attention_fwd with a workspace: the
same kernels over the same plan, so the same bits (O, LSE and the kept counts), on two calls in a
row on one GPU, the second with a smaller input (the scratch keeps the first call's plan, which
the second must replace)."""
import ctypes

import numpy as np
import pytest

import paper_2609_37001_amd as psa
from paper_2609_37001_amd import _lib
from workloads.inputs import bf16_round

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def raw_noalloc(q, k, v, o, grid, block, params, scale, lse, kept):
    import torch
    b, h, _, d = q.shape
    vp = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return _lib.lib().psa_attention_fwd_noalloc(vp(q), vp(k), vp(v), vp(o), b, h, d, _lib.grid_of(*grid), block,
                                                _lib.stripes(params), scale, vp(lse), vp(kept), stream)


CASES = [
    # batch, grid (F, H, W, text), block, head_dim, stripes: the larger call first
    (2, (6, 24, 40, 77), 128, 128, [(2, 0, INF, 3, 1, 5), (1, 0, 2, 2, -1, 3), (1, 1, INF, 1, 0, INF),
                                    (6, 0, INF, 8, 0, INF), (3, -1, 3, 2, 0, INF)]),
    (1, (3, 10, 13, 37), 64, 64, [(1, 0, INF, 1, 0, INF), (2, 1, 3, 2, -1, 3), (1, 1, INF, 1, 0, INF)]),
]


def test_noalloc_equals_workspace_entry_point():
    import torch
    for i, (b, grid, block, d, params) in enumerate(CASES):
        f, hh, ww, nt = grid
        n = f * hh * ww + nt
        h = len(params)
        nb = psa.num_blocks(grid, block)
        assert psa.workspace_size(b, h, grid, block) <= _lib.NOALLOC_SCRATCH_BYTES
        rng = np.random.default_rng(100 + i)
        q, k, v = (torch.from_numpy(bf16_round(rng.standard_normal((b, h, n, d)).astype(np.float32)))
                   .to("cuda:0").bfloat16() for _ in range(3))
        ref, ref_lse, ref_kept = psa.attention_fwd(q, k, v, grid, block, params, 0.1, return_lse=True,
                                                   return_kept_per_row=True)
        o = torch.full_like(q, float("nan"))
        lse = torch.full((b, h, n), float("nan"), device="cuda:0")
        kept = torch.full((h, nb), -1, dtype=torch.int32, device="cuda:0")
        print("case %d: batch %d, grid %s, block %d, d %d, %d heads" % (i, b, grid, block, d, h), flush=True)
        assert raw_noalloc(q, k, v, o, grid, block, params, 0.1, lse, kept) == _lib.PSA_OK
        torch.cuda.synchronize()
        assert torch.equal(o, ref) and torch.equal(lse, ref_lse) and torch.equal(kept, ref_kept)
        # the binding's wrapper over the same entry point
        o2 = torch.empty_like(q)
        psa.attention_fwd_noalloc(q, k, v, grid, block, params, o2, 0.1)
        torch.cuda.synchronize()
        assert torch.equal(o2, ref)
