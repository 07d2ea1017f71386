"""Seeded random GPU parity cases: random grids (ragged ends, text), random stripe parameters
from the paper's ranges, every (head_dim, block) variant, batch 1-2; 1D blocks, the pair engine with
both pairing orders of leftover query blocks, and 3D PSABlocks.
Every output row is compared with the oracle."""
import numpy as np
import pytest

import oracle
import paper_2609_37001_amd as psa
from workloads.inputs import bf16_round

import gpu_util as gu

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def dev(x):
    t = gu.torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").bfloat16()


def random_params(rng, n, tmax, smax):
    return [(int(rng.integers(1, tmax + 1)), int(rng.choice([0, 1, -1, 2, -2])), int(rng.choice([1, 2, 3, INF])),
             int(rng.integers(1, smax + 1)), int(rng.choice([0, 1, -1])), int(rng.choice([1, 3, 5, 6, INF])))
            for _ in range(n)]


def compare(q, k, v, keep, scale, o, lse, block=1, groups=None):
    return gu.compare_all(q, k, v, keep, block, scale, o, lse, groups=groups)


@pytest.mark.parametrize("seed", range(8))
def test_random_1d(seed):
    rng = np.random.default_rng([7, seed])
    d = int(rng.choice([64, 128]))
    block = int(rng.choice([64, 128]))
    f, hh, ww = int(rng.integers(1, 5)), int(rng.integers(1, 13)), int(rng.integers(1, 40))
    nt = int(rng.choice([0, 0, int(rng.integers(1, 200))]))
    n = f * hh * ww + nt
    b, heads = int(rng.integers(1, 3)), int(rng.integers(1, 4))
    sp = -(-(hh * ww) // block)
    params = random_params(rng, heads, f, sp)
    scale = float(rng.uniform(0.05, 0.2))
    q, k, v = (bf16_round(rng.standard_normal((b, heads, n, d)).astype(np.float32)) for _ in range(3))
    o, lse = psa.attention_fwd(dev(q), dev(k), dev(v), (f, hh, ww, nt), block, params, scale, return_lse=True)
    gu.torch().cuda.synchronize()
    keep = oracle.blockmap(params, f, hh, ww, nt, block)
    compare(q, k, v, keep, scale, o.float().cpu().numpy(), lse.cpu().numpy(), block=block).check(
        "seed %d: n=%d d=%d block=%d:" % (seed, n, d, block))


@pytest.mark.parametrize("seed", range(6))
def test_random_3d(seed):
    rng = np.random.default_rng([8, seed])
    d = int(rng.choice([64, 128]))
    tile = int(rng.choice([64, 128]))
    shapes = [(1, 4, 16), (2, 4, 16), (1, 8, 16), (2, 8, 8), (3, 8, 16), (4, 4, 8), (1, 2, 64)]
    pb = [s for s in shapes if (s[0] * s[1] * s[2]) % tile == 0][int(rng.integers(0, 3))]
    f = int(rng.integers(1, 2 * pb[0] + 2))
    hh = int(rng.integers(1, 2 * pb[1] + 3))
    ww = int(rng.integers(1, 2 * pb[2] + 3))
    nt = int(rng.choice([0, int(rng.integers(1, 100))]))
    (tp, hp, wp), _ = oracle.psablock_grid(f, hh, ww, pb)
    heads = int(rng.integers(1, 4))
    params = random_params(rng, heads, tp, hp * wp)
    scale = float(rng.uniform(0.05, 0.2))
    n = f * hh * ww + nt
    q, k, v = (bf16_round(rng.standard_normal((1, heads, n, d)).astype(np.float32)) for _ in range(3))
    grid = (f, hh, ww, nt)
    qb, kb, vb = (psa.to_blocks(dev(x), grid, pb) for x in (q, k, v))
    ob, lseb = psa.attention_fwd_3d(qb, kb, vb, grid, pb, params, tile, scale, return_lse=True)
    o = psa.from_blocks(ob, grid, pb)
    gu.torch().cuda.synchronize()
    lse = np.stack([oracle.from_blocks(lseb[0, h].cpu().numpy()[:, None], f, hh, ww, nt, pb)[:, 0]
                    for h in range(heads)])[None]
    keep = oracle.psablock_map(params, f, hh, ww, nt, pb)
    groups = oracle.token_groups(f, hh, ww, nt, pb)
    compare(q, k, v, keep, scale, o.float().cpu().numpy(), lse, groups=groups).check(
        "seed %d: grid %s pb %s tile %d d %d:" % (seed, grid, pb, tile, d))


def slot_major(m):
    """Whether the plan pairs a head's leftover query blocks slot-major (the kernel's rule)."""
    tw, _, ts, sw, _, ss = m
    return sw < ss and (tw >= ts or tw > sw)


@pytest.mark.parametrize("seed", range(6))
def test_random_pair_engine(seed):
    """Block 128 (the pair engine) on random grids with heads of both leftover pairing orders
    (index and slot-major), odd and even block counts, text and batch 1-2."""
    rng = np.random.default_rng([9, seed])
    d = int(rng.choice([64, 128]))
    f, hh, ww = int(rng.integers(2, 6)), int(rng.integers(4, 17)), int(rng.integers(8, 48))
    nt = int(rng.choice([0, int(rng.integers(1, 300))]))
    n = f * hh * ww + nt
    sp = -(-(hh * ww) // 128)
    params = random_params(rng, 2, f, sp)
    params += [(min(f, 3), 0, INF, 1, 0, 3), (1, 0, INF, min(sp, 2), 0, INF)]   # slot-major, index order
    b = int(rng.integers(1, 3))
    scale = float(rng.uniform(0.05, 0.2))
    q, k, v = (bf16_round(rng.standard_normal((b, len(params), n, d)).astype(np.float32)) for _ in range(3))
    o, lse, kept = psa.attention_fwd(dev(q), dev(k), dev(v), (f, hh, ww, nt), 128, params, scale, return_lse=True,
                                     return_kept_per_row=True)
    gu.torch().cuda.synchronize()
    keep = oracle.blockmap(params, f, hh, ww, nt, 128)
    assert np.array_equal(kept.cpu().numpy(), oracle.kept_per_row(keep))
    assert any(slot_major(m) for m in params) and not all(slot_major(m) for m in params)
    compare(q, k, v, keep, scale, o.float().cpu().numpy(), lse.cpu().numpy(), block=128).check(
        "seed %d: n=%d nb=%d d=%d b=%d:" % (seed, n, keep.shape[1], d, b))
