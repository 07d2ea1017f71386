"""GPU parity of the 3D PSABlock path (layout, PSABlock maps, plan counts, attention with 3D
padding) against the oracle, which works on the original token order with no padding at all."""
import numpy as np
import pytest

import oracle
import paper_2609_37001_amd as psa
from workloads import get_config, stripe_params
from workloads.inputs import bf16_round

import gpu_util as gu
import golden_maps

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def dev(x):
    t = gu.torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").bfloat16()


def random_params(seed, n, tmax, smax):
    rng = np.random.default_rng(seed)
    return [(int(rng.integers(1, tmax + 1)), int(rng.choice([0, 1, -1, 2, -2])), int(rng.choice([1, 2, 3, INF])),
             int(rng.integers(1, smax + 1)), int(rng.choice([0, 1, -1])), int(rng.choice([1, 3, 5, 6, INF])))
            for _ in range(n)]


@pytest.mark.parametrize("grid,pb,d", [((3, 5, 7, 4), (2, 2, 3), 128), ((4, 10, 20, 0), (3, 8, 16), 64),
                                       ((5, 3, 9, 65), (1, 4, 16), 128), ((21, 45, 80, 0), (3, 8, 16), 128)])
def test_layout_matches_oracle_and_round_trips(grid, pb, d):
    f, h, w, nt = grid
    n = f * h * w + nt
    heads = 2 if n < 10000 else 1
    x = bf16_round(np.random.default_rng(n).standard_normal((1, heads, n, d)).astype(np.float32))
    xb = psa.to_blocks(dev(x), grid, pb)
    back = psa.from_blocks(xb, grid, pb)
    gu.torch().cuda.synchronize()
    xbn = xb.float().cpu().numpy()
    for hh in range(heads):
        assert np.array_equal(xbn[0, hh], oracle.to_blocks(x[0, hh], f, h, w, nt, pb))
    assert np.array_equal(back.float().cpu().numpy(), x)


@pytest.mark.parametrize("case", golden_maps.load(golden_maps.PSABLOCK_PATH), ids=lambda c: c["name"])
def test_golden_psablock_maps_on_gpu(case):
    f, h, w, nt = case["grid"]
    bm, per_row, per_head = psa.build_blockmap_3d([case["m"]], (f, h, w, nt), case["pb"], device="cuda:0")
    gu.torch().cuda.synchronize()
    ref = oracle.psablock_map([case["m"]], f, h, w, nt, case["pb"])
    assert np.array_equal(bm.cpu().numpy(), ref)
    assert int(per_head.item()) == case["kept"]
    assert np.array_equal(per_row.cpu().numpy(), ref.sum(2).astype(np.int32))


@pytest.mark.parametrize("grid,pb", [((3, 5, 7, 4), (2, 2, 3)), ((21, 45, 80, 0), (3, 8, 16)),
                                     ((33, 45, 80, 256), (3, 8, 16))])
def test_random_psablock_maps_on_gpu(grid, pb):
    f, h, w, nt = grid
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    params = random_params(tp * hp, 24, tp, hp * wp)
    bm, _, _ = psa.build_blockmap_3d(params, grid, pb, device="cuda:0")
    gu.torch().cuda.synchronize()
    assert np.array_equal(bm.cpu().numpy(), oracle.psablock_map(params, f, h, w, nt, pb))


def tile_groups(f, h, w, nt, pb, tile):
    """Group of every tile of the blocked layout and whether it holds a token (oracle only)."""
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    vol = pb[0] * pb[1] * pb[2]
    valid = oracle.to_blocks(np.ones((f * h * w + nt, 1)), f, h, w, nt, pb)[:, 0] > 0
    n_b = valid.shape[0]
    nt_tiles = -(-n_b // tile)
    pos = np.arange(nt_tiles) * tile
    group = np.where(pos < tp * hp * wp * vol, pos // vol, tp * hp * wp)
    live = np.array([valid[p:p + tile].any() for p in pos])
    return group, live


@pytest.mark.parametrize("grid,pb,tile", [((4, 10, 20, 0), (3, 8, 16), 128), ((3, 6, 20, 40), (2, 4, 16), 64),
                                          ((21, 45, 80, 0), (3, 8, 16), 128)])
def test_plan_counts_per_tile(grid, pb, tile):
    f, h, w, nt = grid
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    params = random_params(7, 6, tp, hp * wp) + [(tp, 0, INF, hp * wp, 0, INF)]
    ws, kept = psa.plan_3d(params, grid, pb, tile, return_kept_per_tile=True)
    gu.torch().cuda.synchronize()
    keep = oracle.psablock_map(params, f, h, w, nt, pb).astype(bool)
    group, live = tile_groups(f, h, w, nt, pb, tile)
    expect = (keep[:, group][:, :, group] & live[None, None, :] & live[None, :, None]).sum(2)
    assert np.array_equal(kept.cpu().numpy(), expect.astype(np.int32))


def compare_3d(q, k, v, grid, pb, params, scale, o, lse):
    """O and LSE in the original order against the oracle (gpu_util.Parity)."""
    f, h, w, nt = grid
    keep = oracle.psablock_map(params, f, h, w, nt, pb)
    groups = oracle.token_groups(f, h, w, nt, pb)
    return gu.compare_all(q, k, v, keep, 1, scale, o, lse, groups=groups)


@pytest.mark.parametrize("d,tile,grid,pb", [
    (128, 128, (3, 6, 20, 40), (2, 4, 16)),     # padding on every axis, text, 1 tile per PSABlock
    (64, 64, (3, 6, 20, 40), (2, 4, 16)),       # 2 tiles per PSABlock
    (128, 64, (4, 10, 20, 13), (1, 4, 16)),
    (64, 128, (4, 10, 20, 0), (3, 8, 16)),      # 3 tiles per PSABlock, tiles of padding only
])
def test_attention_3d_against_oracle(d, tile, grid, pb):
    f, h, w, nt = grid
    n = f * h * w + nt
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    params = [(1, 1, INF, 1, 0, INF), (2, 0, INF, 3, 1, 5), (1, 0, 2, 2, -1, 3), (tp, 0, INF, hp * wp, 0, INF)]
    rng = np.random.default_rng(d + tile)
    q, k, v = (bf16_round(rng.standard_normal((2, len(params), n, d)).astype(np.float32)) for _ in range(3))
    qb, kb, vb = (psa.to_blocks(dev(x), grid, pb) for x in (q, k, v))
    ob, lseb = psa.attention_fwd_3d(qb, kb, vb, grid, pb, params, tile, scale=0.11, return_lse=True)
    o = psa.from_blocks(ob, grid, pb)
    gu.torch().cuda.synchronize()
    lse_b = lseb.cpu().numpy()
    lse = np.stack([np.stack([oracle.from_blocks(lse_b[bi, hi][:, None], f, h, w, nt, pb)[:, 0]
                              for hi in range(len(params))]) for bi in range(2)])
    compare_3d(q, k, v, grid, pb, params, 0.11, o.float().cpu().numpy(), lse).check(
        "3d d=%d tile=%d:" % (d, tile))


def test_attention_3d_plan_reuse_and_deterministic():
    grid, pb, tile = (4, 10, 20, 0), (3, 8, 16), 128
    n = 4 * 10 * 20
    params = [(1, 0, INF, 4, 0, INF), (2, -1, 3, 2, 1, 6)]
    rng = np.random.default_rng(11)
    q, k, v = (psa.to_blocks(dev(bf16_round(rng.standard_normal((1, 2, n, 128)).astype(np.float32))), grid, pb)
               for _ in range(3))
    ws = psa.plan_3d(params, grid, pb, tile)
    a = psa.run_3d(q, k, v, grid, pb, tile, ws, 0.1)
    b = psa.run_3d(q, k, v, grid, pb, tile, ws, 0.1)
    c = psa.attention_fwd_3d(q, k, v, grid, pb, params, tile, 0.1)
    gu.torch().cuda.synchronize()
    assert gu.torch().equal(a, b) and gu.torch().equal(a, c)


def test_wan14b_psablock_workload_sampled():
    """The Wan 2.1 14B layer in the paper's layout (3x8x16 PSABlocks, 21x48x80 after padding) in
    the launch configuration the benchmark times: sampled query rows against the oracle."""
    cfg = get_config("wan14b_3d")
    params = stripe_params("wan14b_3d")
    grid = gu.grid_of(cfg)
    q, k, v = gu.device_qkv("wan14b")
    qb, kb, vb = (psa.to_blocks(x, grid, cfg.psablock) for x in (q, k, v))
    ob, lseb = psa.attention_fwd_3d(qb, kb, vb, grid, cfg.psablock, params, cfg.block, cfg.scale,
                                    return_lse=True)
    o = psa.from_blocks(ob, grid, cfg.psablock)
    gu.torch().cuda.synchronize()
    del qb, kb, vb
    keep = oracle.psablock_map(params, cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.psablock)
    groups = oracle.token_groups(cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.psablock)
    from workloads import make_head_qkv
    from workloads.inputs import rope_tables
    tables = rope_tables(cfg)
    rng = np.random.default_rng(0)
    # rows: a padded-edge row (h = 44), the first and last token, and seeded random ones
    picks = [(0, 44 * 80 + 3), (7, 0), (cfg.heads - 1, cfg.n_tokens - 1)]
    picks += [(int(rng.integers(cfg.heads)), int(rng.integers(cfg.n_tokens))) for _ in range(5)]
    lse_b = lseb.cpu().numpy()
    par = gu.Parity()
    for h, i in picks:
        qh, kh, vh = make_head_qkv(cfg, 0, h, tables)
        rows = np.arange(max(0, i - 63), min(cfg.n_tokens, i + 65))
        og = o[0, h, rows].float().cpu().numpy()
        lse_orig = oracle.from_blocks(lse_b[0, h][:, None], cfg.frames, cfg.height, cfg.width, cfg.n_text,
                                      cfg.psablock)[rows, 0]
        gu.compare_head(par, qh, kh, vh, keep[h], 1, cfg.scale, og, lse_orig, rows=rows, groups=groups)
    par.check("wan14b_3d:")
