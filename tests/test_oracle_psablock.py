"""Pins of the PSABlock oracle (oracle/psablock.py) against what the paper and the
mathematics fix: the PSABlock grids the paper prints for its models, hand-worked token groups,
maps and layouts, reductions to the one-dimensional reading and to token-level Algorithm 1,
and the equivalence of attention in the original order with attention in the padded
PSABlock-centric layout."""
import itertools

import numpy as np
import pytest

import oracle
from oracle import psablock as opsb
import golden_maps

INF = 2 ** 31 - 1


@pytest.mark.parametrize("grid,pb,coarse,padded", [
    # Appendix "Initialization of Mask Candidates": Wan 2.1 21x45x80 padded to 21x48x80 with
    # 3x8x16 PSABlocks (T_w < 7, S_w < 5); HunyuanVideo 720p 33x45x80 padded to 33x48x80 with
    # 3x8x16 (T_w < 11, S_w < 5); HunyuanVideo 768p 30x48x80 unpadded with 6x8x8 (T_w < 5,
    # S_w < 10).  The coarse extents are the bounds the paper gives for T_w and S_w.
    ((21, 45, 80), (3, 8, 16), (7, 6, 5), (21, 48, 80)),
    ((33, 45, 80), (3, 8, 16), (11, 6, 5), (33, 48, 80)),
    ((30, 48, 80), (6, 8, 8), (5, 6, 10), (30, 48, 80)),
])
def test_paper_psablock_grids(grid, pb, coarse, padded):
    assert oracle.psablock_grid(*grid, pb) == (coarse, padded)


def test_padding_ratio_of_the_paper():
    # Sec. 3.2: padding H from 45 to 48 at 720p; 48/45 - 1 = 6.7 % more tokens, of which the
    # paper charges 80 % of the steps: about 5 %.
    _, (t, h, w) = oracle.psablock_grid(21, 45, 80, (3, 8, 16))
    r = t * h * w / (21 * 45 * 80) - 1
    assert abs(r - 3 / 45) < 1e-12 and abs(0.8 * r - 0.0533) < 1e-3


def test_hand_worked_token_groups():
    g = oracle.token_groups(2, 3, 4, 0, (1, 2, 2)).reshape(2, 3, 4)
    frame0 = np.array([[0, 0, 1, 1], [0, 0, 1, 1], [2, 2, 3, 3]])
    assert (g[0] == frame0).all() and (g[1] == frame0 + 4).all()
    g = oracle.token_groups(3, 5, 5, 2, (2, 2, 2))
    # (t, h, w) -> t*25 + h*5 + w:  (2,4,4)=74 -> 9+6+2;  (0,0,4)=4 -> 2;  (1,3,1)=41 -> 3;
    # (2,0,0)=50 -> 9;  text tokens 75, 76 -> the global group 18.
    assert [g[74], g[4], g[41], g[50], g[75], g[76]] == [17, 2, 3, 9, 18, 18]


@pytest.mark.parametrize("case", golden_maps.load(golden_maps.PSABLOCK_PATH), ids=lambda c: c["name"])
def test_golden_psablock_maps(case):
    f, h, w, nt = case["grid"]
    bmap = oracle.psablock_map([case["m"]], f, h, w, nt, case["pb"])[0]
    assert int(bmap.sum()) == case["kept"]
    if case["map"] is not None:
        assert (bmap == case["map"]).all()
    if case["empty"] is not None:
        assert list(np.nonzero(bmap.sum(1) == 0)[0]) == case["empty"]


def _random_params(rng, n, tmax, smax):
    out = []
    for _ in range(n):
        out.append((int(rng.integers(1, tmax + 1)), int(rng.choice([0, 1, -1, 2, -2])),
                    int(rng.choice([1, 2, 3, INF])), int(rng.integers(1, smax + 1)),
                    int(rng.choice([0, 1, -1])), int(rng.choice([1, 3, 5, 6, INF]))))
    return out


@pytest.mark.parametrize("grid,b", [((4, 16, 16, 0), 16), ((3, 4, 12, 5), 4), ((2, 6, 8, 0), 8)])
def test_one_row_psablocks_are_the_one_dimensional_blocks(grid, b):
    """PSABlocks of 1 x 1 x B with B dividing W are runs of B consecutive tokens, and their
    coordinates are the first-token coordinates of the one-dimensional reading."""
    f, h, w, nt = grid
    params = _random_params(np.random.default_rng(b), 12, f, h * w // b)
    groups = oracle.token_groups(f, h, w, nt, (1, 1, b))
    n_video = f * h * w
    assert (groups[:n_video] == np.arange(n_video) // b).all()
    one_d = oracle.blockmap(params, f, h, w, 0, b)
    assert (oracle.psablock_map(params, f, h, w, 0, (1, 1, b)) == one_d).all()


def test_unit_psablocks_are_token_level_algorithm1():
    f, h, w = 3, 2, 3
    rng = np.random.default_rng(3)
    for m in _random_params(rng, 20, f, h * w):
        bmap = oracle.psablock_map([m], f, h, w, 0, (1, 1, 1))[0]
        for i, j in itertools.product(range(f * h * w), repeat=2):
            assert bool(bmap[i, j]) == bool(oracle.is_attending(i, j, m, h, w))


def test_brute_force_token_pairs_with_padding():
    """Every token pair of a padded grid, coordinates computed straight from (t, h, w)."""
    f, h, w, nt, pb = 3, 5, 7, 2, (2, 2, 3)
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    for m in _random_params(np.random.default_rng(5), 10, tp, hp * wp):
        bmap = oracle.psablock_map([m], f, h, w, nt, pb)[0]
        g = oracle.token_groups(f, h, w, nt, pb)
        n = f * h * w + nt
        for i in range(0, n, 3):
            for j in range(n):
                if i >= f * h * w or j >= f * h * w:
                    expect = True
                else:
                    ti, hi, wi = i // (h * w), (i // w) % h, i % w
                    tj, hj, wj = j // (h * w), (j // w) % h, j % w
                    dt = tj // pb[0] - ti // pb[0]
                    ds = (hj // pb[1] * wp + wj // pb[2]) - (hi // pb[1] * wp + wi // pb[2])
                    expect = (abs(dt - m[1]) % m[2] <= m[0] - 1) and (abs(ds - m[4]) % m[5] <= m[3] - 1)
                assert bool(bmap[g[i], g[j]]) == expect


def test_hand_worked_layout():
    # Grid 1x2x3 + 2 text tokens, PSABlock 1x2x2: padded to 1x2x4, W' = 2.  PSABlock 0 holds
    # (h, w) = (0,0) (0,1) (1,0) (1,1) = tokens 0 1 3 4; PSABlock 1 holds (0,2) (0,3) (1,2)
    # (1,3) = token 2, padding, token 5, padding; then the text tokens 6 7.
    x = (np.arange(8, dtype=np.float64) + 1)[:, None]
    xb = oracle.to_blocks(x, 1, 2, 3, 2, (1, 2, 2))
    assert xb[:, 0].tolist() == [1, 2, 4, 5, 3, 0, 6, 0, 7, 8]
    assert (oracle.from_blocks(xb, 1, 2, 3, 2, (1, 2, 2)) == x).all()


@pytest.mark.parametrize("grid,pb", [((3, 5, 7, 4), (2, 2, 3)), ((4, 6, 8, 0), (2, 3, 4)), ((5, 3, 9, 1), (3, 2, 2))])
def test_layout_round_trip_and_block_contiguity(grid, pb):
    f, h, w, nt = grid
    x = np.random.default_rng(1).standard_normal((f * h * w + nt, 3))
    xb = oracle.to_blocks(x, f, h, w, nt, pb)
    assert (oracle.from_blocks(xb, f, h, w, nt, pb) == x).all()
    # every PSABlock is contiguous: position p of the video part lies in PSABlock p div P
    groups = oracle.token_groups(f, h, w, nt, pb).astype(np.float64)[:, None] + 1
    gb = oracle.to_blocks(groups, f, h, w, nt, pb)[:, 0]
    p = pb[0] * pb[1] * pb[2]
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    n_blk = tp * hp * wp * p
    valid = gb[:n_blk] > 0
    assert (gb[:n_blk][valid] - 1 == (np.arange(n_blk) // p)[valid]).all()
    assert valid.sum() == f * h * w and (gb[n_blk:] == tp * hp * wp + 1).all()


def test_attention_in_the_padded_layout_equals_the_original_order():
    """Attention over the PSABlock-centric layout, with padded keys excluded and PSABlocks as
    runs of P consecutive tokens, returns the original-order result after from_blocks."""
    f, h, w, nt, pb = 3, 5, 5, 3, (2, 2, 2)
    n = f * h * w + nt
    rng = np.random.default_rng(7)
    q, k, v = (rng.standard_normal((n, 8)) for _ in range(3))
    params = [(1, 0, INF, 2, 1, 3)]
    keep = oracle.psablock_map(params, f, h, w, nt, pb)[0]
    o, lse = oracle.masked_attention(q, k, v, keep, 1, 0.3, groups=oracle.token_groups(f, h, w, nt, pb))
    (tp, hp, wp), _ = oracle.psablock_grid(f, h, w, pb)
    n_p, p = tp * hp * wp, 8
    qb, kb, vb = (oracle.to_blocks(x, f, h, w, nt, pb) for x in (q, k, v))
    valid = oracle.to_blocks(np.ones((n, 1)), f, h, w, nt, pb)[:, 0] > 0
    gb = np.concatenate([np.arange(n_p * p) // p, np.full(nt, n_p)])
    gb = np.where(valid, gb, n_p + 1)                       # padding: a group nobody keeps
    keep_b = np.zeros((n_p + 2, n_p + 2), dtype=np.uint8)
    keep_b[:n_p + 1, :n_p + 1] = keep
    ob, lb = oracle.masked_attention(qb, kb, vb, keep_b, 1, 0.3, groups=gb)
    assert np.allclose(oracle.from_blocks(ob, f, h, w, nt, pb), o, atol=1e-12)
    assert np.allclose(oracle.from_blocks(lb[:, None], f, h, w, nt, pb)[:, 0], lse, atol=1e-12)


def test_grouped_attention_with_runs_is_the_block_form():
    rng = np.random.default_rng(2)
    q, k, v = (rng.standard_normal((50, 4)) for _ in range(3))
    keep = rng.integers(0, 2, (7, 7)).astype(np.uint8)
    a = oracle.masked_attention(q, k, v, keep, 8, 0.5)
    b = oracle.masked_attention(q, k, v, keep, 999, 0.5, groups=np.arange(50) // 8)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# Plant plausible slips in the oracle: each must fail a pin above.
def _mutant_plane_transposed(frames, height, width, n_text, pb):
    t, s, glob = _orig_coords(frames, height, width, n_text, pb)
    (tp, hp, wp), _ = oracle.psablock_grid(frames, height, width, pb)
    s2 = np.where(glob, s, (s % wp) * hp + s // wp)        # w' H' + h' instead of h' W' + w'
    return t, s2, glob


def _mutant_floor_grid(frames, height, width, pb):
    (tp, hp, wp), padded = _orig_grid(frames, height, width, pb)
    return (frames // pb[0] or 1, height // pb[1] or 1, width // pb[2] or 1), padded


def _orig_coords(*a):
    return opsb.__dict__["_saved_coords"](*a)


def _orig_grid(*a):
    return opsb.__dict__["_saved_grid"](*a)


def _pins_pass():
    try:
        for case in golden_maps.load(golden_maps.PSABLOCK_PATH):
            test_golden_psablock_maps(case)
        test_hand_worked_token_groups()
        test_paper_psablock_grids((21, 45, 80), (3, 8, 16), (7, 6, 5), (21, 48, 80))
        test_brute_force_token_pairs_with_padding()
    except (AssertionError, IndexError, ValueError):
        return False
    return True


def test_mutant_transposed_plane_is_caught(monkeypatch):
    monkeypatch.setitem(opsb.__dict__, "_saved_coords", opsb.group_coordinates)
    monkeypatch.setattr(opsb, "group_coordinates", _mutant_plane_transposed)
    assert not _pins_pass()


def test_mutant_floor_grid_is_caught(monkeypatch):
    monkeypatch.setitem(opsb.__dict__, "_saved_grid", opsb.psablock_grid)
    monkeypatch.setattr(opsb, "psablock_grid", _mutant_floor_grid)
    monkeypatch.setattr(oracle, "psablock_grid", _mutant_floor_grid)
    assert not _pins_pass()


def test_mutant_query_minus_key_is_caught(monkeypatch):
    real = opsb.psablock_map

    def flipped(params, *a):
        return np.transpose(real(params, *a), (0, 2, 1))
    monkeypatch.setattr(oracle, "psablock_map", flipped)
    assert not _pins_pass()
