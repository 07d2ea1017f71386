"""Pins for the oracle's stripe-to-mask definition (Algorithm 1 on block coordinates).

Nothing here re-types the oracle's formula: each check compares it with something fixed
independently -- maps worked by hand, closed-form counts, invariants of the formula, the
paper's own special cases (SVG / STA tuples, "infinite stride = one diagonal") and the literal
token-level Algorithm 1 -- and the mutation tests show that plausible slips fail these pins.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import stripe as ostripe
from golden_maps import load as load_golden

INF = oracle.STRIDE_INF
T_STRIDES = (1, 2, 3, INF)
S_STRIDES = (1, 3, 5, 6, INF)


def golden_failures():
    """Names of golden cases the current oracle gets wrong."""
    bad = []
    for c in load_golden():
        f, h, w, nt, b = c["grid"]
        bm = oracle.blockmap([c["m"]], f, h, w, nt, b)[0]
        ok = int(bm.sum()) == c["kept"]
        if c["map"] is not None:
            ok &= bm.shape == c["map"].shape and bool((bm == c["map"]).all())
        if c["empty"] is not None:
            ok &= sorted(np.nonzero(bm.sum(1) == 0)[0].tolist()) == c["empty"]
        if not ok:
            bad.append(c["name"])
    return bad


def test_golden_maps():
    assert golden_failures() == []


def test_golden_counts_consistent():
    rows = oracle.kept_per_row(oracle.blockmap([(2, -1, 3, 3, 1, 5)], 4, 16, 16, 0, 64))
    assert rows.shape == (1, 16) and rows.sum() == 156
    assert oracle.kept_per_head(oracle.blockmap([(1, 0, INF, 1, 0, INF), (4, 0, INF, 4, 0, INF)],
                                                4, 16, 16, 0, 64)).tolist() == [16, 256]


def random_m(rng, tp, sp, strides_t=T_STRIDES, strides_s=S_STRIDES):
    return (int(rng.integers(1, tp + 1)), int(rng.integers(-2, 3)), int(rng.choice(strides_t)),
            int(rng.integers(1, sp + 1)), int(rng.integers(-1, 2)), int(rng.choice(strides_s)))


@pytest.mark.parametrize("grid", [(3, 2, 3), (2, 3, 4), (4, 2, 2)])
def test_block1_is_token_level_algorithm1(grid):
    """At block size 1 the block map is Algorithm 1 applied to every token pair."""
    f, h, w = grid
    rng = np.random.default_rng(7)
    n = f * h * w
    for _ in range(25):
        m = random_m(rng, f, h * w, strides_t=(1, 2, 3, INF), strides_s=(1, 2, 3, 5, INF))
        bm = oracle.blockmap([m], f, h, w, 0, 1)[0]
        ref = np.array([[oracle.is_attending(i, j, m, h, w) for j in range(n)] for i in range(n)])
        assert (bm.astype(bool) == ref).all(), m


def test_token_level_examples():
    # 2 frames of 2x2 tokens; M = (1,1,inf | 1,0,inf): only dt = 1 and ds = 0.
    m = (1, 1, INF, 1, 0, INF)
    assert oracle.is_attending(0, 4, m, 2, 2) and oracle.is_attending(3, 7, m, 2, 2)
    assert not oracle.is_attending(4, 0, m, 2, 2)          # dt = -1: offset has a direction
    assert not oracle.is_attending(0, 5, m, 2, 2)          # ds = 1
    assert not oracle.is_attending(0, 0, m, 2, 2)          # dt = 0


@pytest.mark.parametrize("grid", [(4, 16, 16, 0, 64), (2, 3, 4, 0, 5), (5, 6, 7, 0, 8), (3, 5, 5, 4, 6)])
def test_zero_offsets_give_symmetric_map(grid):
    rng = np.random.default_rng(1)
    f, h, w, nt, b = grid
    sp = -(-(h * w) // b)
    for _ in range(40):
        m = list(random_m(rng, f, sp))
        m[1] = m[4] = 0
        bm = oracle.blockmap([tuple(m)], *grid)[0]
        assert (bm == bm.T).all(), m


def test_axis_condition_even_about_offset_and_periodic():
    rng = np.random.default_rng(2)
    for _ in range(300):
        w, o, s = int(rng.integers(1, 8)), int(rng.integers(-3, 4)), int(rng.choice([1, 2, 3, 5, 6, 7]))
        x = np.arange(0, 40)
        a = ostripe.axis_condition(o + x, w, o, s)
        assert (a == ostripe.axis_condition(o - x, w, o, s)).all()            # evenness
        assert (ostripe.axis_condition(o + x + s, w, o, s) == a).all()        # period s for x >= 0
        # within one period the kept distances from the offset are exactly 0..w-1
        assert a[:s].tolist() == [i <= w - 1 for i in range(s)]


def test_full_axis_when_width_reaches_stride():
    for w, s in [(1, 1), (3, 1), (3, 3), (5, 3), (6, 6)]:
        d = np.arange(-50, 51)
        assert ostripe.axis_condition(d, w, 0, s).all()
        assert ostripe.axis_condition(d, w, 2, s).all()


def test_large_stride_equals_infinite_stride():
    """A stride no smaller than the extent plus |offset| acts as one diagonal (appendix)."""
    rng = np.random.default_rng(3)
    f, h, w, b = 5, 8, 8, 16
    tp, sp = f, 4
    for _ in range(60):
        m = random_m(rng, tp, sp)
        mi = (m[0], m[1], INF, m[3], m[4], INF)
        big = (m[0], m[1], tp + abs(m[1]) + int(rng.integers(0, 5)), m[3], m[4], sp + abs(m[4]) + int(rng.integers(0, 5)))
        assert (oracle.blockmap([mi], f, h, w, 0, b) == oracle.blockmap([big], f, h, w, 0, b)).all()


def pair_count(n, w, o, s):
    """Closed form: number of ordered pairs (a, b) in [0, n) with the axis condition on b - a."""
    return sum((n - abs(d)) for d in range(-(n - 1), n) if (abs(d - o) % s) <= w - 1)


@pytest.mark.parametrize("grid", [(4, 16, 16, 64), (6, 8, 8, 16), (3, 4, 6, 8), (7, 3, 10, 5)])
def test_separable_kronecker_on_aligned_grids(grid):
    """When blocks tile frames exactly the map is T (x) S and the count is K_t * K_s."""
    f, h, w, b = grid
    hw = h * w
    assert hw % b == 0
    sp = hw // b
    rng = np.random.default_rng(4)
    for _ in range(40):
        m = random_m(rng, f, sp)
        bm = oracle.blockmap([m], f, h, w, 0, b)[0]
        tt = np.array([[ostripe.axis_condition(tk - tq, *m[:3]) for tk in range(f)] for tq in range(f)])
        ss = np.array([[ostripe.axis_condition(sk - sq, *m[3:]) for sk in range(sp)] for sq in range(sp)])
        assert (bm == np.kron(tt, ss).astype(np.uint8)).all()
        assert bm.sum() == pair_count(f, *m[:3]) * pair_count(sp, *m[3:])


def test_band_closed_form():
    """SVG-style band (stride inf, offset 0): n(2w-1) - w(w-1) pairs for w <= n."""
    for n in range(1, 12):
        for w in range(1, n + 1):
            assert pair_count(n, w, 0, INF) == n * (2 * w - 1) - w * (w - 1)
    bm = oracle.blockmap([(2, 0, INF, 3, 0, INF)], 4, 16, 16, 0, 64)[0]
    assert bm.sum() == (4 * 3 - 2) * (4 * 5 - 6)


def test_svg_and_sta_special_cases():
    """SVG = M(T_w,0,inf,S_w,0,inf), STA = M(T_w,0,inf,S_w,0,S_s) (Sec. 3.2): banded maps."""
    f, h, w, b = 6, 8, 8, 16   # T' = 6, S' = 4
    for tw, sw in [(1, 1), (2, 2), (3, 1)]:
        bm = oracle.blockmap([(tw, 0, INF, sw, 0, INF)], f, h, w, 0, b)[0]
        for qb, kb in itertools.product(range(24), repeat=2):
            band = abs(kb // 4 - qb // 4) < tw and abs(kb % 4 - qb % 4) < sw
            assert bm[qb, kb] == band
    bm = oracle.blockmap([(2, 0, INF, 1, 0, 2)], f, h, w, 0, b)[0]
    for qb, kb in itertools.product(range(24), repeat=2):
        assert bm[qb, kb] == (abs(kb // 4 - qb // 4) < 2 and (kb % 4 - qb % 4) % 2 == 0)


def test_coarsening_invariance():
    """If block | HW, the map equals block size 1 on the coarse (F, HW/B, 1) grid."""
    rng = np.random.default_rng(5)
    for (f, h, w, b) in [(4, 16, 16, 64), (3, 6, 8, 12), (5, 4, 4, 8)]:
        sp = h * w // b
        for _ in range(30):
            m = random_m(rng, f, sp)
            assert (oracle.blockmap([m], f, h, w, 0, b) == oracle.blockmap([m], f, sp, 1, 0, 1)).all()


def test_monotone_in_width():
    rng = np.random.default_rng(6)
    for _ in range(50):
        m = list(random_m(rng, 5, 6))
        a = oracle.blockmap([tuple(m)], 5, 6, 8, 0, 8)[0]
        m2 = list(m)
        m2[0] += 1
        m2[3] += 1
        b = oracle.blockmap([tuple(m2)], 5, 6, 8, 0, 8)[0]
        assert (b >= a).all()


def test_text_blocks_are_global():
    f, h, w, nt, b = 3, 5, 6, 40, 16     # N_video = 90, N = 130, 9 blocks; blocks 5.. hold text
    t, s, ln, g = oracle.block_coordinates(f, h, w, nt, b)
    assert g.tolist() == [False] * 5 + [True] * 4 and ln[-1] == 2
    bm = oracle.blockmap([(1, 0, INF, 1, 0, INF)], f, h, w, nt, b)[0]
    assert bm[5:].all() and bm[:, 5:].all()
    # the video-only part is the text-free map of the same blocks
    bm0 = oracle.blockmap([(1, 0, INF, 1, 0, INF)], f, h, w, 0, b)[0]
    assert (bm[:5, :5] == bm0[:5, :5]).all()


@pytest.mark.parametrize("grid,spots", [
    ((21, 30, 52, 0, 128), {12: (0, 12, 128), 13: (1, 0, 128), 24: (1, 11, 128), 25: (2, 0, 128),
                            255: (20, 11, 120)}),
    ((21, 45, 80, 0, 128), {28: (0, 28, 128), 29: (1, 0, 128), 590: (20, 27, 80)}),
    ((33, 45, 80, 256, 128), {927: (32, 27, 128)}),
])
def test_large_grid_coordinates(grid, spots):
    t, s, ln, g = oracle.block_coordinates(*grid)
    for b, (tb, sb, lb) in spots.items():
        assert (t[b], s[b], ln[b], g[b]) == (tb, sb, lb, False)
    if grid[3]:
        assert g[928:].all() and not g[:928].any() and ln[930] == 16 and len(g) == 931


def test_invalid_parameters_rejected():
    with pytest.raises(ValueError):
        oracle.blockmap([(0, 0, 1, 1, 0, 1)], 2, 2, 2, 0, 1)
    with pytest.raises(ValueError):
        oracle.blockmap([(1, 0, 0, 1, 0, 1)], 2, 2, 2, 0, 1)


# --- mutation tests: plausible slips planted in the oracle (on the CPU) must fail the pins ---

def _mutant_no_abs(delta, width, offset, stride):
    d = np.asarray(delta, dtype=np.int64) - offset
    return (d % stride) <= width - 1


def _mutant_sign(delta, width, offset, stride):
    d = np.abs(-np.asarray(delta, dtype=np.int64) - offset)
    return (d % stride) <= width - 1


def _mutant_strict_width(delta, width, offset, stride):
    d = np.abs(np.asarray(delta, dtype=np.int64) - offset)
    return (d % stride) < width - 1


def _mutant_offset_sign(delta, width, offset, stride):
    d = np.abs(np.asarray(delta, dtype=np.int64) + offset)
    return (d % stride) <= width - 1


def _mutant_last_token_coords(frames, height, width, n_text, block):
    t, s, length, g = ostripe.__dict__["_orig_coords"](frames, height, width, n_text, block)
    hw = height * width
    last = np.arange(len(t)) * block + length - 1
    return last // hw, (last % hw) // block, length, g


@pytest.mark.parametrize("mutant", [_mutant_no_abs, _mutant_sign, _mutant_strict_width, _mutant_offset_sign])
def test_mutants_of_axis_condition_are_caught(monkeypatch, mutant):
    monkeypatch.setattr(ostripe, "axis_condition", mutant)
    assert golden_failures() != []


def test_mutant_coordinates_are_caught(monkeypatch):
    monkeypatch.setitem(ostripe.__dict__, "_orig_coords", ostripe.block_coordinates)
    monkeypatch.setattr(ostripe, "block_coordinates", _mutant_last_token_coords)
    assert golden_failures() != []


def test_mutant_transposed_map_is_caught(monkeypatch):
    orig = ostripe.blockmap

    def transposed(*a, **k):
        return np.ascontiguousarray(orig(*a, **k).transpose(0, 2, 1))
    monkeypatch.setattr(oracle, "blockmap", transposed)
    assert golden_failures() != []
