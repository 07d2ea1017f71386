"""Property tests of the oracle on random small grids and random stripe parameters (hypothesis):
token-level Algorithm 1 at block size 1, transpose symmetry for zero offsets, periodicity and
evenness of the axis test, monotonicity in the widths, 1 x 1 x B PSABlocks equal to
one-dimensional blocks, the Kronecker count on aligned grids, and attention invariants."""
import itertools

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle

INF = 2 ** 31 - 1
SETTINGS = settings(max_examples=40, deadline=None, derandomize=True)

strides = st.sampled_from([1, 2, 3, 5, 6, INF])
offsets = st.integers(-3, 3)
widths = st.integers(1, 4)
stripe = st.tuples(widths, offsets, strides, widths, offsets, strides)


@SETTINGS
@given(f=st.integers(1, 3), h=st.integers(1, 3), w=st.integers(1, 4), m=stripe)
def test_block_size_one_is_token_level_algorithm1(f, h, w, m):
    bmap = oracle.blockmap([m], f, h, w, 0, 1)[0]
    n = f * h * w
    for i, j in itertools.product(range(n), repeat=2):
        assert bool(bmap[i, j]) == bool(oracle.is_attending(i, j, m, h, w))


@SETTINGS
@given(f=st.integers(1, 4), h=st.integers(1, 6), w=st.integers(1, 6), nt=st.integers(0, 5),
       block=st.integers(1, 9), tw=widths, ts=strides, sw=widths, ss=strides)
def test_zero_offsets_give_a_symmetric_map(f, h, w, nt, block, tw, ts, sw, ss):
    bmap = oracle.blockmap([(tw, 0, ts, sw, 0, ss)], f, h, w, nt, block)[0]
    assert (bmap == bmap.T).all()


@SETTINGS
@given(delta=st.integers(-50, 50), w=widths, o=offsets, s=st.sampled_from([1, 2, 3, 5, 6]))
def test_axis_condition_is_even_about_the_offset_and_periodic(delta, w, o, s):
    x = abs(delta)
    assert oracle.axis_condition(o + x, w, o, s) == oracle.axis_condition(o - x, w, o, s)
    assert oracle.axis_condition(o + x + s, w, o, s) == oracle.axis_condition(o + x, w, o, s)


@SETTINGS
@given(f=st.integers(1, 4), h=st.integers(1, 6), w=st.integers(1, 6), nt=st.integers(0, 4),
       block=st.integers(1, 8), m=stripe)
def test_kept_set_grows_with_the_widths(f, h, w, nt, block, m):
    tw, to, ts, sw, so, ss = m
    small = oracle.blockmap([m], f, h, w, nt, block)[0]
    wider = oracle.blockmap([(tw + 1, to, ts, sw + 1, so, ss)], f, h, w, nt, block)[0]
    assert (wider >= small).all()


@SETTINGS
@given(f=st.integers(1, 3), hq=st.integers(1, 3), wq=st.integers(1, 3), b=st.sampled_from([1, 2, 4]),
       nt=st.integers(0, 3), m=stripe)
def test_one_row_psablocks_equal_one_dimensional_blocks(f, hq, wq, b, nt, m):
    h, w = hq, wq * b                       # b divides W, so 1 x 1 x b PSABlocks are runs of b tokens
    one_d = oracle.blockmap([m], f, h, w, 0, b)[0]
    assert (oracle.psablock_map([m], f, h, w, 0, (1, 1, b))[0] == one_d).all()


@SETTINGS
@given(f=st.integers(1, 4), s_slots=st.integers(1, 4), b=st.sampled_from([1, 2, 4]), m=stripe)
def test_aligned_grids_factor_into_axes(f, s_slots, b, m):
    """When blocks tile frames (B | HW), kept = K_t * K_s with K_x = sum over axis pairs."""
    h, w = 1, s_slots * b
    tw, to, ts, sw, so, ss = m
    bmap = oracle.blockmap([m], f, h, w, 0, b)[0]
    kt = sum(oracle.axis_condition(t2 - t1, tw, to, ts) for t1 in range(f) for t2 in range(f))
    ks = sum(oracle.axis_condition(s2 - s1, sw, so, ss) for s1 in range(s_slots) for s2 in range(s_slots))
    assert int(bmap.sum()) == int(kt) * int(ks)


@SETTINGS
@given(seed=st.integers(0, 10 ** 6), nb=st.integers(1, 5), block=st.integers(1, 6))
def test_attention_invariants(seed, nb, block):
    rng = np.random.default_rng(seed)
    n = nb * block - int(rng.integers(0, block))
    q, k = rng.standard_normal((n, 4)), rng.standard_normal((n, 4))
    keep = rng.integers(0, 2, (nb, nb)).astype(np.uint8)
    o, lse = oracle.masked_attention(q, k, np.ones((n, 3)), keep, block, 0.7)
    live = np.isfinite(lse)
    assert np.allclose(o[live], 1.0) and (o[~live] == 0).all()
    # permuting keys (with their values) inside one block changes nothing
    v = rng.standard_normal((n, 3))
    perm = np.arange(n)
    b0 = int(rng.integers(0, nb))
    lo, hi = b0 * block, min(n, (b0 + 1) * block)
    perm[lo:hi] = rng.permutation(np.arange(lo, hi))
    a = oracle.masked_attention(q, k, v, keep, block, 0.7)
    b_ = oracle.masked_attention(q, k[perm], v[perm], keep, block, 0.7)
    assert np.allclose(a[0], b_[0], atol=1e-12) and np.allclose(a[1], b_[1], atol=1e-12, equal_nan=True)
