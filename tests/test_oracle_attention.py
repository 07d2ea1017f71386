"""Pins for the oracle's masked softmax attention.

References that are independent of the oracle: torch's CPU scaled_dot_product_attention
(float64, explicit boolean mask), closed forms (V == 1, Q == 0, per-frame attention),
invariance under permuting keys inside one key block, and a pure-Python brute force.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.attention import masked_attention

INF = oracle.STRIDE_INF


def rand_qkv(rng, n, d):
    return (rng.standard_normal((n, d)), rng.standard_normal((n, d)), rng.standard_normal((n, d)))


def sdpa(q, k, v, tokmask, scale):
    t = lambda x: torch.from_numpy(np.asarray(x, np.float64))[None, None]
    out = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), attn_mask=torch.from_numpy(tokmask)[None, None], scale=scale)
    return out[0, 0].numpy()


def token_mask(keep, block, n):
    kb = np.arange(n) // block
    return np.asarray(keep, bool)[kb][:, kb]


def test_full_map_is_dense_attention():
    rng = np.random.default_rng(0)
    n, d, b = 200, 32, 16
    q, k, v = rand_qkv(rng, n, d)
    nb = -(-n // b)
    o, lse = masked_attention(q, k, v, np.ones((nb, nb), bool), b, 0.2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        *(torch.from_numpy(x)[None, None] for x in (q, k, v)), scale=0.2)[0, 0].numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    ref_lse = torch.logsumexp(0.2 * torch.from_numpy(q) @ torch.from_numpy(k).T, dim=1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_stripe_mask_matches_library_masked_attention(seed):
    rng = np.random.default_rng(10 + seed)
    f, h, w, nt, b = 3, 4, 5, 7, 6           # N = 67, 12 blocks, ragged tail, text blocks
    n = f * h * w + nt
    d = 16
    q, k, v = rand_qkv(rng, n, d)
    m = (int(rng.integers(1, 3)), int(rng.integers(-1, 2)), int(rng.choice([1, 2, INF])),
         int(rng.integers(1, 3)), int(rng.integers(-1, 2)), int(rng.choice([1, 3, INF])))
    keep = oracle.blockmap([m], f, h, w, nt, b)[0]
    o, lse = masked_attention(q, k, v, keep, b, 0.25)
    tm = token_mask(keep, b, n)
    live = tm.any(1)
    ref = sdpa(q, k, v, tm, 0.25)
    np.testing.assert_allclose(o[live], ref[live], rtol=1e-11, atol=1e-12)
    s = 0.25 * (q @ k.T)
    s[~tm] = -np.inf
    ref_lse = torch.logsumexp(torch.from_numpy(s), dim=1).numpy()
    np.testing.assert_allclose(lse[live], ref_lse[live], rtol=1e-12)
    assert (o[~live] == 0).all() and np.isneginf(lse[~live]).all()


def test_asymmetric_mask_transpose_would_fail():
    """A transposed mask (query/key swapped) is detected by the library reference."""
    rng = np.random.default_rng(3)
    n, d, b = 64, 8, 8
    q, k, v = rand_qkv(rng, n, d)
    keep = oracle.blockmap([(1, 1, INF, 1, 0, INF)], 8, 8, 1, 0, 8)[0]   # dt = 1 only
    assert not (keep == keep.T).all()
    o, _ = masked_attention(q, k, v, keep, b, 0.3)
    o_t, _ = masked_attention(q, k, v, keep.T, b, 0.3)
    tm = token_mask(keep, b, n)
    live = tm.any(1)
    ref = sdpa(q, k, v, tm, 0.3)
    assert np.allclose(o[live], ref[live])
    assert not np.allclose(o_t[live], ref[live])


def test_wrong_scale_would_fail():
    rng = np.random.default_rng(4)
    q, k, v = rand_qkv(rng, 48, 8)
    keep = np.ones((6, 6), bool)
    ref = sdpa(q, k, v, np.ones((48, 48), bool), 0.35)
    assert np.allclose(masked_attention(q, k, v, keep, 8, 0.35)[0], ref)
    assert not np.allclose(masked_attention(q, k, v, keep, 8, 1.0)[0], ref)


def test_constant_values_give_one():
    rng = np.random.default_rng(5)
    n, d, b = 96, 8, 8
    q, k, _ = rand_qkv(rng, n, d)
    keep = oracle.blockmap([(1, 1, INF, 2, 0, INF)], 4, 6, 4, 0, b)[0]   # rows of the last frame are empty
    o, lse = masked_attention(q, k, np.ones((n, d)), keep, b, 0.5)
    live = keep.any(1)[np.arange(n) // b]
    assert not live.all() and live.any()
    np.testing.assert_allclose(o[live], 1.0, rtol=0, atol=1e-13)
    assert (o[~live] == 0).all() and np.isneginf(lse[~live]).all()


def test_zero_queries_give_mean_of_kept_values():
    rng = np.random.default_rng(6)
    n, d, b = 80, 8, 10
    _, k, v = rand_qkv(rng, n, d)
    keep = oracle.blockmap([(2, 0, 3, 1, 1, INF)], 4, 4, 5, 0, b)[0]
    o, lse = masked_attention(np.zeros((n, d)), k, v, keep, b, 0.5)
    for i in range(n):
        kept = keep[i // b][np.arange(n) // b].astype(bool)
        if kept.any():
            np.testing.assert_allclose(o[i], v[kept].mean(0), rtol=1e-12, atol=1e-14)
            assert math.isclose(lse[i], math.log(kept.sum()), rel_tol=1e-12)


def test_per_frame_map_is_per_frame_attention():
    """(T_w=1,T_o=0,T_s=inf | S_w=S',S_o=0,S_s=inf) on an aligned grid: attention within a frame."""
    rng = np.random.default_rng(7)
    f, h, w, b = 3, 4, 8, 8                # HW = 32, S' = 4
    n = f * h * w
    q, k, v = rand_qkv(rng, n, 16)
    keep = oracle.blockmap([(1, 0, INF, 4, 0, INF)], f, h, w, 0, b)[0]
    o, _ = masked_attention(q, k, v, keep, b, 0.25)
    for t in range(f):
        sl = slice(t * 32, (t + 1) * 32)
        ref = torch.nn.functional.scaled_dot_product_attention(
            *(torch.from_numpy(x[sl])[None, None] for x in (q, k, v)), scale=0.25)[0, 0].numpy()
        np.testing.assert_allclose(o[sl], ref, rtol=1e-12, atol=1e-13)


def test_permuting_keys_inside_a_block_is_invariant():
    rng = np.random.default_rng(8)
    n, d, b = 64, 8, 16
    q, k, v = rand_qkv(rng, n, d)
    keep = oracle.blockmap([(1, 0, 2, 2, 1, 3)], 4, 4, 4, 0, b)[0]
    perm = np.arange(n)
    perm[16:32] = rng.permutation(np.arange(16, 32))
    o1, l1 = masked_attention(q, k, v, keep, b, 0.4)
    o2, l2 = masked_attention(q, k[perm], v[perm], keep, b, 0.4)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-12)


def test_brute_force_python():
    rng = np.random.default_rng(9)
    n, d, b = 20, 4, 3
    q, k, v = rand_qkv(rng, n, d)
    keep = rng.random((7, 7)) < 0.5
    keep[2] = False
    o, lse = masked_attention(q, k, v, keep, b, 0.7, rows=[0, 5, 6, 7, 19])
    for r, i in enumerate([0, 5, 6, 7, 19]):
        js = [j for j in range(n) if keep[i // b][j // b]]
        if not js:
            assert (o[r] == 0).all() and lse[r] == -math.inf
            continue
        s = [0.7 * sum(q[i][c] * k[j][c] for c in range(d)) for j in js]
        mx = max(s)
        p = [math.exp(x - mx) for x in s]
        l = math.fsum(p)
        for c in range(d):
            assert math.isclose(o[r][c], math.fsum(pj * v[j][c] for pj, j in zip(p, js)) / l,
                                rel_tol=1e-11, abs_tol=1e-13)
        assert math.isclose(lse[r], mx + math.log(l), rel_tol=1e-12)
