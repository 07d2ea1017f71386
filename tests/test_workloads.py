"""Seeded workloads: stored stripe parameters, densities and input synthesis."""
import numpy as np
import pytest

import oracle
from workloads import CONFIGS, get_config, make_head_qkv, make_qkv, stripe_params
from workloads import make_stripe_params as msp
from workloads.inputs import bf16_bits, bf16_round, bits_to_float, rope_tables
from workloads.params import STRIDE_INF, coarse_extent, load_json


@pytest.mark.parametrize("name", ["wan1_3b", "wan14b", "hunyuan"])
def test_stored_densities_match_oracle_blockmap(name):
    cfg = get_config(name)
    params = stripe_params(name)
    assert len(params) == cfg.heads
    bm = oracle.blockmap(params, cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)
    dens = oracle.kept_per_head(bm) / float(cfg.n_blocks ** 2)
    np.testing.assert_allclose(dens, load_json()[name]["density"], rtol=0, atol=1e-12)
    lo, hi = cfg.density_band
    assert dens.min() >= lo - 0.01 and dens.max() <= hi + 0.01


def test_psablock_workload_densities_match_oracle_map():
    cfg = get_config("wan14b_3d")
    params = stripe_params("wan14b_3d")
    assert len(params) == cfg.heads and cfg.coarse_grid == (7, 6, 5)
    bm = oracle.psablock_map(params, cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.psablock)
    dens = bm.reshape(cfg.heads, -1).sum(1) / float(bm.shape[1] ** 2)
    np.testing.assert_allclose(dens, load_json()["wan14b_3d"]["density"], rtol=0, atol=1e-12)
    tp, sp = coarse_extent(cfg)
    assert (tp, sp) == (7, 30)
    for m in params:
        assert 1 <= m[0] <= tp and 1 <= m[3] <= sp


def test_headline_mean_density_near_quarter():
    assert abs(np.mean(load_json()["wan14b"]["density"]) - 0.25) < 0.03


def test_sweep_runs():
    cfg = get_config("sweep")
    data = load_json()["sweep"]
    tp, sp = coarse_extent(cfg)
    for key, run in data.items():
        target = float(key)
        assert abs(np.mean(run["density"]) - target) < 0.02, key
        for h, m in enumerate(run["params"]):
            assert m[2] == 1 + (h % tp) and m[5] == sp - (h % sp)
    full = stripe_params("sweep", 1.0)
    bm = oracle.blockmap(full, cfg.frames, cfg.height, cfg.width, 0, cfg.block)
    assert bm.all()


def test_stored_params_regenerate():
    data = msp.build()
    stored = load_json()
    for name in ("wan1_3b", "wan14b", "hunyuan", "wan14b_3d"):
        assert data[name]["params"] == stored[name]["params"]
    assert data["sweep"]["0.30"]["params"] == stored["sweep"]["0.30"]["params"]


def test_tiny_params_in_paper_ranges():
    ps = stripe_params("tiny")
    assert len(ps) == 2 and ps == stripe_params("tiny")
    for m in ps:
        assert 1 <= m[0] <= 4 and m[1] in (0, 1, -1, 2, -2) and m[2] in (1, 2, 3, STRIDE_INF)
        assert 1 <= m[3] <= 4 and m[4] in (0, 1, -1) and m[5] in (1, 3, 5, 6, STRIDE_INF)


def test_bf16_round_matches_torch():
    import torch
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 7
    assert (bf16_round(x) == torch.from_numpy(x).bfloat16().float().numpy()).all()
    assert (bits_to_float(bf16_bits(bf16_round(x))) == bf16_round(x)).all()


def test_inputs_are_bf16_and_seeded():
    cfg = get_config("tiny")
    q, k, v = make_head_qkv(cfg, 0, 1)
    for x in (q, k, v):
        assert x.shape == (1024, 64) and (bf16_round(x) == x).all()
    q2, _, _ = make_head_qkv(cfg, 0, 1)
    assert (q == q2).all()
    Q, K, V = make_qkv(cfg, bits=False)
    assert (Q[0, 1] == q).all() and (V[0, 1] == v).all()
    assert not (Q[0, 0] == Q[0, 1]).all()


def test_rope_rotates_pairs():
    """Rotation keeps each channel pair's norm; text tokens are untouched."""
    cfg = CONFIGS["hunyuan"]
    small = type(cfg)("t", 1, 1, 128, 2, 3, 4, 5, 8, (44, 42, 42), None)
    cos, sin = rope_tables(small)
    assert cos.shape == (24, 64)
    np.testing.assert_allclose(cos ** 2 + sin ** 2, 1.0, atol=1e-6)
    q, _, v = make_head_qkv(small, 0, 0)
    rng = np.random.default_rng([small.seed, 0, 0, 0])
    raw = bf16_round(rng.standard_normal((29, 128), dtype=np.float32))
    assert (q[24:] == raw[24:]).all()                     # text tokens not rotated
    n_rot = np.hypot(q[:24, 0::2], q[:24, 1::2])
    n_raw = np.hypot(raw[:24, 0::2], raw[:24, 1::2])
    np.testing.assert_allclose(n_rot, n_raw, rtol=2e-2, atol=1e-2)
    assert (q[0] == raw[0]).all()                         # position (0,0,0): angle 0


def test_search_candidates_in_paper_space():
    from workloads.candidates import candidates
    cfg = get_config("wan14b")
    tp, sp = coarse_extent(cfg)
    cands = candidates("wan14b", 100)
    assert len(cands) == cfg.heads and all(len(c) == 100 and len(set(c)) == 100 for c in cands)
    for head in cands:
        for m in head:
            assert 1 <= m[0] <= tp and m[1] in (0, 1, -1, 2, -2) and m[2] in (1, 2, 3, STRIDE_INF)
            assert 1 <= m[3] <= sp and m[4] in (0, 1, -1) and m[5] in (1, 3, 5, 6, STRIDE_INF)
    assert cands[0] != cands[1] and candidates("wan14b", 100) == cands
