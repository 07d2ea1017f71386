"""GPU parity of PSA-Search scoring: the L2 distance kernel against its plain definition, and
per-head candidate losses against the oracle's (Algorithm 3's L2 loss on the same inputs)."""
import numpy as np
import pytest

import oracle
from oracle import search as osearch
import paper_2609_37001_amd as psa
from paper_2609_37001_amd import search
from workloads import get_config
from workloads.candidates import candidates
from workloads.inputs import bf16_round

import gpu_util as gu

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def dev(x):
    t = gu.torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").bfloat16()


@pytest.mark.parametrize("shape", [(1, 3, 1000, 128), (2, 5, 4097, 64), (1, 1, 1, 8)])
def test_l2_distance_against_definition(shape):
    rng = np.random.default_rng(sum(shape))
    a = bf16_round(rng.standard_normal(shape).astype(np.float32))
    b = bf16_round((a + 0.05 * rng.standard_normal(shape)).astype(np.float32))
    ta, tb = dev(a), dev(b)
    e1, r1 = psa.l2_distance(ta, tb)
    e2, r2 = psa.l2_distance(ta, tb)
    gu.torch().cuda.synchronize()
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    ref_e = ((a64 - b64) ** 2).sum(axis=(2, 3))
    ref_r = (b64 ** 2).sum(axis=(2, 3))
    np.testing.assert_allclose(e1.cpu().numpy(), ref_e, rtol=1e-5)
    np.testing.assert_allclose(r1.cpu().numpy(), ref_r, rtol=1e-5)
    assert gu.torch().equal(e1, e2) and gu.torch().equal(r1, r2)          # fixed reduction order
    e0, _ = psa.l2_distance(tb, tb)
    gu.torch().cuda.synchronize()
    assert (e0.cpu().numpy() == 0).all()


def test_scores_against_oracle_and_selection():
    cfg = get_config("tiny")                                # 4x16x16, d = 64, block 64, 2 heads
    grid = gu.grid_of(cfg)
    q, k, v = gu.device_qkv("tiny")
    cands = candidates("tiny", 24)
    full = (4, 0, INF, 4, 0, INF)                           # every block: loss exactly 0
    cands = [c[:23] + [full] for c in cands]
    res = search.score(q, k, v, grid, cfg.block, cands, cfg.scale)
    qn, kn, vn = (x.float().cpu().numpy() for x in (q, k, v))
    alpha_checked = 0
    for h in range(cfg.heads):
        keeps = oracle.blockmap(cands[h], cfg.frames, cfg.height, cfg.width, cfg.n_text, cfg.block)
        ref = osearch.head_results(qn[0, h], kn[0, h], vn[0, h], keeps, cfg.block, cfg.scale)
        ref_loss = np.array([l for l, _ in ref])
        ref_sp = np.array([s for _, s in ref])
        assert np.array_equal(res.sparsity[h], ref_sp)
        # Each output is within tau = REL_L2_TOL of the oracle relative to its own norm, and
        # |O_M| <= |O_full| (1 + loss): the relative distance moves by at most tau (2 + 2 loss).
        bound = gu.REL_L2_TOL * (2.0 + 2.0 * ref_loss)
        assert (np.abs(res.loss[h] - ref_loss) <= bound).all()
        assert res.loss[h][-1] == 0.0
        print("head %d: max |loss - oracle| %.2e (losses %.3f..%.3f)"
              % (h, np.abs(res.loss[h] - ref_loss).max(), ref_loss.min(), ref_loss.max()))
        one = search.HeadResults([cands[h]], res.loss[h:h + 1], res.sparsity[h:h + 1])
        # Where no loss lies within its bound of alpha, both sides qualify the same candidates,
        # so they select the same one.
        s = np.sort(ref_loss)
        for alpha in 0.5 * (s[1:] + s[:-1]):
            if (np.abs(ref_loss - alpha) > bound).all():
                assert search.select(one, alpha)[0] == osearch.select_alpha(ref, alpha)
                alpha_checked += 1
        for target in (0.2, 0.5, 0.8):
            pick = search.select_target(one, target)[0]
            assert res.sparsity[h][pick] >= target or res.sparsity[h][pick] == res.sparsity[h].max()
    assert alpha_checked > 0
