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


def check_scores(qn, kn, vn, grid, block, scale, cands, res):
    """Candidate losses of search.score against the oracle's (Algorithm 3), per head and
    candidate within a bound derived from the measured error of the library's outputs: with a, b
    the device outputs of the candidate and of full attention and a', b' the oracle's,
    |(|a - b| / |b|) - (|a' - b'| / |b'|)| <= (|a - a'| + |b - b'| (1 + loss')) / |b| (triangle
    inequality for the numerator, |b'| - |b| for the denominator), plus 1e-5 relative for the fp32
    partial sums of the distance kernel.  Sparsities exact.  Returns (oracle results per head,
    bounds [heads, C])."""
    torch = gu.torch()
    f, hh, ww, nt = grid
    heads, n = qn.shape[1], qn.shape[2]
    n_cand = len(cands[0])
    q, k, v = dev(qn), dev(kn), dev(vn)
    full_d = psa.dense_fwd(q, k, v, block, scale).float().cpu().numpy()[0].astype(np.float64)
    outs = [psa.attention_fwd(q, k, v, grid, block, [cands[h][c] for h in range(heads)], scale)
            .float().cpu().numpy()[0].astype(np.float64) for c in range(n_cand)]
    torch.cuda.synchronize()
    nb = -(-n // block)
    refs, bounds, worst = [], np.zeros((heads, n_cand)), 0.0
    for h in range(heads):
        keeps = oracle.blockmap(cands[h], f, hh, ww, nt, block)
        ref = osearch.head_results(qn[0, h], kn[0, h], vn[0, h], keeps, block, scale)
        refs.append(ref)
        ref_loss = np.array([l for l, _ in ref])
        assert np.array_equal(res.sparsity[h], np.array([sp for _, sp in ref]))
        b_ref, _ = oracle.masked_attention(qn[0, h], kn[0, h], vn[0, h], np.ones((nb, nb)), block, scale)
        e_b, norm_b = np.linalg.norm(full_d[h] - b_ref), np.linalg.norm(full_d[h])
        for c in range(n_cand):
            a_ref, _ = oracle.masked_attention(qn[0, h], kn[0, h], vn[0, h], keeps[c], block, scale)
            e_a = np.linalg.norm(outs[c][h] - a_ref)
            bounds[h, c] = (e_a + e_b * (1.0 + ref_loss[c])) / norm_b + 1e-5 * ref_loss[c] + 1e-9
            diff = abs(res.loss[h][c] - ref_loss[c])
            assert diff <= bounds[h, c], "head %d candidate %d: |loss - oracle| %.3e > bound %.3e" % (
                h, c, diff, bounds[h, c])
            worst = max(worst, diff / bounds[h, c])
        print("head %d: losses %.3f..%.3f, max |loss - oracle| %.2e, bounds %.2e..%.2e"
              % (h, ref_loss.min(), ref_loss.max(), np.abs(res.loss[h] - ref_loss).max(), bounds[h].min(),
                 bounds[h].max()))
    print("largest |loss - oracle| / bound: %.3f" % worst)
    return refs, bounds


def check_selection(res, refs, bounds):
    """Wherever the oracle's choice is separated from the alternatives by more than the bounds,
    the host selection over the device losses makes the same choice (alpha and target sparsity)."""
    checked = 0
    for h, ref in enumerate(refs):
        ref_loss = np.array([l for l, _ in ref])
        bnd = bounds[h]
        one = search.HeadResults([res.candidates[h]], res.loss[h:h + 1], res.sparsity[h:h + 1])
        s = np.sort(ref_loss)
        for alpha in 0.5 * (s[1:] + s[:-1]):
            if (np.abs(ref_loss - alpha) > bnd).all():
                assert search.select(one, alpha)[0] == osearch.select_alpha(ref, alpha)
                checked += 1
        sp = res.sparsity[h]
        for target in (0.2, 0.5, 0.8):
            ok = np.nonzero(sp >= target)[0]
            if len(ok) == 0:
                ok = np.nonzero(sp == sp.max())[0]
            best = ok[np.argmin(ref_loss[ok])]
            if all(ref_loss[j] - ref_loss[best] > bnd[j] + bnd[best] for j in ok if j != best):
                assert search.select_target(one, target)[0] == osearch.select_target(ref, target) == best
                checked += 1
    assert checked > 0


def test_scores_against_oracle_and_selection():
    """Block 64, head_dim 64 (the one-row engine): the tiny workload's 2 heads x 24 candidates
    (23 from the paper's candidate space and the full map, whose loss is exactly 0)."""
    cfg = get_config("tiny")                                # 4x16x16, d = 64, block 64, 2 heads
    grid = gu.grid_of(cfg)
    q, k, v = gu.device_qkv("tiny")
    cands = candidates("tiny", 24)
    full = (4, 0, INF, 4, 0, INF)                           # every block: loss exactly 0
    cands = [c[:23] + [full] for c in cands]
    res = search.score(q, k, v, grid, cfg.block, cands, cfg.scale)
    qn, kn, vn = (x.float().cpu().numpy() for x in (q, k, v))
    refs, bounds = check_scores(qn, kn, vn, grid, cfg.block, cfg.scale, cands, res)
    assert (res.loss[:, -1] == 0.0).all()
    check_selection(res, refs, bounds)


def test_scores_pair_engine_against_oracle():
    """Block 128, head_dim 128 (the pair engine, the path of the video workloads): 3 heads x 13
    candidates (12 drawn from the paper's candidate space and the full map) on a 4 x 16 x 32 grid
    with 40 text tokens (17 blocks; 4 frames of 4 slots and a global text block)."""
    from workloads.params import S_OFFSETS, S_STRIDES, T_OFFSETS, T_STRIDES
    f, hh, ww, nt, block, d, heads, scale = 4, 16, 32, 40, 128, 128, 3, 0.15
    n = f * hh * ww + nt
    grid = (f, hh, ww, nt)
    tp, sp = f, -(-(hh * ww) // block)
    rng = np.random.default_rng(31)
    qn, kn, vn = (bf16_round(rng.standard_normal((1, heads, n, d)).astype(np.float32)) for _ in range(3))
    cands = []
    for _ in range(heads):
        seen = []
        while len(seen) < 12:
            m = (int(rng.integers(1, tp + 1)), int(rng.choice(T_OFFSETS)), int(rng.choice(T_STRIDES)),
                 int(rng.integers(1, sp + 1)), int(rng.choice(S_OFFSETS)), int(rng.choice(S_STRIDES)))
            if m not in seen:
                seen.append(m)
        cands.append(seen + [(tp, 0, INF, sp, 0, INF)])
    res = search.score(dev(qn), dev(kn), dev(vn), grid, block, cands, scale)
    refs, bounds = check_scores(qn, kn, vn, grid, block, scale, cands, res)
    assert (res.loss[:, -1] == 0.0).all()
    check_selection(res, refs, bounds)
