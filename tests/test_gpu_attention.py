"""GPU attention parity against the oracle (sampled rows at full size, full tensors when small)."""
import numpy as np
import pytest

import oracle
import paper_2609_37001_amd as psa
from workloads import get_config
from workloads.inputs import bf16_round

import gpu_util as gu

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def dev(x):
    t = gu.torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").bfloat16()


def full_compare(q, k, v, keep, block, scale, o, lse):
    """Every row of a [B, H, N, d] problem against the oracle (gpu_util.Parity)."""
    return gu.compare_all(q, k, v, keep, block, scale, o.float().cpu().numpy(), lse.cpu().numpy())


def random_problem(b, h, n, d, seed):
    rng = np.random.default_rng(seed)
    return [bf16_round(rng.standard_normal((b, h, n, d)).astype(np.float32)) for _ in range(3)]


def test_tiny_config_full():
    cfg = get_config("tiny")
    params = gu.params_of("tiny")
    q, k, v = gu.device_qkv("tiny")
    o, lse, kept = psa.attention_fwd(q, k, v, gu.grid_of(cfg), cfg.block, params, cfg.scale,
                                     return_lse=True, return_kept_per_row=True)
    gu.torch().cuda.synchronize()
    bmap = gu.oracle_map(cfg, params)
    assert (kept.cpu().numpy() == oracle.kept_per_row(bmap)).all()
    qn, kn, vn = (x.float().cpu().numpy() for x in (q, k, v))
    full_compare(qn, kn, vn, bmap, cfg.block, cfg.scale, o, lse).check("tiny:")


@pytest.mark.parametrize("d,block", [(64, 64), (128, 128), (128, 64), (64, 128)])
def test_shapes_ragged_text_batch(d, block):
    """Every (head_dim, block) variant on a ragged sequence with text tokens, batch 2, 5 heads
    (including an empty-row offset head and a full head)."""
    f, hh, ww, nt = 3, 10, 13, 37            # N = 427: several blocks and a ragged tail
    n = f * hh * ww + nt
    params = [(1, 1, INF, 1, 0, INF), (2, 0, INF, 3, 1, 5), (1, 0, 2, 2, -1, 3), (3, 0, INF, 4, 0, INF),
              (1, -1, INF, 1, 1, INF)]
    q, k, v = random_problem(2, len(params), n, d, seed=d + block)
    keep = oracle.blockmap(params, f, hh, ww, nt, block)
    o, lse = psa.attention_fwd(dev(q), dev(k), dev(v), (f, hh, ww, nt), block, params, 0.11, return_lse=True)
    gu.torch().cuda.synchronize()
    full_compare(q, k, v, keep, block, 0.11, o, lse).check("d=%d block=%d:" % (d, block))


def test_long_text_rows_scheduled_first():
    """Text rows keep every key block while the video rows keep one block plus the text: the
    text rows' work is far above three times the mean, so the plan lists them ahead of the
    head-ordered ranges.  Batch 2 x 6 heads x 3 text blocks = 36 such items over 8 queues."""
    f, hh, ww, nt = 8, 16, 32, 300
    n = f * hh * ww + nt
    params = [(1, 0, INF, 1, 0, INF)] * 4 + [(1, 1, INF, 1, 0, INF), (2, 0, INF, 1, 0, INF)]
    q, k, v = random_problem(2, len(params), n, 64, seed=23)
    keep = oracle.blockmap(params, f, hh, ww, nt, 128)
    rows = oracle.kept_per_row(keep) + 2
    assert (rows[:, -3:] * rows.size > 3 * rows.sum()).all() and (rows[:, :-3] * rows.size <= 3 * rows.sum()).all()
    o, lse = psa.attention_fwd(dev(q), dev(k), dev(v), (f, hh, ww, nt), 128, params, 0.1, return_lse=True)
    gu.torch().cuda.synchronize()
    full_compare(q, k, v, keep, 128, 0.1, o, lse).check("long text rows:")


@pytest.mark.parametrize("d,block", [(64, 64), (128, 128)])
def test_dense_full(d, block):
    n = 3 * block + 29
    q, k, v = random_problem(1, 3, n, d, seed=7)
    nb = -(-n // block)
    keep = np.ones((3, nb, nb), np.uint8)
    o, lse = psa.dense_fwd(dev(q), dev(k), dev(v), block, 0.09, return_lse=True)
    gu.torch().cuda.synchronize()
    full_compare(q, k, v, keep, block, 0.09, o, lse).check("dense d=%d:" % d)


@pytest.mark.parametrize("d,block", [(64, 64), (128, 128), (128, 64), (64, 128)])
def test_dense_persistent_equals_fixed_grid(d, block):
    """With a workspace the dense call runs a persistent grid over armed per-XCD queues; without
    one a fixed grid.  Same bits, including a reused workspace on the second call."""
    torch = gu.torch()
    n = 5 * block + 37
    q, k, v = (dev(x) for x in random_problem(2, 3, n, d, seed=d + 3 * block))
    o_f, l_f = psa.dense_fwd(q, k, v, block, 0.1, return_lse=True, balanced=False)
    ws = torch.empty(psa.dense_workspace_size(), dtype=torch.uint8, device="cuda:0")
    for _ in range(2):
        o_p, l_p = psa.dense_fwd(q, k, v, block, 0.1, return_lse=True, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(o_p, o_f) and torch.equal(l_p, l_f)


def test_full_density_sparse_equals_dense_bitwise():
    f, hh, ww = 4, 16, 24
    n = f * hh * ww
    q, k, v = (dev(x) for x in random_problem(1, 3, n, 128, seed=11))
    params = [(4, 0, INF, 3, 0, INF), (1, 0, 1, 1, 0, 1), (5, 1, 2, 7, -1, 3)]
    keep = oracle.blockmap(params, f, hh, ww, 0, 128)
    assert keep.all()
    o_s, l_s = psa.attention_fwd(q, k, v, (f, hh, ww, 0), 128, params, 0.08, return_lse=True)
    o_d, l_d = psa.dense_fwd(q, k, v, 128, 0.08, return_lse=True)
    gu.torch().cuda.synchronize()
    assert gu.torch().equal(o_s, o_d) and gu.torch().equal(l_s, l_d)


def test_deterministic():
    cfg = get_config("tiny")
    params = gu.params_of("tiny")
    q, k, v = gu.device_qkv("tiny")
    a = psa.attention_fwd(q, k, v, gu.grid_of(cfg), cfg.block, params, cfg.scale)
    b = psa.attention_fwd(q, k, v, gu.grid_of(cfg), cfg.block, params, cfg.scale)
    gu.torch().cuda.synchronize()
    assert gu.torch().equal(a, b)


def test_constant_values_and_empty_rows():
    f, hh, ww = 4, 8, 16                      # HW = 128: one block per frame
    n = f * hh * ww
    q, k, _ = random_problem(1, 1, n, 128, seed=5)
    v = np.ones_like(q)
    params = [(1, 1, INF, 1, 0, INF)]        # dt = 1 only: the last frame has no keys
    o, lse = psa.attention_fwd(dev(q), dev(k), dev(v), (f, hh, ww, 0), 128, params, 0.1, return_lse=True)
    gu.torch().cuda.synchronize()
    o = o.float().cpu().numpy()[0, 0]
    lse = lse.cpu().numpy()[0, 0]
    assert (o[: 3 * 128] == 1.0).all()
    assert (o[3 * 128:] == 0).all() and np.isneginf(lse[3 * 128:]).all()


def test_plan_once_run_many_equals_fwd():
    """One plan serves repeated runs (the queue counters re-arm): every run returns the bits of
    attention_fwd, for two different inputs over the same plan."""
    torch = gu.torch()
    f, hh, ww, nt = 3, 10, 13, 37
    params = [(2, 0, INF, 3, 1, 5), (1, 0, 2, 2, -1, 3), (1, 1, INF, 1, 0, INF)]
    grid = (f, hh, ww, nt)
    ws, kept = psa.plan(params, grid, 64, batch=2, return_kept_per_row=True)
    keep = oracle.blockmap(params, f, hh, ww, nt, 64)
    assert (kept.cpu().numpy() == oracle.kept_per_row(keep)).all()
    for seed in (3, 4):
        q, k, v = (dev(x) for x in random_problem(2, 3, f * hh * ww + nt, 128, seed=seed))
        ref, lref = psa.attention_fwd(q, k, v, grid, 64, params, 0.1, return_lse=True)
        for _ in range(3):
            o, l = psa.run(q, k, v, grid, 64, ws, 0.1, return_lse=True)
            torch.cuda.synchronize()
            assert torch.equal(o, ref) and torch.equal(l, lref)


def test_run_without_matching_plan_writes_nothing():
    """The kernel checks the plan header: an unplanned workspace, or one planned for another
    grid, leaves o and lse untouched (checked through the C ABI, past the binding's own check)."""
    import ctypes
    from paper_2609_37001_amd import _lib
    torch = gu.torch()
    grid, other = (2, 8, 16, 0), (2, 8, 16, 5)
    n = 2 * 8 * 16
    q, k, v = (dev(x) for x in random_problem(1, 1, n, 128, seed=9))
    size = max(psa.workspace_size(1, 1, grid, 128), psa.workspace_size(1, 1, other, 128))
    vp = lambda t: ctypes.c_void_p(t.data_ptr())

    def raw_run(ws, o, lse):
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        return _lib.lib().psa_attention_run(vp(q), vp(k), vp(v), vp(o), 1, 1, 128,
                                            _lib.grid_of(*grid), 128, 0.1, vp(ws), size, vp(lse), stream)

    ws = torch.zeros(size, dtype=torch.uint8, device="cuda:0")          # no plan at all
    o = torch.full_like(q, 7.0)
    lse = torch.full((1, 1, n), 3.0, device="cuda:0")
    assert raw_run(ws, o, lse) == _lib.PSA_OK
    torch.cuda.synchronize()
    assert (o == 7.0).all() and (lse == 3.0).all()
    params = [(1, 0, INF, 1, 0, INF)]
    assert _lib.lib().psa_attention_plan(1, 1, _lib.grid_of(*other), 128, _lib.stripes(params),
                                         vp(ws), size, None,
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)) == 0
    assert raw_run(ws, o, lse) == _lib.PSA_OK                           # planned for 5 text tokens
    torch.cuda.synchronize()
    assert (o == 7.0).all() and (lse == 3.0).all()
    with pytest.raises(ValueError):
        psa.run(q, k, v, grid, 128, psa.Workspace(1, 1, grid, 128, "cuda:0"))


def test_layer_attention_follows_the_timestep_policy():
    """Sec. 4 setup: the first 20 % of the denoising steps stay dense.  Over 10 steps the exempt
    steps 0-1 give full attention and steps 2-9 the layer's stripes, each against the oracle (full
    map, and the masked attention of the stripes' map); the layer plans once, and its outputs carry
    the bits of the direct dense and sparse calls."""
    from paper_2609_37001_amd.policy import LayerAttention, TimestepPolicy
    torch = gu.torch()
    f, hh, ww, nt = 4, 16, 24, 40
    grid = (f, hh, ww, nt)
    n = f * hh * ww + nt
    params = [(1, 0, INF, 2, 0, INF), (2, 1, 3, 1, 0, INF)]
    qn, kn, vn = random_problem(1, 2, n, 128, seed=21)
    q, k, v = dev(qn), dev(kn), dev(vn)
    layer = LayerAttention(params, grid, 128, 1, TimestepPolicy(10, 0.2), scale=0.1)
    assert [layer.policy.is_dense(s) for s in range(10)] == [True] * 2 + [False] * 8
    outs = [layer(q, k, v, step) for step in range(10)]
    dense = psa.dense_fwd(q, k, v, 128, 0.1)
    sparse = psa.attention_fwd(q, k, v, grid, 128, params, 0.1)
    torch.cuda.synchronize()
    ws = layer.workspace
    assert all(torch.equal(o, dense) for o in outs[:2])
    assert all(torch.equal(o, sparse) for o in outs[2:])
    assert layer.workspace is ws
    nb = -(-n // 128)
    full = np.ones((2, nb, nb), dtype=np.uint8)
    keep = oracle.blockmap(params, f, hh, ww, nt, 128)
    assert not keep.all()
    on = lambda o: o.float().cpu().numpy()
    gu.compare_all(qn, kn, vn, full, 128, 0.1, on(outs[0]), None).check("exempt step 0 vs full attention:")
    gu.compare_all(qn, kn, vn, keep, 128, 0.1, on(outs[5]), None).check("step 5 vs the stripes' map:")
