"""Edge cases of the sparse attention on the GPU against the oracle: a one-token sequence, the
largest block count the library accepts, the largest batch x heads, degenerate stripes (every
block kept, whole axes, offsets beyond the grid) and input validation in the binding."""
import numpy as np
import pytest

import oracle
import paper_2609_37001_amd as psa
from paper_2609_37001_amd import _lib
from workloads.inputs import bf16_round

import gpu_util as gu

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF


def dev(x):
    t = gu.torch()
    return t.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda:0").bfloat16()


def check(q, k, v, keep, block, scale, o, lse, rows=None, label=""):
    """Rows `rows` (all if None) of every (batch, head) against the oracle (gpu_util.Parity)."""
    if rows is not None:
        o, lse = o[:, :, rows], lse[:, :, rows]
    gu.compare_all(q, k, v, keep, block, scale, o, lse, rows=rows).check(label)


@pytest.mark.parametrize("d,block", [(64, 64), (128, 128)])
def test_one_token(d, block):
    rng = np.random.default_rng(d)
    q, k, v = (bf16_round(rng.standard_normal((1, 2, 1, d)).astype(np.float32)) for _ in range(3))
    params = [(1, 0, INF, 1, 0, INF), (3, 2, 3, 1, -1, 5)]       # the second keeps nothing
    o, lse = psa.attention_fwd(dev(q), dev(k), dev(v), (1, 1, 1), block, params, 0.125, return_lse=True)
    gu.torch().cuda.synchronize()
    on = o.float().cpu().numpy()
    assert np.array_equal(on[0, 0, 0], v[0, 0, 0])              # softmax over one key: V itself
    assert (on[0, 1] == 0).all() and np.isneginf(lse[0, 1].cpu().numpy()).all()
    keep = oracle.blockmap(params, 1, 1, 1, 0, block)
    check(q, k, v, keep, block, 0.125, on, lse.cpu().numpy())


def test_largest_block_count():
    """nb = PSA_MAX_BLOCKS = 7936 blocks of 128 (62 frames of 128 x 128 tokens, N = 1015808).  The
    first head pairs its leftover query blocks in index order, the second (T_w > S_w) slot-major:
    the pairing kernel's sorts run at their largest size."""
    f, hh, ww, block = 62, 128, 128, 128
    n = f * hh * ww
    assert psa.num_blocks((f, hh, ww), block) == _lib.MAX_BLOCKS
    rng = np.random.default_rng(5)
    q, k, v = (bf16_round(rng.standard_normal((1, 2, n, 128)).astype(np.float32)) for _ in range(3))
    params = [(1, 0, INF, 2, 0, INF), (3, 1, INF, 1, 0, 3)]      # own frame / three frames, nearby slots
    torch = gu.torch()
    qd = dev(q)
    o = torch.full_like(qd, float("nan"))                         # a row never written stays NaN
    o, lse, kept = psa.attention_fwd(qd, dev(k), dev(v), (f, hh, ww), block, params, 0.09, out=o,
                                     return_lse=True, return_kept_per_row=True)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    keep = oracle.blockmap(params, f, hh, ww, 0, block)
    assert np.array_equal(kept.cpu().numpy(), oracle.kept_per_row(keep))
    rows = np.concatenate([np.arange(0, 8), np.arange(n // 2, n // 2 + 8), np.arange(n - 8, n)])
    check(q, k, v, keep, block, 0.09, o.float().cpu().numpy(), lse.cpu().numpy(), rows)
    with pytest.raises(ValueError):                               # tensors shorter than the grid
        psa.attention_fwd(dev(q[:, :, :128]), dev(k[:, :, :128]), dev(v[:, :, :128]), (f, hh, ww), block,
                          params, 0.09)


@pytest.mark.parametrize("block,d", [(64, 64), (128, 128)])
def test_largest_batch_heads(block, d):
    """batch x heads = PSA_MAX_BATCH_HEADS = 1024 (4 x 256 heads, each with its own stripes); block
    128 runs the pair engine, one pairing workgroup per head."""
    b, h, grid = 4, 256, (2, 8, 16, 5)
    n = 2 * 8 * 16 + 5
    rng = np.random.default_rng(9)
    params = [(int(rng.integers(1, 3)), int(rng.choice([0, 1, -1])), int(rng.choice([1, 2, INF])),
               int(rng.integers(1, 3)), int(rng.choice([0, 1])), int(rng.choice([1, 3, INF]))) for _ in range(h)]
    q, k, v = (bf16_round(rng.standard_normal((b, h, n, d)).astype(np.float32)) for _ in range(3))
    torch = gu.torch()
    qd = dev(q)
    o = torch.full_like(qd, float("nan"))
    o, lse = psa.attention_fwd(qd, dev(k), dev(v), grid, block, params, 0.1, out=o, return_lse=True)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all())
    keep = oracle.blockmap(params, *grid, block)
    check(q, k, v, keep, block, 0.1, o.float().cpu().numpy(), lse.cpu().numpy())


@pytest.mark.parametrize("nt", [0, 70])
def test_degenerate_stripes(nt):
    """Stride 1 and width >= stride keep whole axes; offsets beyond the grid keep no video pair
    (with text, rows still attend the global text blocks)."""
    f, hh, ww, block = 3, 8, 24, 64
    n = f * hh * ww + nt
    big = 1 << 24
    params = [(1, 0, 1, 1, 0, 1), (4, 0, 2, 7, 0, 3), (1, big, INF, 1, 0, INF), (1, 0, INF, 1, -big, INF),
              (1, -big, 1, 2, big, 1)]
    rng = np.random.default_rng(nt)
    q, k, v = (bf16_round(rng.standard_normal((1, len(params), n, 128)).astype(np.float32)) for _ in range(3))
    o, lse = psa.attention_fwd(dev(q), dev(k), dev(v), (f, hh, ww, nt), block, params, 0.1, return_lse=True)
    gu.torch().cuda.synchronize()
    keep = oracle.blockmap(params, f, hh, ww, nt, block)
    assert keep[0].all() and keep[1].all()
    check(q, k, v, keep, block, 0.1, o.float().cpu().numpy(), lse.cpu().numpy())


def test_binding_rejects_bad_tensors():
    torch = gu.torch()
    x = torch.zeros((1, 1, 128, 128), dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(TypeError):
        psa.attention_fwd(x.float(), x, x, (1, 8, 16), 128, [(1, 0, INF, 1, 0, INF)])
    with pytest.raises(ValueError):
        psa.attention_fwd(x.transpose(2, 3), x, x, (1, 8, 16), 128, [(1, 0, INF, 1, 0, INF)])
    with pytest.raises(ValueError):
        psa.attention_fwd(x, x, x, (1, 8, 16), 128, [(1, 0, INF, 1, 0, INF)] * 2)
    with pytest.raises(psa.PsaError):
        psa.attention_fwd(x[:, :, :, :96].contiguous(), x[:, :, :, :96].contiguous(),
                          x[:, :, :, :96].contiguous(), (1, 8, 16), 128, [(1, 0, INF, 1, 0, INF)])


def test_binding_rejects_misaligned_tensors():
    """A contiguous view that starts one element into its storage is not 16-byte aligned: the
    library rejects it (PSA_ERR_INVALID) before any kernel runs, and the binding raises."""
    torch = gu.torch()
    x = torch.zeros((1, 1, 128, 128), dtype=torch.bfloat16, device="cuda:0")
    flat = torch.zeros(128 * 128 + 8, dtype=torch.bfloat16, device="cuda:0")
    y = flat[1:1 + 128 * 128].view(1, 1, 128, 128)
    assert y.is_contiguous() and y.data_ptr() % 16 != 0
    stripes = [(1, 0, INF, 1, 0, INF)]
    for args in ((y, x, x), (x, y, x), (x, x, y)):
        with pytest.raises(psa.PsaError) as e:
            psa.attention_fwd(*args, (1, 8, 16), 128, stripes)
        assert e.value.status == _lib.PSA_ERR_INVALID
    with pytest.raises(psa.PsaError):
        psa.dense_fwd(y, x, x, 128, 0.1)
    with pytest.raises(psa.PsaError):
        psa.attention_fwd(x, x, x, (1, 8, 16), 128, stripes, out=y)
    torch.cuda.synchronize()
    o = psa.attention_fwd(x, x, x, (1, 8, 16), 128, stripes)     # the library still works
    torch.cuda.synchronize()
    assert torch.isfinite(o.float()).all()
