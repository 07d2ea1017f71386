"""Every row of the full-size workloads against the oracle, within one bf16 ulp, on structured
inputs, in the launch configuration the benchmark times.

With Q = 0 every score is 0, so each key a row keeps gets weight exactly 1 (in the kernel too:
exp2(0) = 1, and the normaliser and the P V products are sums of small integers, exact in fp32):
O is the mean of V over the row's kept keys (Algorithm 2 over the KV blocks GetKVBlocks lists,
keys past the end of the sequence set to -inf).  V is 0/1 and each channel counts one class of
keys, with a per-head shift h:

  channel c < 64   -- keys of key blocks kb with (kb + h) mod 64 == c;
  channel c >= 64  -- keys at position p of their block with (p + h) mod 64 == c - 64;

so O[i, c] = (kept keys of the class) / (all kept keys of row i), a ratio of integers below 2^24
that the kernel forms up to the rounding of 1/l, of the product and of the bf16 store, i.e.
within one bf16 ulp of the exact value.  Dropping, repeating or misplacing one key block in any
row changes a block class by a whole block; admitting a key past the end of the sequence, or
dropping one of the partial last block, changes a position class; a swap of heads changes the
shift.  LSE = ln(kept keys) exactly.  The outputs start as NaN, so a row the kernel never writes
fails.  The expected values come from the oracle's block map (pinned bit-exact against the
paper's Algorithm 1); on sampled rows they are also checked to equal the oracle's attention of
the same inputs exactly.
"""
import numpy as np
import pytest

import oracle
import paper_2609_37001_amd as psa
from workloads import get_config
from workloads.configs import SWEEP_TARGETS

import gpu_util as gu

pytestmark = pytest.mark.gpu
INF = 0x7FFFFFFF
D = 128


def indicator_v_device(heads, n, block):
    """V [1, heads, n, 128] bf16 on cuda:0 (the classes above)."""
    torch = gu.torch()
    j = torch.arange(n, device="cuda:0")
    hs = torch.arange(heads, device="cuda:0")[:, None]
    blk = ((j // block)[None, :] + hs) % 64
    pos = 64 + ((j % block)[None, :] + hs) % 64
    v = torch.zeros((1, heads, n, D), dtype=torch.bfloat16, device="cuda:0")
    v.scatter_(3, blk[None, :, :, None], 1.0)
    v.scatter_(3, pos[None, :, :, None], 1.0)
    return v


def indicator_v_host(h, n, block):
    """V [n, 128] float64 of head h (the same classes, built on the host)."""
    j = np.arange(n)
    v = np.zeros((n, D))
    v[j, ((j // block) + h) % 64] = 1.0
    v[j, 64 + ((j % block) + h) % 64] = 1.0
    return v


def expected_means(keep, h, n, block):
    """O of every query block of head h under its kept-block row `keep` [nb, nb] (float64
    [nb, 128]: the share of each key class among the kept keys; 0 for a row that keeps nothing)
    and the kept key count of each query block."""
    nb = keep.shape[0]
    lens = np.minimum(block, n - block * np.arange(nb)).astype(np.float64)
    counts = np.zeros((nb, D))
    counts[np.arange(nb), (np.arange(nb) + h) % 64] = lens
    for p in range(block):
        counts[:, 64 + (p + h) % 64] += (p < lens)
    kept = keep.astype(np.float64)
    total = kept @ lens
    num = kept @ counts
    mean = np.divide(num, total[:, None], out=np.zeros_like(num), where=total[:, None] > 0)
    return mean, total


def bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (x > 0): 8 significant bits."""
    return np.exp2(np.floor(np.log2(x)) - 7)


def check_head(o_bits, lse, keep, h, n, block):
    """All rows of one head: rows of a query block are identical, and each block's row is within
    one bf16 ulp of the expected mean; returns (elements not correctly rounded, worst ulp error)."""
    nb = keep.shape[0]
    mean, total = expected_means(keep, h, n, block)
    full = (n // block) * block
    first = np.empty((nb, D), dtype=np.uint16)
    if full:
        blocks = o_bits[:full].reshape(n // block, block, D)
        assert (blocks == blocks[:, :1, :]).all(), "head %d: rows of one query block differ" % h
        first[:n // block] = blocks[:, 0]
    if full < n:
        tail = o_bits[full:]
        assert (tail == tail[:1]).all(), "head %d: rows of the last query block differ" % h
        first[-1] = tail[0]
    got = (first.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.isfinite(got).all(), "head %d: unwritten or non-finite output" % h
    zero = mean == 0
    assert (got[zero] == 0).all(), "head %d: a class with no kept key is not 0" % h
    err = np.abs(got[~zero] - mean[~zero]) / bf16_ulp(mean[~zero])
    worst = float(err.max()) if err.size else 0.0
    assert worst <= 1.0, "head %d: %.3f bf16 ulp from the kept-key mean" % (h, worst)
    rne = (mean.astype(np.float32).view(np.uint32) + 0x7FFF +
           ((mean.astype(np.float32).view(np.uint32) >> 16) & 1)) >> 16
    off = int((first.astype(np.uint32) != rne).sum())
    row_total = total[np.arange(n) // block]
    live = row_total > 0
    assert np.isneginf(lse[~live]).all(), "head %d: empty rows must give lse = -inf" % h
    assert np.abs(lse[live] - np.log(row_total[live])).max(initial=0.0) <= 1e-5, "head %d: lse" % h
    return off, worst


def check_against_oracle(keep, picks, n, block):
    """The expected means equal the oracle's attention of Q = 0 and the indicator V exactly (on
    the first and last row of each sampled query block)."""
    by_head = {}
    for h, qb in picks:
        by_head.setdefault(h, []).append(qb)
    zeros = np.zeros((n, D))
    for h, qbs in by_head.items():
        rows = np.unique([r for qb in qbs for r in (qb * block, min(n, (qb + 1) * block) - 1)])
        o_ref, lse_ref = oracle.masked_attention(zeros, zeros, indicator_v_host(h, n, block), keep[h], block,
                                                 1.0, rows)
        mean, total = expected_means(keep[h], h, n, block)
        assert np.array_equal(o_ref, mean[rows // block]), "head %d: closed form differs from the oracle" % h
        live = total[rows // block] > 0
        assert np.isneginf(lse_ref[~live]).all()
        assert np.allclose(lse_ref[live], np.log(total[rows // block][live]), rtol=0, atol=1e-12)


def run_structured(grid, block, params, keep, k, label, dense=False):
    """Q = 0, the workload's K, the indicator V; every row of every head checked."""
    torch = gu.torch()
    f, hh, ww, nt = grid
    n = f * hh * ww + nt
    heads = len(params)
    q0 = torch.zeros((1, heads, n, D), dtype=torch.bfloat16, device="cuda:0")
    v = indicator_v_device(heads, n, block)
    o = torch.full_like(q0, float("nan"))
    if dense:
        o, lse = psa.dense_fwd(q0, k, v, block, 0.1, out=o, return_lse=True)
    else:
        o, lse = psa.attention_fwd(q0, k, v, grid, block, params, 0.1, out=o, return_lse=True)
    torch.cuda.synchronize()
    del q0, v
    lse = lse.cpu().numpy()
    off = 0
    worst = 0.0
    for h in range(heads):
        bits = o[0, h].view(torch.int16).cpu().numpy().view(np.uint16)
        c, w = check_head(bits, lse[0, h], keep[h], h, n, block)
        off += c
        worst = max(worst, w)
    print("%s: %d heads x %d rows exact to one bf16 ulp (worst %.3f ulp); %d of %d block-row elements "
          "differ from the correctly rounded mean" % (label, heads, n, worst, off, heads * keep.shape[1] * D))


def workload_case(name, target=None):
    cfg = get_config(name)
    params = gu.params_of(name, target)
    grid = gu.grid_of(cfg)
    keep = gu.oracle_map(cfg, params)
    _, k, _ = gu.device_qkv("wan14b" if name == "sweep" else name)
    check_against_oracle(keep, gu.sample_blocks(cfg, keep, n_random=4), cfg.n_tokens, cfg.block)
    return cfg, params, grid, keep, k


@pytest.mark.parametrize("name", ["wan1_3b", "wan14b", "hunyuan"])
def test_workload_every_row(name):
    cfg, params, grid, keep, k = workload_case(name)
    run_structured(grid, cfg.block, params, keep, k, name)


@pytest.mark.parametrize("target", SWEEP_TARGETS)
def test_sweep_every_row(target):
    cfg, params, grid, keep, k = workload_case("sweep", target)
    run_structured(grid, cfg.block, params, keep, k, "sweep %.2f" % target)


def test_dense_every_row():
    """The dense baseline visits every key block of every row (Wan 2.1 14B shape)."""
    cfg = get_config("wan14b")
    nb = cfg.n_blocks
    keep = np.ones((cfg.heads, nb, nb), dtype=np.uint8)
    _, k, _ = gu.device_qkv("wan14b")
    run_structured(gu.grid_of(cfg), cfg.block, [None] * cfg.heads, keep, k, "dense wan14b", dense=True)


def test_largest_block_count_every_row():
    """nb = 7936 blocks of 128 (62 frames of 128 x 128 tokens), the pairing sorts at their largest
    size, one head of each leftover pairing order."""
    grid, block = (62, 128, 128, 0), 128
    params = [(1, 0, INF, 2, 0, INF), (3, 1, INF, 1, 0, 3)]
    keep = oracle.blockmap(params, *grid, block)
    n = 62 * 128 * 128
    torch = gu.torch()
    k = torch.randn((1, 2, n, D), device="cuda:0", generator=torch.Generator("cuda:0").manual_seed(3)).bfloat16()
    picks = [(0, 0), (1, 3967), (1, 7935), (0, 5000)]
    check_against_oracle(keep, picks, n, block)
    run_structured(grid, block, params, keep, k, "largest block count")
