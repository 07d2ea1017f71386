"""Oracle, part 3: PSABlock granularity, the PSABlock-centric layout and 3D padding (test
infrastructure only).

What is computed, from Sec. 3.2 ("Hardware-Aware Design" and "3D-Padding for Resolution
Flexibility") and Algorithm 1:

* A PSABlock is a bt x bh x bw tile of the (T, H, W) video grid; the mask is decided per pair of
  PSABlocks, never per token.
* 3D padding: each axis is padded to the smallest multiple of its block size, so the grid of
  PSABlocks is T' = ceil(T / bt), H' = ceil(H / bh), W' = ceil(W / bw) and the padded extents are
  T' bt, H' bh, W' bw.
* Algorithm 1 runs on that coarse grid: PSABlock (t', h', w') has temporal coordinate t' and
  spatial coordinate s' = h' W' + w' (Algorithm 1 flattens the in-frame position, i mod HW; on
  the coarse grid the plane has H' W' cells).  Distances are key minus query.
* Text tokens, appended after the video tokens, are global (kept in every row and column), as
  in the one-dimensional reading.
* The PSABlock-centric layout orders the padded grid as (T', H', W', bt, bh, bw): PSABlocks in
  row-major (t', h', w') order, and inside each PSABlock its tokens in row-major (t, h, w)
  order; padded positions hold zeros; the text tokens follow, in their own order.

Padded positions do not exist in the original token order; masking their scores with -inf
(Algorithm 2) is exactly their exclusion.  The plain definition of the attention therefore
works on the original tokens, each carrying the PSABlock it falls into: see
``oracle.masked_attention(..., groups=token_groups(...))``.
"""
import numpy as np

from .stripe import axis_condition


def psablock_grid(frames, height, width, pb):
    """((T', H', W'), (padded T, H, W)) for PSABlock shape pb = (bt, bh, bw)."""
    bt, bh, bw = (int(x) for x in pb)
    if min(bt, bh, bw) < 1 or min(frames, height, width) < 1:
        raise ValueError("grid and PSABlock sizes must be >= 1")
    coarse = (-(-frames // bt), -(-height // bh), -(-width // bw))
    return coarse, (coarse[0] * bt, coarse[1] * bh, coarse[2] * bw)


def token_groups(frames, height, width, n_text, pb):
    """Group of every original token, int64 [F*H*W + n_text]: the PSABlock index
    (t' H' + h') W' + w' of a video token, and n_P = T' H' W' (one global group) for text."""
    (tp, hp, wp), _ = psablock_grid(frames, height, width, pb)
    bt, bh, bw = pb
    t, h, w = np.meshgrid(np.arange(frames), np.arange(height), np.arange(width), indexing="ij")
    video = ((t // bt) * hp + (h // bh)) * wp + (w // bw)
    text = np.full(int(n_text), tp * hp * wp, dtype=np.int64)
    return np.concatenate([video.ravel().astype(np.int64), text])


def group_coordinates(frames, height, width, n_text, pb):
    """Per group: (t', s', is_global).  Groups 0 .. n_P - 1 are the PSABlocks in row-major
    (t', h', w') order; group n_P, present when n_text > 0, is the text."""
    (tp, hp, wp), _ = psablock_grid(frames, height, width, pb)
    n_p = tp * hp * wp
    g = np.arange(n_p)
    t = g // (hp * wp)
    s = g % (hp * wp)                         # h' W' + w'
    glob = np.zeros(n_p, dtype=bool)
    if n_text > 0:
        t = np.append(t, 0)
        s = np.append(s, 0)
        glob = np.append(glob, True)
    return t.astype(np.int64), s.astype(np.int64), glob


def psablock_map(params, frames, height, width, n_text, pb):
    """Kept (query group, key group) pairs, uint8 [heads, G, G], G = n_P (+1 with text)."""
    t, s, glob = group_coordinates(frames, height, width, n_text, pb)
    dt = t[None, :] - t[:, None]              # key minus query
    ds = s[None, :] - s[:, None]
    gl = glob[:, None] | glob[None, :]
    out = np.zeros((len(params), t.shape[0], t.shape[0]), dtype=np.uint8)
    for i, (tw, to, ts, sw, so, ss) in enumerate(params):
        if min(tw, ts, sw, ss) < 1:
            raise ValueError("widths and strides must be >= 1")
        out[i] = gl | (axis_condition(dt, tw, to, ts) & axis_condition(ds, sw, so, ss))
    return out


def to_blocks(x, frames, height, width, n_text, pb):
    """PSABlock-centric layout of one (batch, head): x [F*H*W + n_text, d] -> [T' H' W' bt bh bw
    + n_text, d], zeros at padded positions."""
    (tp, hp, wp), (tpad, hpad, wpad) = psablock_grid(frames, height, width, pb)
    bt, bh, bw = pb
    x = np.asarray(x)
    d = x.shape[1]
    n_video = frames * height * width
    grid = np.zeros((tpad, hpad, wpad, d), dtype=x.dtype)
    grid[:frames, :height, :width] = x[:n_video].reshape(frames, height, width, d)
    blocks = grid.reshape(tp, bt, hp, bh, wp, bw, d).transpose(0, 2, 4, 1, 3, 5, 6)
    return np.concatenate([blocks.reshape(-1, d), x[n_video:]], axis=0)


def from_blocks(xb, frames, height, width, n_text, pb):
    """Inverse of to_blocks: drops the padded positions."""
    (tp, hp, wp), (tpad, hpad, wpad) = psablock_grid(frames, height, width, pb)
    bt, bh, bw = pb
    xb = np.asarray(xb)
    d = xb.shape[1]
    n_blk = tpad * hpad * wpad
    grid = xb[:n_blk].reshape(tp, hp, wp, bt, bh, bw, d).transpose(0, 3, 1, 4, 2, 5, 6)
    grid = grid.reshape(tpad, hpad, wpad, d)[:frames, :height, :width]
    return np.concatenate([grid.reshape(-1, d), xb[n_blk:]], axis=0)
