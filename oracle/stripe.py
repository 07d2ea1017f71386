"""Oracle, part 1: the PSA stripe mask (test infrastructure only).

Definition followed: Algorithm 1 (PSA mask definition, IsAttending) in Sec. 3.2 of the paper,
with the unified representation M(T_w, T_o, T_s, S_w, S_o, S_s) of the same section.  For a
query q_i and a key k_j of a video laid out frame-major as (t, h, w):

    t = index div (H*W),  s = index mod (H*W)
    dt = t_k - t_q,       ds = s_k - s_q               (key minus query)
    keep  iff  (|dt - T_o| mod T_s) <= T_w - 1   and   (|ds - S_o| mod S_s) <= S_w - 1

An infinite stride ("a single diagonal", appendix on candidate initialisation) is
STRIDE_INF = 2^31 - 1: |x| mod STRIDE_INF == |x| for every distance that can occur.

Masking happens per block, never per token (Sec. 3.2, PSABlock paragraph).  Readings taken
where the paper does not fix the block geometry (the latent grids used here are flattened
frame-major and cut into 1D blocks of ``block`` consecutive tokens):

* block b covers tokens [b*B, min((b+1)*B, N)); its coordinates are those of its first token,
  t_b = (b*B) div HW and s_b = ((b*B) mod HW) div B, so parameters count frames and block
  slots.  At B = 1 this is Algorithm 1 token by token; when blocks tile frames exactly it is
  the coarse (T', S') grid of PSABlocks.
* text tokens appended after the N_video video tokens are global: a block holding any text
  token is kept in its whole row and its whole column.
"""
import numpy as np

STRIDE_INF = 2 ** 31 - 1


def axis_condition(delta, width, offset, stride):
    """One axis of Algorithm 1: (|delta - offset| mod stride) <= width - 1 (elementwise)."""
    d = np.abs(np.asarray(delta, dtype=np.int64) - np.int64(offset))
    return (d % np.int64(stride)) <= np.int64(width) - 1


def is_attending(i, j, m, height, width):
    """Algorithm 1 for one (query token i, key token j) pair of a pure video sequence."""
    hw = height * width
    t_q, s_q = i // hw, i % hw
    t_k, s_k = j // hw, j % hw
    if not axis_condition(t_k - t_q, m[0], m[1], m[2]):
        return False
    return bool(axis_condition(s_k - s_q, m[3], m[4], m[5]))


def block_coordinates(frames, height, width, n_text, block):
    """Per block: (t, s, length, is_global) arrays, using first-token coordinates."""
    hw = height * width
    n_video = frames * hw
    n = n_video + n_text
    nb = -(-n // block)
    start = np.arange(nb, dtype=np.int64) * block
    length = np.minimum(block, n - start)
    is_global = (n_text > 0) & (start + length > n_video)
    t = start // hw
    s = (start % hw) // block
    return t, s, length, is_global


def _check(params, block):
    for m in params:
        if len(m) != 6:
            raise ValueError("a stripe tuple has six integers")
        if m[0] < 1 or m[3] < 1 or m[2] < 1 or m[5] < 1:
            raise ValueError("widths and strides must be >= 1")
    if block < 1:
        raise ValueError("block must be >= 1")


def blockmap(params, frames, height, width, n_text, block):
    """Kept (query block, key block) pairs: uint8 array [heads, nb, nb], row = query block."""
    _check(params, block)
    t, s, _, is_global = block_coordinates(frames, height, width, n_text, block)
    nb = t.shape[0]
    out = np.zeros((len(params), nb, nb), dtype=np.uint8)
    dt = t[None, :] - t[:, None]          # key minus query; rows are query blocks
    ds = s[None, :] - s[:, None]
    forced = is_global[:, None] | is_global[None, :]
    for h, m in enumerate(params):
        keep = axis_condition(dt, m[0], m[1], m[2]) & axis_condition(ds, m[3], m[4], m[5])
        out[h] = keep | forced
    return out


def kept_per_row(bmap):
    """Kept key blocks per (head, query block), int32."""
    return np.asarray(bmap, dtype=np.int64).sum(axis=2).astype(np.int32)


def kept_per_head(bmap):
    """Kept tiles per head, int64."""
    return np.asarray(bmap, dtype=np.int64).sum(axis=(1, 2))
