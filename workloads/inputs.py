"""Seeded synthetic Q/K/V shaped like a video DiT attention layer.

Recipe (per batch element b, head h, tensor id 0/1/2 for Q/K/V):

1. draw float32 N(0,1) values of shape [N, d] from ``numpy.random.default_rng([seed, id, b, h])``,
   so every head can be regenerated on its own;
2. round to bf16 (round to nearest even);
3. for Q and K only, apply a 3D rotary position embedding to the video tokens: the head
   dimension is split into (t, h, w) channel ranges, adjacent channel pairs (2j, 2j+1) of an
   axis with d_a channels rotate by pos_a * theta^(-2j/d_a), theta = 10000; appended text
   tokens are not rotated;
4. round to bf16 again.

The returned float32 arrays hold exact bf16 values; ``bf16_bits`` gives their 16-bit patterns.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROPE_THETA = 10000.0


def bf16_round(x):
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(x):
    """16-bit patterns of float32 arrays that already hold bf16 values."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


def bits_to_float(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def rope_tables(cfg):
    """cos/sin tables [N_video, d/2] (float32) for the 3D rotary embedding of ``cfg``."""
    hw = cfg.height * cfg.width
    idx = np.arange(cfg.n_video, dtype=np.int64)
    pos = (idx // hw, (idx % hw) // cfg.width, idx % cfg.width)
    angles = []
    for p, d_axis in zip(pos, cfg.rope_split):
        j = np.arange(d_axis // 2, dtype=np.float64)
        freq = ROPE_THETA ** (-2.0 * j / d_axis)
        angles.append(p[:, None].astype(np.float64) * freq[None, :])
    ang = np.concatenate(angles, axis=1)
    assert ang.shape[1] * 2 == cfg.head_dim
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def _apply_rope(x, cos, sin):
    nv = cos.shape[0]
    xe = x[:nv, 0::2].copy()
    xo = x[:nv, 1::2].copy()
    x[:nv, 0::2] = xe * cos - xo * sin
    x[:nv, 1::2] = xe * sin + xo * cos
    return x


def _draw(cfg, tensor_id, b, h):
    rng = np.random.default_rng([cfg.seed, tensor_id, b, h])
    return bf16_round(rng.standard_normal((cfg.n_tokens, cfg.head_dim), dtype=np.float32))


def make_head_qkv(cfg, b, h, tables=None):
    """(q, k, v) float32 [N, d] holding exact bf16 values for batch element b, head h."""
    cos, sin = rope_tables(cfg) if tables is None else tables
    q = bf16_round(_apply_rope(_draw(cfg, 0, b, h), cos, sin))
    k = bf16_round(_apply_rope(_draw(cfg, 1, b, h), cos, sin))
    v = _draw(cfg, 2, b, h)
    return q, k, v


def make_qkv(cfg, heads=None, bits=True, workers=8):
    """Q, K, V for every batch element and the given heads (default all), shape [B, H, N, d].

    With ``bits=True`` the arrays are uint16 bf16 patterns (ready for device upload),
    otherwise float32 holding exact bf16 values.
    """
    heads = list(range(cfg.heads)) if heads is None else list(heads)
    tables = rope_tables(cfg)
    dtype = np.uint16 if bits else np.float32
    shape = (cfg.batch, len(heads), cfg.n_tokens, cfg.head_dim)
    out = [np.empty(shape, dtype) for _ in range(3)]

    def one(job):
        b, hi = job
        for t, x in enumerate(make_head_qkv(cfg, b, heads[hi], tables)):
            out[t][b, hi] = bf16_bits(x) if bits else x

    jobs = [(b, hi) for b in range(cfg.batch) for hi in range(len(heads))]
    with ThreadPoolExecutor(max_workers=max(1, workers)) as ex:
        list(ex.map(one, jobs))
    return tuple(out)
