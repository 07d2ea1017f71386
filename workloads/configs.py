"""The five attention workloads (shapes of the paper's video DiT attention layers).

* ``tiny``      -- 1 x 2 heads, d=64, latent grid 4x16x16 (N=1024), block 64.
* ``wan1_3b``   -- Wan 2.1 1.3B 480p layer: 1 x 12 heads, d=128, grid 21x30x52 (N=32760), block 128.
* ``wan14b``    -- Wan 2.1 14B 720p layer: 1 x 40 heads, d=128, grid 21x45x80 (N=75600), block 128.
* ``hunyuan``   -- HunyuanVideo 720p joint attention: 1 x 24 heads, d=128, grid 33x45x80 plus
                   256 text tokens appended (N=119056), block 128.
* ``sweep``     -- the Wan 2.1 14B shape with eight forced kept-tile densities.
* ``wan14b_3d`` -- the Wan 2.1 14B layer in the paper's own PSABlock layout: 3x8x16 PSABlocks,
                   the grid 3D-padded to 21x48x80 (appendix on mask-candidate initialisation),
                   attention tiles of 128 positions; same Q/K/V as ``wan14b``.

The model shapes follow the paper's experimental setup (Sec. 4, "Models"; the latent grids
21x45x80 and 33x45x80 appear in the appendix on mask-candidate initialisation).
"""
from dataclasses import dataclass


@dataclass(frozen=True)
class Config:
    name: str
    batch: int
    heads: int
    head_dim: int
    frames: int
    height: int
    width: int
    n_text: int
    block: int
    rope_split: tuple          # channels per axis (t, h, w) of the 3D rotary embedding
    density_band: tuple        # (lo, hi) of the per-head kept-tile density targets, or None
    seed: int = 0              # seed of the Q/K/V draws
    psablock: tuple = None     # (bt, bh, bw) for the PSABlock-centric layout; `block` is the tile

    @property
    def n_video(self) -> int:
        return self.frames * self.height * self.width

    @property
    def n_tokens(self) -> int:
        return self.n_video + self.n_text

    @property
    def n_blocks(self) -> int:
        return -(-self.n_tokens // self.block)

    @property
    def dense_flops(self) -> float:
        """4 N^2 d per (batch, head): the paper's FLOP convention for its kernel table."""
        return 4.0 * self.n_tokens ** 2 * self.head_dim * self.heads * self.batch

    @property
    def scale(self) -> float:
        return self.head_dim ** -0.5

    @property
    def coarse_grid(self) -> tuple:
        """(T', H', W') of the PSABlock layout (3D padding: ceil of each axis)."""
        bt, bh, bw = self.psablock
        return (-(-self.frames // bt), -(-self.height // bh), -(-self.width // bw))

    @property
    def n_blocked(self) -> int:
        """Positions of the PSABlock-centric layout."""
        tp, hp, wp = self.coarse_grid
        bt, bh, bw = self.psablock
        return tp * hp * wp * bt * bh * bw + self.n_text


SWEEP_TARGETS = (0.05, 0.10, 0.20, 0.30, 0.50, 0.70, 0.90, 1.00)

CONFIGS = {
    "tiny": Config("tiny", 1, 2, 64, 4, 16, 16, 0, 64, (24, 20, 20), None),
    "wan1_3b": Config("wan1_3b", 1, 12, 128, 21, 30, 52, 0, 128, (44, 42, 42), (0.15, 0.40)),
    "wan14b": Config("wan14b", 1, 40, 128, 21, 45, 80, 0, 128, (44, 42, 42), (0.10, 0.40)),
    "hunyuan": Config("hunyuan", 1, 24, 128, 33, 45, 80, 256, 128, (44, 42, 42), (0.10, 0.35)),
    "sweep": Config("sweep", 1, 40, 128, 21, 45, 80, 0, 128, (44, 42, 42), None),
    "wan14b_3d": Config("wan14b_3d", 1, 40, 128, 21, 45, 80, 0, 128, (44, 42, 42), (0.10, 0.40),
                        psablock=(3, 8, 16)),
}


def get_config(name: str) -> Config:
    return CONFIGS[name]
