"""Shapes of the synthetic workloads.

The five configurations stand in for the paper's 480x832 / 81-frame
Wan2.1 text-to-video workloads (Sec. 5.1 "Model Architecture"): the latent
grid 21x30x52 is the 480x832, 81-frame video after the 4x temporal,
8x spatial VAE compression and the 1x2x2 patchify; 21x45x80 is the 720p
counterpart.  No dataset, prompt or checkpoint is used.

Patch features Cp = 16 latent channels x 1x2x2 patch = 64 for every config.
"""
from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class Config:
    name: str
    dim: int                 # model width D
    n_heads: int             # attention heads H
    head_dim: int            # per-head width dh (D == H * dh)
    ffn_dim: int             # FFN hidden width F
    n_layers: int            # transformer blocks N
    grid: Tuple[int, int, int]  # latent token grid (frames, rows, cols)
    text_len: int            # text tokens Lc
    dtype: str               # "f32" or "bf16": storage / MFMA input type
    patch_dim: int = 64      # Cp
    freq_dim: int = 256      # sinusoidal timestep features
    batch: int = 1
    eps: float = 1e-6
    rope_theta: float = 10000.0
    timesteps: Tuple[int, ...] = (999, 750, 500, 250)
    # per-step kept counts (None: recipe-driven, see synth.make_masks)
    keep_heads: Tuple[int, ...] = field(default=None)
    keep_ffn: Tuple[int, ...] = field(default=None)
    ffn_chunk: int = 8       # FFN gate granularity C (App. A, "FFN Reordering and Chunking")
    std: float = 0.02

    @property
    def seq_len(self) -> int:
        f, h, w = self.grid
        return f * h * w

    def with_(self, **kw) -> "Config":
        return replace(self, **kw)


CONFIGS = {
    # C1: tiny fp32 two-layer stack, full 4-step denoise
    "tiny": Config(
        name="tiny", dim=256, n_heads=4, head_dim=64, ffn_dim=1024, n_layers=2,
        grid=(2, 8, 8), text_len=16, dtype="f32",
        keep_heads=(4, 3, 3, 2), keep_ffn=(1024, 768, 640, 512)),
    # C2: Wan-1.3B-shaped single block
    "wan1.3b_block": Config(
        name="wan1.3b_block", dim=1536, n_heads=12, head_dim=128, ffn_dim=8960,
        n_layers=1, grid=(21, 30, 52), text_len=512, dtype="bf16",
        keep_heads=(9,), keep_ffn=(6720,)),
    # C3: Wan-14B-shaped single block, four step structures
    "wan14b_block": Config(
        name="wan14b_block", dim=5120, n_heads=40, head_dim=128, ffn_dim=13824,
        n_layers=1, grid=(21, 30, 52), text_len=512, dtype="bf16",
        keep_heads=(40, 32, 28, 24), keep_ffn=(13824, 11059, 9677, 8294), ffn_chunk=1),
    # C4: Wan-14B-shaped 40-layer stack, 4-step 480p denoise
    "wan14b_480p": Config(
        name="wan14b_480p", dim=5120, n_heads=40, head_dim=128, ffn_dim=13824,
        n_layers=40, grid=(21, 30, 52), text_len=512, dtype="bf16"),
    # C5: Wan-14B-shaped 40-layer stack at 720p
    "wan14b_720p": Config(
        name="wan14b_720p", dim=5120, n_heads=40, head_dim=128, ffn_dim=13824,
        n_layers=40, grid=(21, 45, 80), text_len=512, dtype="bf16"),
}


def get_config(name: str) -> Config:
    return CONFIGS[name]
