"""Seeded synthetic inputs and the named workloads (sizes only).

This module is shared by the tests, the benchmark and the oracle checks.  It
holds no arithmetic of the method: it only draws random tensors from a seed
and records the shapes of the workloads.

Inputs stand in for Flux.1-dev activations, which are not available: Q, K, V
are drawn N(0, 1) in float32 from ``torch.Generator('cpu').manual_seed(seed)``
in the order Q, K, V with shape [B, H, N_tot, D], then rounded to bfloat16
(round-to-nearest-even, torch's cast) when the workload is bf16.  Hidden
states for the token gather are N(0, 1) of shape [B, N_img, C].
"""

from dataclasses import dataclass, field

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    grid: int             # latent grid side (grid x grid image tokens)
    n_txt: int            # text tokens, placed before the image tokens
    batch: int
    heads: int
    head_dim: int
    dtype: str            # "f32" or "bf16"
    tile: int             # tokens per tile, N_T
    delta: int            # per-layer slide of the tile boundaries
    shared: int           # side of the central shared region
    layers: tuple = (0,)
    hidden: int = 3072    # hidden size of the token gather workload
    seed: int = 0
    moved: bool = False   # shared tokens gathered next to the text (Appendix A)
    grid_w: int = 0       # grid columns when the grid is not square (0: square)

    @property
    def cols(self):
        return self.grid_w or self.grid

    @property
    def n_img(self):
        """Image tokens of the grid (grid x cols cells)."""
        return self.grid * self.cols

    @property
    def n_tot(self):
        """Text plus image tokens.  A grid that is not a square power of two
        runs attention over a longer, padded sequence (see image_span in the
        binding)."""
        return self.n_txt + self.n_img


WORKLOADS = {
    # 16x16 grid, no text, fp32: small enough for the loop oracle
    "tiny-16": Workload("tiny-16", 16, 0, 1, 2, 64, "f32", 64, 32, 4,
                        layers=(0, 1, 2, 3), hidden=64),
    # Flux.1-dev at 1024x1024: 64x64 latent grid plus 512 text tokens
    "flux-64": Workload("flux-64", 64, 512, 1, 24, 128, "bf16", 256, 128, 8),
    # the same tensors swept over the 57 transformer blocks of Flux.1-dev
    "flux-64-sweep": Workload("flux-64-sweep", 64, 512, 1, 24, 128, "bf16", 256, 128, 8,
                              layers=tuple(range(57))),
    # Flux.1-dev at 2048x2048: 128x128 latent grid plus 512 text tokens
    "flux-128": Workload("flux-128", 128, 512, 1, 24, 128, "bf16", 1024, 512, 16),
    # 4096x4096 stress shape: 256x256 latent grid plus 512 text tokens
    "stress-256": Workload("stress-256", 256, 512, 1, 24, 128, "bf16", 2048, 1024, 32),
    # the settings of the paper's Table 1: G = 4 or 16 tiles (N_T = N_img/G),
    # a slide cycle of 4 (Delta = N_T/4), a 16x16 shared region at 1024x1024
    # and 32x32 at 2048x2048
    "table1-64-g4": Workload("table1-64-g4", 64, 512, 1, 24, 128, "bf16", 1024, 256, 16),
    "table1-64-g16": Workload("table1-64-g16", 64, 512, 1, 24, 128, "bf16", 256, 64, 16),
    "table1-128-g4": Workload("table1-128-g4", 128, 512, 1, 24, 128, "bf16", 4096, 1024, 32),
    "table1-128-g16": Workload("table1-128-g16", 128, 512, 1, 24, 128, "bf16", 1024, 256, 32),
    # the same settings in the moved-prefix layout of Appendix A: the shared
    # tokens follow the text and the other N_img - N_sh tokens form G tiles
    # general shapes (Appendix D): Flux.1-dev at 1536x1536 (96x96 latent) and
    # at 1024x1536 portrait (64 rows x 96 columns), both in the 128x128
    # enclosing curve
    "flux-96": Workload("flux-96", 96, 512, 1, 24, 128, "bf16", 1024, 512, 16),
    "flux-64x96": Workload("flux-64x96", 64, 512, 1, 24, 128, "bf16", 1024, 512, 16, grid_w=96),
    "moved-64-g4": Workload("moved-64-g4", 64, 512, 1, 24, 128, "bf16", 960, 240, 16, moved=True),
    "moved-64-g16": Workload("moved-64-g16", 64, 512, 1, 24, 128, "bf16", 240, 60, 16, moved=True),
    "moved-128-g4": Workload("moved-128-g4", 128, 512, 1, 24, 128, "bf16", 3840, 960, 32, moved=True),
    "moved-128-g16": Workload("moved-128-g16", 128, 512, 1, 24, 128, "bf16", 960, 240, 32, moved=True),
}


def torch_dtype(name):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def qkv(batch, heads, n, head_dim, dtype="bf16", seed=0):
    """Q, K, V as CPU tensors [B, H, N, D] of the requested dtype."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (batch, heads, n, head_dim)
    out = []
    for _ in range(3):
        t = torch.randn(shape, generator=g, dtype=torch.float32)
        out.append(t.to(torch_dtype(dtype)))
    return tuple(out)


def hidden_states(batch, n, channels, dtype="bf16", seed=1):
    """Hidden states [B, N, C] for the token gather / scatter."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    t = torch.randn((batch, n, channels), generator=g, dtype=torch.float32)
    return t.to(torch_dtype(dtype))
