"""Seeded synthetic token grids shaped like ViT encoder activations.

This module only draws inputs. It holds none of the merging arithmetic, so the
HIP path and the CPU oracle can both be fed from it without sharing any of the
method's code.

The paper measures on ADE20K (512x512 -> 32x32 patches), Cityscapes
(768x768 -> 48x48) and 1024x1024 inputs (64x64), with patch size 16 and ViT
widths 192/384/768/1024 (Sec. 3.1 Preliminaries, Sec. 4 tables). Neither the
datasets nor trained weights are available, so each image here is a token grid
whose structure imitates what a ViT block sees: piecewise-constant regions
(a Voronoi partition of the grid, one random centroid per region) plus Gaussian
noise, optionally a smooth spatial gradient, and a low-affinity i.i.d. case
with some images built from exact duplicated 2x2 patches.

Every image has an independent stream: ``numpy.random.default_rng([seed, cfg, b])``.
Values are drawn in float64, rounded to float32 (round-to-nearest-even) and,
for bfloat16 configs, to bfloat16 (round-to-nearest-even).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

__all__ = ["GridConfig", "CONFIGS", "config", "make_image", "make_batch", "to_storage"]


@dataclass(frozen=True)
class GridConfig:
    """One synthetic workload: B images of a G x G token grid with D channels."""

    index: int          # 1-based workload number used in the RNG stream key
    name: str
    B: int
    G: int              # grid side; N = G * G tokens per image
    D: int
    dtype: str          # "f32" or "bf16"
    kind: str           # "voronoi" or "iid_dup"
    regions: int = 0    # Voronoi regions per image
    sigma: float = 0.0  # per-token noise standard deviation
    gradient: float = 0.0  # weight of the linear spatial gradient term (0 = off)
    insertions: int = 2

    @property
    def N(self) -> int:
        return self.G * self.G


CONFIGS = {
    # ViT-Ti/16 at 512x512: one insertion.
    "vit_ti_512": GridConfig(1, "vit_ti_512", B=1, G=32, D=192, dtype="f32", kind="voronoi",
                             regions=12, sigma=0.3, insertions=1),
    # ViT-S/16 at 512x512: two insertions.
    "vit_s_512": GridConfig(2, "vit_s_512", B=32, G=32, D=384, dtype="bf16", kind="voronoi",
                            regions=20, sigma=0.25, insertions=2),
    # ViT-B/16 at 512x512: insertions before blocks 2 and 5.
    "vit_b_512": GridConfig(3, "vit_b_512", B=64, G=32, D=768, dtype="bf16", kind="voronoi",
                            regions=30, sigma=0.2, gradient=0.05, insertions=2),
    # ViT-L/16 at 1024x1024: second insertion runs on ragged packed survivors.
    "vit_l_1024": GridConfig(4, "vit_l_1024", B=16, G=64, D=1024, dtype="bf16", kind="voronoi",
                             regions=60, sigma=0.2, insertions=2),
    # 768x768 low-affinity stress case: i.i.d. tokens, every tenth image made of
    # exact duplicated 2x2 patches.
    "stress_768": GridConfig(5, "stress_768", B=32, G=48, D=768, dtype="bf16", kind="iid_dup",
                             insertions=2),
}


def config(name: str) -> GridConfig:
    return CONFIGS[name]


def _voronoi_image(rng: np.random.Generator, cfg: GridConfig) -> np.ndarray:
    G, D, R = cfg.G, cfg.D, cfg.regions
    seeds = rng.uniform(0.0, float(G), size=(R, 2))          # (row, col) of each region seed
    centroids = rng.standard_normal((R, D))
    noise = cfg.sigma * rng.standard_normal((G * G, D))
    grad = rng.standard_normal((2, D)) if cfg.gradient else None
    rows, cols = np.divmod(np.arange(G * G), G)
    centre = np.stack([rows + 0.5, cols + 0.5], axis=1)      # token centres on the grid
    d2 = ((centre[:, None, :] - seeds[None, :, :]) ** 2).sum(-1)
    label = np.argmin(d2, axis=1)                            # first (lowest) seed on ties
    x = centroids[label] + noise
    if grad is not None:
        x = x + cfg.gradient * (rows[:, None] * grad[0][None, :] + cols[:, None] * grad[1][None, :])
    return x


def _iid_dup_image(rng: np.random.Generator, cfg: GridConfig, b: int) -> np.ndarray:
    G, D = cfg.G, cfg.D
    if b % 10 == 5:
        base = rng.standard_normal((G // 2, G // 2, D))
        grid = np.repeat(np.repeat(base, 2, axis=0), 2, axis=1)  # exact 2x2 duplicates
        return grid.reshape(G * G, D)
    return rng.standard_normal((G * G, D))


def make_image(cfg: GridConfig, seed: int, b: int) -> np.ndarray:
    """float64 [N, D] tokens of image ``b`` (before storage rounding)."""
    rng = np.random.default_rng([seed, cfg.index, b])
    if cfg.kind == "voronoi":
        return _voronoi_image(rng, cfg)
    if cfg.kind == "iid_dup":
        return _iid_dup_image(rng, cfg, b)
    raise ValueError(f"unknown generator kind {cfg.kind!r}")


def to_storage(x64: np.ndarray, dtype: str):
    """Round float64 values to the storage dtype; returns a CPU torch tensor.

    float64 -> float32 and float32 -> bfloat16 both round to nearest even.
    """
    import torch

    x32 = torch.from_numpy(np.ascontiguousarray(x64, dtype=np.float64).astype(np.float32))
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return x32.to(torch.bfloat16)
    raise ValueError(f"unknown dtype {dtype!r}")


def make_batch(cfg: GridConfig, seed: int = 0, images=None):
    """CPU torch tensor [len(images), N, D] in the storage dtype.

    ``images`` selects image indices (default: all B); each image's values do
    not depend on which other images are drawn.
    """
    import torch

    idx = range(cfg.B) if images is None else list(images)
    out = [to_storage(make_image(cfg, seed, b), cfg.dtype) for b in idx]
    return torch.stack(out, 0)
