"""Seeded synthetic inputs shaped like one video-DiT attention layer.

This module only draws random numbers and rounds them to the storage dtype.
It contains none of PARK's arithmetic; the CPU oracle and the HIP library
both consume what it produces.

Recipe (per configuration and head ``h``):

* RNG: ``numpy.random.Generator(PCG64(SeedSequence([0, h])))``.  Draws happen
  in this fixed order: ``n_c`` Gaussian centres in R^d (entries N(0,1));
  ``n_c`` Voronoi sites in [0,1)^3; then the Q, K and V noise matrices
  ``[N_video, d]`` with entries N(0, 0.5^2) (float32 draws).
* Token (t, y, x) of a ``T_g x H_g x W_g`` latent grid, raster order
  t-major, belongs to the centre whose site is nearest to
  ``((t+1/2)/T_g, (y+1/2)/H_g, (x+1/2)/W_g)`` (ties -> lower centre id).
  Each of Q, K, V is ``2 * centre + noise`` (independent noise per tensor).
* Wan-shaped layer: one per-head scale ``s_h ~ U[0.5, 2]`` (drawn after the
  noise) multiplies Q, so heads differ in how peaked their attention is.
* HunyuanVideo-shaped layer: 256 text-like tokens are appended after the
  video tokens; their Q, K and V are N(0,1) (drawn last, Q then K then V).
* bf16 configurations are rounded to bfloat16 with round-to-nearest-even;
  the arrays returned here are float32 holding bf16-representable values.
* Re-use probe: step s >= 1 of a denoising run perturbs the previous
  step's Q and K by N(0, 0.05^2) drawn from ``SeedSequence([0, h, s])``
  (the second call of the sweep is step 1).

The paper measures on activations of Wan2.1-14B and HunyuanVideo generating
720p video from VBench prompts; those models and prompts are not available,
so these seeded tensors stand in for them with the same head counts, token
grids and head dimension.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np


@dataclass(frozen=True)
class LayerConfig:
    """One attention layer workload (all heads share the shape)."""

    name: str
    H: int
    grid: tuple  # (T_g, H_g, W_g) latent grid of the video tokens
    d: int
    dtype: str  # "f32" or "bf16"
    n_centres: int
    block: int = 64  # mean tokens per block; C = ceil(N / block) per side
    iters: int = 10  # k-means iterations
    select: str = "topk"  # "topk" or "topp"
    ratio: float = 0.25  # top-k fraction of key blocks
    topp: float = 0.9  # cumulative-mass threshold
    q_scale: tuple | None = None  # (lo, hi) of the per-head Q scale
    text_tokens: int = 0
    noise_sigma: float = 0.5
    seed: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def n_video(self) -> int:
        t, y, x = self.grid
        return t * y * x

    @property
    def N(self) -> int:
        return self.n_video + self.text_tokens

    @property
    def C(self) -> int:
        return -(-self.N // self.block)

    def with_(self, **kw) -> "LayerConfig":
        return replace(self, **kw)


CONFIGS = {
    # tiny case: 1 head, 4x32x32 grid, d=64, fp32, top-25%
    "tiny": LayerConfig("tiny", 1, (4, 32, 32), 64, "f32", 16, select="topk", ratio=0.25),
    # 8 heads, 8x32x64 grid, d=128, bf16, top-20%
    "medium": LayerConfig("medium", 8, (8, 32, 64), 128, "bf16", 64, select="topk", ratio=0.20),
    # Wan2.1-14B-shaped layer: 40 heads, 21x45x80 grid, top-p 0.9, per-head Q scale
    "wan": LayerConfig("wan", 40, (21, 45, 80), 128, "bf16", 128, select="topp", topp=0.9,
                       q_scale=(0.5, 2.0)),
    # HunyuanVideo-shaped layer: 24 heads, 33x45x80 grid + 256 text tokens, top-10%
    "hunyuan": LayerConfig("hunyuan", 24, (33, 45, 80), 128, "bf16", 128, select="topk",
                           ratio=0.10, text_tokens=256),
}
# the sweep runs on the Wan-shaped layer (same tensors as "wan")
CONFIGS["wan_sweep"] = CONFIGS["wan"].with_(name="wan_sweep")


def bf16_round(a: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _centre_of_tokens(sites: np.ndarray, grid: tuple) -> np.ndarray:
    """Index of the nearest site for every grid token (raster order, t-major).

    Squared distances are separable over the three grid axes."""
    axes = [((np.arange(n) + 0.5) / n)[:, None] - sites[None, :, i] for i, n in enumerate(grid)]
    dt, dy, dx = (a ** 2 for a in axes)
    d2 = dt[:, None, None, :] + dy[None, :, None, :] + dx[None, None, :, :]
    return np.argmin(d2.reshape(-1, sites.shape[0]), axis=1)  # ties -> lower id


def make_head(cfg: LayerConfig, h: int):
    """Q, K, V of head ``h`` as float32 arrays ``[N, d]``."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, h])))
    d = cfg.d
    centres = rng.standard_normal((cfg.n_centres, d))
    sites = rng.random((cfg.n_centres, 3))
    owner = _centre_of_tokens(sites, cfg.grid)
    base = (2.0 * centres).astype(np.float32)[owner]
    out = []
    for _ in range(3):
        noise = rng.standard_normal((cfg.n_video, d), dtype=np.float32)
        out.append(base + np.float32(cfg.noise_sigma) * noise)
    q, k, v = out
    if cfg.q_scale is not None:
        s = rng.uniform(cfg.q_scale[0], cfg.q_scale[1])
        q = q * np.float32(s)
    if cfg.text_tokens:
        txt = [rng.standard_normal((cfg.text_tokens, d), dtype=np.float32) for _ in range(3)]
        q, k, v = (np.concatenate([a, b]) for a, b in zip((q, k, v), txt))
    if cfg.dtype == "bf16":
        q, k, v = bf16_round(q), bf16_round(k), bf16_round(v)
    return q, k, v


def make_layer(cfg: LayerConfig, heads=None, workers: int = 8):
    """Stacked ``[H', N, d]`` float32 Q, K, V for ``heads`` (default: all)."""
    from concurrent.futures import ThreadPoolExecutor

    heads = list(range(cfg.H) if heads is None else heads)
    out = [np.empty((len(heads), cfg.N, cfg.d), dtype=np.float32) for _ in range(3)]

    def one(i):
        for dst, src in zip(out, make_head(cfg, heads[i])):
            dst[i] = src

    with ThreadPoolExecutor(max_workers=max(1, min(workers, len(heads)))) as ex:
        list(ex.map(one, range(len(heads))))
    return tuple(out)


def perturb_head(cfg: LayerConfig, h: int, q: np.ndarray, k: np.ndarray, sigma: float = 0.05,
                 step: int = 1):
    """Re-use probe: Q and K of diffusion step ``step`` (>= 1), the previous
    step's drifted by N(0, sigma^2) from ``SeedSequence([seed, h, step])``."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, h, step])))
    q2 = q + np.float32(sigma) * rng.standard_normal(q.shape, dtype=np.float32)
    k2 = k + np.float32(sigma) * rng.standard_normal(k.shape, dtype=np.float32)
    if cfg.dtype == "bf16":
        q2, k2 = bf16_round(q2), bf16_round(k2)
    return q2.astype(np.float32), k2.astype(np.float32)


def perturb_layer(cfg: LayerConfig, q: np.ndarray, k: np.ndarray, heads=None, workers: int = 8):
    """perturb_head over the stacked ``[H', N, d]`` Q and K (threads over heads)."""
    from concurrent.futures import ThreadPoolExecutor

    heads = list(range(q.shape[0]) if heads is None else heads)
    q2, k2 = np.empty_like(q), np.empty_like(k)

    def one(i):
        q2[i], k2[i] = perturb_head(cfg, heads[i], q[i], k[i])

    with ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(one, range(len(heads))))
    return q2, k2

