"""Seeded synthetic ConvCRF workloads.

Stands in for the PASCAL VOC frames and noisy unaries of the paper's synthetic
denoising experiment (Sec. 5.1), which are not available here.  Each image is
a Voronoi partition into piecewise-constant coloured regions; each region gets
a true class label, a fixed fraction of regions get a wrong label, and the
unary logits are a scaled one-hot of the (possibly wrong) label plus Gaussian
noise.

This module draws random numbers only.  It contains none of the method's
arithmetic, so both the HIP library's callers and the CPU oracle's callers can
take their inputs from it.  Arrays are float32, C-contiguous:
unary [B,C,H,W] (logits, i.e. minus the unary energy), image [B,3,H,W]
(integer-valued RGB in 0..255), labels [B,H,W] int64 (ground truth).
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

try:  # nearest-seed assignment; a chunked brute force is used without scipy
    from scipy.spatial import cKDTree as _KDTree
except Exception:  # pragma: no cover
    _KDTree = None


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, window, blur, iterations, generator."""
    name: str
    B: int
    C: int
    H: int
    W: int
    filter_size: int
    blur: int = 1
    iters: int = 5
    regions: int = 40
    wrong_frac: float = 0.2
    onehot_scale: float = 2.0
    logit_noise: float = 1.0
    pixel_noise: float = 8.0
    # Eq. 4 parameters: appearance w=10, theta_alpha=80, theta_beta=13;
    # smoothness w=3, theta_gamma=3 (the DenseCRF defaults the paper adopts
    # in Sec. 5.1), held fixed for every window size.
    w_app: float = 10.0
    theta_alpha: float = 80.0
    theta_beta: float = 13.0
    w_smooth: float = 3.0
    theta_gamma: float = 3.0
    seed_base: int = 0

    @property
    def pixels(self) -> int:
        return self.B * self.H * self.W

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads: a tiny smoke case, a PASCAL-sized frame, the pooled
# ("blur") variant with a wider window, a batch of 8 frames, and a
# street-scene-sized frame with 19 classes.
WORKLOADS = {
    "tiny": Workload("tiny", 1, 21, 64, 64, 5, regions=12, seed_base=1000),
    "pascal": Workload("pascal", 1, 21, 512, 512, 7, regions=40, seed_base=2000),
    "blur": Workload("blur", 1, 21, 512, 512, 11, blur=4, regions=40, seed_base=3000),
    "batched": Workload("batched", 8, 21, 512, 512, 7, regions=40, seed_base=4000),
    "street": Workload("street", 1, 19, 1024, 2048, 7, regions=300, seed_base=5000),
}


def _nearest_seed(H: int, W: int, seeds: np.ndarray) -> np.ndarray:
    """Index of the nearest seed (Euclidean) for every pixel centre."""
    ys, xs = np.meshgrid(np.arange(H) + 0.5, np.arange(W) + 0.5, indexing="ij")
    pts = np.stack([ys.ravel(), xs.ravel()], axis=1)
    if _KDTree is not None:
        _, idx = _KDTree(seeds).query(pts, k=1)
        return idx.reshape(H, W).astype(np.int64)
    out = np.empty(pts.shape[0], dtype=np.int64)
    step = 65536
    for a in range(0, pts.shape[0], step):
        d = ((pts[a:a + step, None, :] - seeds[None, :, :]) ** 2).sum(-1)
        out[a:a + step] = d.argmin(1)
    return out.reshape(H, W)


def voronoi_frame(wl: Workload, rng: np.random.Generator):
    """One image, its unary logits and its ground-truth labels."""
    H, W, R, C = wl.H, wl.W, wl.regions, wl.C
    seeds = rng.uniform(0.0, 1.0, size=(R, 2)) * np.array([H, W], dtype=np.float64)
    region = _nearest_seed(H, W, seeds)
    colours = rng.uniform(0.0, 255.0, size=(R, 3))
    img = colours[region].transpose(2, 0, 1) + rng.normal(0.0, wl.pixel_noise, size=(3, H, W))
    img = np.clip(np.rint(img), 0.0, 255.0).astype(np.float32)

    true_lab = rng.integers(0, C, size=R)
    noisy_lab = true_lab.copy()
    n_wrong = int(round(wl.wrong_frac * R))
    if C > 1 and n_wrong > 0:
        wrong = rng.choice(R, size=n_wrong, replace=False)
        noisy_lab[wrong] = (true_lab[wrong] + rng.integers(1, C, size=n_wrong)) % C
    unary = rng.normal(0.0, wl.logit_noise, size=(C, H, W)).astype(np.float32)
    yy, xx = np.indices((H, W))
    unary[noisy_lab[region], yy, xx] += np.float32(wl.onehot_scale)
    return unary, img, true_lab[region].astype(np.int64)


def make_inputs(wl: Workload, seed: int | None = None):
    """Generate (unary [B,C,H,W], image [B,3,H,W], labels [B,H,W]); batch item
    b uses numpy PCG64 seeded with ``seed_base + b`` unless ``seed`` is given."""
    base = wl.seed_base if seed is None else int(seed)
    U = np.empty((wl.B, wl.C, wl.H, wl.W), dtype=np.float32)
    I = np.empty((wl.B, 3, wl.H, wl.W), dtype=np.float32)
    L = np.empty((wl.B, wl.H, wl.W), dtype=np.int64)
    for b in range(wl.B):
        U[b], I[b], L[b] = voronoi_frame(wl, np.random.default_rng(base + b))
    return U, I, L


def random_compat(C: int, seed: int, symmetric: bool = False) -> np.ndarray:
    """A random C x C compatibility matrix (for the learnable 1x1-convolution
    compatibility of Sec. 4.2); float32, row-major mu[l][l']."""
    rng = np.random.default_rng(seed)
    mu = rng.uniform(-0.5, 1.5, size=(C, C))
    if symmetric:
        mu = 0.5 * (mu + mu.T)
    return mu.astype(np.float32)
