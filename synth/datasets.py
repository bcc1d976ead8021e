"""Seeded synthetic datasets (stand-ins for the paper's MNIST and CelebA).

All generators use numpy's PCG64 from the recipe's seed and return a C-contiguous
float32 array of shape [n, x_dim] (images flattened row-major, NHWC for colour).
"""
import numpy as np


def ring8(n, seed=0, radius=2.0, sigma=0.02):
    """2-D mixture of 8 Gaussians on a circle of the given radius."""
    rng = np.random.default_rng(seed)
    k = rng.integers(0, 8, size=n)
    ang = 2.0 * np.pi * k / 8.0
    centres = np.stack([radius * np.cos(ang), radius * np.sin(ang)], axis=1)
    x = centres + sigma * rng.standard_normal((n, 2))
    return np.ascontiguousarray(x, dtype=np.float32)


def _blob_prototypes(rng, n_proto=10, h=28, w=28):
    yy, xx = np.mgrid[0:h, 0:w].astype(np.float64)
    protos = np.empty((n_proto, h, w))
    for p in range(n_proto):
        img = np.zeros((h, w))
        for _ in range(rng.integers(3, 7)):
            cy, cx = rng.uniform(5, h - 5), rng.uniform(5, w - 5)
            sy, sx = rng.uniform(1.5, 4.5), rng.uniform(1.5, 4.5)
            amp = rng.uniform(0.5, 1.0)
            img += amp * np.exp(-0.5 * (((yy - cy) / sy) ** 2 + ((xx - cx) / sx) ** 2))
        img = (img - img.min()) / (img.max() - img.min())
        protos[p] = 2.0 * img - 1.0
    return protos.reshape(n_proto, h * w)


def mnist_like(n, seed=0, noise=0.1, chunk=8192):
    """784-dim vectors in [-1, 1]: one of 10 seeded blob prototypes plus N(0, noise^2)."""
    rng = np.random.default_rng(seed)
    protos = _blob_prototypes(rng)
    labels = rng.integers(0, 10, size=n)
    out = np.empty((n, 784), dtype=np.float32)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = protos[labels[s:e]] + noise * rng.standard_normal((e - s, 784))
        out[s:e] = np.clip(x, -1.0, 1.0)
    return out


def celeba_like(n, seed=0, h=64, w=64, c=3, chunk=1024):
    """64x64x3 NHWC images in [-1, 1]: smooth random colour fields plus 1-4 blobs, tanh-squashed."""
    rng = np.random.default_rng(seed)
    yy, xx = np.mgrid[0:h, 0:w].astype(np.float32) / np.float32(h)
    out = np.empty((n, h * w * c), dtype=np.float32)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        m = e - s
        img = np.zeros((m, h, w, c), dtype=np.float32)
        for _ in range(3):
            fy = rng.uniform(0.5, 3.0, size=(m, 1, 1, c)).astype(np.float32)
            fx = rng.uniform(0.5, 3.0, size=(m, 1, 1, c)).astype(np.float32)
            ph = rng.uniform(0, 2 * np.pi, size=(m, 1, 1, c)).astype(np.float32)
            a = rng.uniform(0.2, 0.6, size=(m, 1, 1, c)).astype(np.float32)
            img += a * np.cos(2 * np.pi * (fy * yy[None, :, :, None] + fx * xx[None, :, :, None]) + ph)
        nb = rng.integers(1, 5, size=m)
        for b in range(4):
            on = (nb > b).astype(np.float32)[:, None, None, None]
            cy = rng.uniform(0.2, 0.8, size=(m, 1, 1, 1)).astype(np.float32)
            cx = rng.uniform(0.2, 0.8, size=(m, 1, 1, 1)).astype(np.float32)
            sg = rng.uniform(0.05, 0.2, size=(m, 1, 1, 1)).astype(np.float32)
            col = rng.uniform(-1.0, 1.0, size=(m, 1, 1, c)).astype(np.float32)
            g = np.exp(-0.5 * ((yy[None, :, :, None] - cy) ** 2 + (xx[None, :, :, None] - cx) ** 2) / sg ** 2)
            img += on * 1.5 * col * g
        out[s:e] = np.tanh(img).reshape(m, -1)
    return out


def make_dataset(recipe):
    """Build the dataset described by a workload's ``data`` dict."""
    kind = recipe["kind"]
    n = int(recipe["n"])
    seed = int(recipe.get("seed", 0))
    if kind == "ring8":
        return ring8(n, seed)
    if kind == "mnist_like":
        return mnist_like(n, seed)
    if kind == "celeba_like":
        return celeba_like(n, seed, h=int(recipe.get("h", 64)), w=int(recipe.get("w", 64)),
                           c=int(recipe.get("c", 3)))
    raise ValueError(f"unknown dataset kind {kind!r}")
