"""Seeded synthetic camera frames.

The paper evaluates on R2R-CE episodes rendered by the VLN-CE simulator, which
is not available here.  These generators stand in for it with camera-like RGB
frames in [0, 1] that show the effects the paper analyses in Sec. 3: viewpoint
translation and rotation, hard edges, smooth regions, brightness change and
sensor noise.  All arrays are float32, NCHW, and fully determined by the seed.

Frame model (one canvas):
  * 32 Gaussian blobs: centre uniform on the canvas, sigma ~ U[P/2, 4P] px,
    RGB amplitude ~ U[0,1]^3; the blob sum is divided by its maximum;
  * 8 axis-aligned hard-edged rectangles painted over it, sides ~ U[P, 6P] px,
    RGB ~ U[0,1]^3;
  * (episode textures only) thin bars standing in for door frames and
    obstacle outlines;
  * noise, where a configuration asks for it, is added last and the frame is
    clipped to [0, 1].
"""
from __future__ import annotations

import numpy as np

PATCH = 14

# Configuration constants (sizes follow the workloads the paper's model sees:
# Qwen2.5-VL's 14-px patches, 2x2 token merge, 448/896-px camera frames).
TINY = dict(size=224, patch=PATCH, merge=1, margin=8, max_shift=8, noise=0.01,
            alpha_fixed=0.5)
SEL = dict(batch=64, size=448, patch=PATCH, merge=1, margin=64, max_shift=20,
           max_rot_deg=5.0, bright=(0.9, 1.1), noise=0.02)
EPISODE = dict(size=448, texture=2048, patch=PATCH, merge=2, steps=32, warmup=7,
               max_step=24, shear=0.05, window=8, text=128)
BATCH = dict(size=896, texture=2048, patch=PATCH, merge=2, steps=32, warmup=3,
             episodes=16, max_step=24, shear=0.05, window=4, text=128)


def canvas(rng: np.random.Generator, h: int, w: int, patch: int = PATCH,
           n_blobs: int = 32, n_rects: int = 8, n_bars: int = 0) -> np.ndarray:
    """Return a float64 [3, h, w] canvas in [0, 1] (blobs, rectangles, bars)."""
    img = np.zeros((3, h, w), dtype=np.float64)
    for _ in range(n_blobs):
        cy, cx = rng.uniform(0, h), rng.uniform(0, w)
        sig = rng.uniform(patch / 2, 4 * patch)
        amp = rng.uniform(0, 1, size=3)
        r = int(np.ceil(4 * sig))
        y0, y1 = max(0, int(cy) - r), min(h, int(cy) + r + 1)
        x0, x1 = max(0, int(cx) - r), min(w, int(cx) + r + 1)
        if y0 >= y1 or x0 >= x1:
            continue
        yy = np.arange(y0, y1) - cy
        xx = np.arange(x0, x1) - cx
        # the isotropic Gaussian is separable: exp(-(y^2 + x^2) / 2s^2) = gy(y) gx(x)
        gy = np.exp(-(yy * yy) / (2 * sig * sig))
        gx = np.exp(-(xx * xx) / (2 * sig * sig))
        for c in range(3):
            img[c, y0:y1, x0:x1] += np.outer(amp[c] * gy, gx)
    mx = img.max()
    if mx > 0:
        img /= mx
    for _ in range(n_rects):
        rh = int(rng.integers(patch, 6 * patch + 1))
        rw = int(rng.integers(patch, 6 * patch + 1))
        y0 = int(rng.integers(-rh // 2, h - rh // 2))
        x0 = int(rng.integers(-rw // 2, w - rw // 2))
        col = rng.uniform(0, 1, size=3)
        img[:, max(0, y0):max(0, min(h, y0 + rh)), max(0, x0):max(0, min(w, x0 + rw))] = \
            col[:, None, None]
    for _ in range(n_bars):
        thick = int(rng.integers(2, 5))
        length = int(rng.integers(4 * patch, 16 * patch + 1))
        col = rng.uniform(0, 1, size=3)
        y0 = int(rng.integers(0, h))
        x0 = int(rng.integers(0, w))
        if rng.uniform() < 0.5:
            img[:, y0:min(h, y0 + thick), x0:min(w, x0 + length)] = col[:, None, None]
        else:
            img[:, y0:min(h, y0 + length), x0:min(w, x0 + thick)] = col[:, None, None]
    return img


def _bilinear(img: np.ndarray, ys: np.ndarray, xs: np.ndarray) -> np.ndarray:
    """Sample a [3, H, W] image at real coordinates (ys, xs) (same shape), edge-clamped."""
    h, w = img.shape[1:]
    ys = np.clip(ys, 0, h - 1)
    xs = np.clip(xs, 0, w - 1)
    y0 = np.minimum(np.floor(ys).astype(np.int64), h - 2)
    x0 = np.minimum(np.floor(xs).astype(np.int64), w - 2)
    fy = ys - y0
    fx = xs - x0
    a = img[:, y0, x0]
    b = img[:, y0, x0 + 1]
    c = img[:, y0 + 1, x0]
    d = img[:, y0 + 1, x0 + 1]
    return (a * (1 - fy) * (1 - fx) + b * (1 - fy) * fx + c * fy * (1 - fx) + d * fy * fx)


def tiny_pair(seed: int = 0):
    """One 224x224 pair: frame1 = frame0 translated by an integer (dy, dx) in [-8, 8]
    (new content enters at the border) plus N(0, 0.01) noise.

    Returns (prev [1,3,224,224] f32, cur [1,3,224,224] f32, (dy, dx)); content at
    prev (y, x) appears in cur at (y + dy, x + dx).
    """
    rng = np.random.default_rng(seed)
    s, m = TINY["size"], TINY["margin"]
    cv = canvas(rng, s + 2 * m, s + 2 * m)
    dy, dx = (int(v) for v in rng.integers(-TINY["max_shift"], TINY["max_shift"] + 1, 2))
    f0 = cv[:, m:m + s, m:m + s]
    f1 = cv[:, m - dy:m - dy + s, m - dx:m - dx + s] + rng.normal(0, TINY["noise"], (3, s, s))
    f1 = np.clip(f1, 0.0, 1.0)
    return f0.astype(np.float32)[None], f1.astype(np.float32)[None], (dy, dx)


def sel_pairs(seed: int = 1, batch: int = SEL["batch"], size: int = SEL["size"]):
    """`batch` independent pairs at size x size: frame1 = frame0 translated by an
    integer (dy, dx) in [-20, 20], rotated by U[0, 5] degrees about the frame
    centre (bilinear), scaled in brightness by U[0.9, 1.1], plus N(0, 0.02) noise.

    Returns (prev [B,3,S,S] f32, cur [B,3,S,S] f32, list of (dy, dx, deg, gain)).
    """
    rng = np.random.default_rng(seed)
    m = SEL["margin"]
    prev = np.empty((batch, 3, size, size), np.float32)
    cur = np.empty((batch, 3, size, size), np.float32)
    meta = []
    yy, xx = np.meshgrid(np.arange(size, dtype=np.float64), np.arange(size, dtype=np.float64),
                         indexing="ij")
    c = (size - 1) / 2.0
    for b in range(batch):
        cv = canvas(rng, size + 2 * m, size + 2 * m)
        dy, dx = (int(v) for v in rng.integers(-SEL["max_shift"], SEL["max_shift"] + 1, 2))
        deg = float(rng.uniform(0.0, SEL["max_rot_deg"]))
        gain = float(rng.uniform(*SEL["bright"]))
        th = np.deg2rad(deg)
        # cur(q) = canvas(R(-th) (q - c - d) + c + margin): content rotated then shifted.
        qy, qx = yy - c - dy, xx - c - dx
        sy = np.cos(th) * qy + np.sin(th) * qx + c + m
        sx = -np.sin(th) * qy + np.cos(th) * qx + c + m
        f1 = _bilinear(cv, sy, sx) * gain + rng.normal(0, SEL["noise"], (3, size, size))
        prev[b] = cv[:, m:m + size, m:m + size]
        cur[b] = np.clip(f1, 0.0, 1.0)
        meta.append((dy, dx, deg, gain))
    return prev, cur, meta


def episode_frames(seed: int, size: int = EPISODE["size"], n_frames: int | None = None,
                   texture: int = EPISODE["texture"], max_step: int = EPISODE["max_step"],
                   shear: float = EPISODE["shear"]) -> np.ndarray:
    """A seeded camera trajectory over one synthetic texture.

    The camera does a random walk (integer translation in [-max_step, max_step]
    px per axis per step) plus a fresh yaw-like horizontal shear
    x' = x + s (y - y_c), s ~ U[-shear, shear], per frame.  Returns
    [n_frames, 3, size, size] float32 (default n_frames = warmup + steps).
    """
    if n_frames is None:
        n_frames = EPISODE["warmup"] + EPISODE["steps"]
    rng = np.random.default_rng(seed)
    area = (texture / 576.0) ** 2
    tex = canvas(rng, texture, texture, n_blobs=int(32 * area), n_rects=int(8 * area),
                 n_bars=int(4 * area))
    pad = int(np.ceil(shear * size / 2)) + 2
    lo, hi = pad, texture - size - pad
    pos = np.array([(lo + hi) // 2, (lo + hi) // 2], dtype=np.int64)
    yy, xx = np.meshgrid(np.arange(size, dtype=np.float64), np.arange(size, dtype=np.float64),
                         indexing="ij")
    out = np.empty((n_frames, 3, size, size), np.float32)
    for k in range(n_frames):
        if k > 0:
            pos = np.clip(pos + rng.integers(-max_step, max_step + 1, 2), lo, hi)
        s = rng.uniform(-shear, shear)
        ys = yy + pos[0]
        xs = xx + pos[1] + s * (yy - (size - 1) / 2.0)
        out[k] = _bilinear(tex, ys, xs)
    return np.clip(out, 0.0, 1.0)
