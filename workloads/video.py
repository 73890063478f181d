"""Seeded synthetic video chunks with temporally continuous content.

Every generator returns a list of NHWC float32 frames whose values are
exactly representable in the requested storage dtype.  Frame 0 is the
chunk's reference frame; each later frame copies its predecessor and
re-draws a structured subset of pixels, so consecutive frames differ on a
controlled fraction of spatial sites (all channels of a changed site are
re-drawn).  These stand in for the paper's video datasets (UCF101, MOT16),
which are not available here; no item of those datasets is reproduced.
"""

from typing import List

import numpy as np
import torch
import torch.nn.functional as F

from .nets import to_storage


def toy_video(seed: int = 0, n_frames: int = 4, N: int = 1, H: int = 64,
              W: int = 64, C: int = 16, frac: float = 0.10, patch: int = 8,
              dtype: str = "f32") -> List[np.ndarray]:
    """Reference frame ~ U[0,1); every later frame copies the previous one
    and re-draws all channels of ``patch`` x ``patch`` squares at uniform
    positions until the union of squares covers at least ``frac`` of the
    sites of each image."""
    rng = np.random.default_rng(seed)
    f0 = rng.random((N, H, W, C), dtype=np.float32)
    frames = [to_storage(f0, dtype)]
    for _ in range(1, n_frames):
        f = frames[-1].copy()
        for n in range(N):
            cover = np.zeros((H, W), bool)
            while cover.sum() < frac * H * W:
                y = int(rng.integers(0, H - patch + 1))
                x = int(rng.integers(0, W - patch + 1))
                cover[y:y + patch, x:x + patch] = True
            vals = rng.random((int(cover.sum()), C), dtype=np.float32)
            f[n][cover] = vals
        frames.append(to_storage(f, dtype))
    return frames


def textline_video(seed: int = 0, n_frames: int = 16, N: int = 1,
                   H: int = 32, W: int = 128, band: int = 7,
                   dtype: str = "f32") -> List[np.ndarray]:
    """Grayscale text-line frames: background 0.85 with dark strokes (0.1)
    set with probability 0.3 inside glyph cells of the text rows.  Each
    later frame re-renders a ``band``-column stripe (about 5.5% of the
    columns at W=128) whose start advances by ``band`` columns per frame,
    as text scrolling through a fixed window would."""
    rng = np.random.default_rng(seed)

    def render(h, w):
        img = np.full((h, w), 0.85, np.float32)
        top, bot = h // 6, h - h // 6
        strokes = rng.random((bot - top, w)) < 0.3
        img[top:bot][strokes] = 0.1
        # blank gaps between glyph cells
        for x in range(0, w, 6):
            img[top:bot, x] = 0.85
        return img

    f0 = np.stack([render(H, W) for _ in range(N)])[..., None]
    frames = [to_storage(f0, dtype)]
    start = 0
    for _ in range(1, n_frames):
        f = frames[-1].copy()
        cols = [(start + j) % W for j in range(band)]
        for n in range(N):
            stripe = render(H, band)
            # make sure every site of the stripe really changes
            old = f[n, :, cols, 0].T
            same = np.isclose(stripe, old)
            stripe[same] = np.where(stripe[same] > 0.5, 0.1, 0.85)
            f[n, :, cols, 0] = stripe.T
        start = (start + band) % W
        frames.append(to_storage(f, dtype))
    return frames


def _smooth_noise(rng, N, H, W, C, octaves=4):
    out = torch.zeros((N, C, H, W))
    amp = 1.0
    for o in range(octaves):
        gh, gw = max(2, H // (64 >> o)), max(2, W // (64 >> o))
        g = torch.from_numpy(rng.random((N, C, gh, gw), dtype=np.float32))
        out += amp * F.interpolate(g, size=(H, W), mode="bilinear",
                                   align_corners=False)
        amp *= 0.5
    out /= (2.0 - 2.0 ** (1 - octaves))
    return out.permute(0, 2, 3, 1).numpy()


def driving_video(seed: int = 0, n_frames: int = 10, N: int = 1,
                  H: int = 1024, W: int = 2048, C: int = 3,
                  density: float = 0.10, side=(32, 256),
                  dtype: str = "bf16") -> List[np.ndarray]:
    """Driving-like frames: multi-octave smooth noise plus a vertical
    brightness gradient.  Each later frame copies the previous one and
    re-draws the union of random rectangles (sides uniform in ``side``)
    until the union covers at least ``density`` of the sites; re-drawn
    sites get fresh smooth content plus per-site noise, so every channel
    changes.  Changes are spatially clustered, as moving objects are."""
    rng = np.random.default_rng(seed)
    grad = np.linspace(0.2, -0.2, H, dtype=np.float32)[None, :, None, None]
    f0 = np.clip(_smooth_noise(rng, N, H, W, C) + grad, 0.0, 1.0)
    frames = [to_storage(f0, dtype)]
    lo, hi = side
    lo, hi = min(lo, H, W), min(hi, H, W)
    for _ in range(1, n_frames):
        f = frames[-1].copy()
        for n in range(N):
            cover = np.zeros((H, W), bool)
            target = density * H * W
            while cover.sum() < target:
                h = int(rng.integers(lo, hi + 1))
                w = int(rng.integers(lo, hi + 1))
                y = int(rng.integers(0, H - h + 1))
                x = int(rng.integers(0, W - w + 1))
                cover[y:y + h, x:x + w] = True
            k = int(cover.sum())
            new = (0.5 * rng.random((k, C), dtype=np.float32)
                   + 0.5 * f[n][cover])
            new = to_storage(np.clip(new, 0.0, 1.0), dtype)
            same = new == f[n][cover]
            new[same] = to_storage(1.0 - new[same] * 0.5 - 0.01, dtype)
            f[n][cover] = new
        frames.append(to_storage(f, dtype))
    return frames


def random_sparse_video(seed: int, n_frames: int, N: int, H: int, W: int,
                        C: int, frac: float, dtype: str = "f32",
                        scale: float = 1.0) -> List[np.ndarray]:
    """Reference ~ U[0,scale); each later frame re-draws an unstructured
    random subset (fraction ``frac``) of the sites of every image.  Used for
    small parity cases with ragged, scattered activity."""
    rng = np.random.default_rng(seed)
    f0 = scale * rng.random((N, H, W, C), dtype=np.float32)
    frames = [to_storage(f0, dtype)]
    for _ in range(1, n_frames):
        f = frames[-1].copy()
        m = rng.random((N, H, W)) < frac
        f[m] = scale * rng.random((int(m.sum()), C), dtype=np.float32)
        frames.append(to_storage(f, dtype))
    return frames


def object_video(seed: int = 0, n_frames: int = 8, N: int = 1, H: int = 512,
                 W: int = 512, C: int = 3, obj_frac: float = 0.03,
                 obj: int = 32, dtype: str = "f16") -> List[np.ndarray]:
    """Detection-like frames: a Gaussian-blurred (sigma = 4 px) noise canvas
    scaled to [0, 1] translated by 1-2 px per frame along a random
    direction, plus ceil(obj_frac * H * W / obj^2) textured obj x obj objects
    moving 2-4 px per frame."""
    rng = np.random.default_rng(seed)
    pad = 8 * n_frames + 16
    canvas = torch.from_numpy(rng.random((N * C, 1, H + 2 * pad,
                                          W + 2 * pad), dtype=np.float32))
    r = torch.arange(-12, 13, dtype=torch.float32)
    k1 = torch.exp(-r ** 2 / (2 * 4.0 ** 2))
    k1 = (k1 / k1.sum())
    canvas = F.conv2d(canvas, k1.view(1, 1, 1, -1), padding=(0, 12))
    canvas = F.conv2d(canvas, k1.view(1, 1, -1, 1), padding=(12, 0))
    canvas = canvas.view(N, C, H + 2 * pad, W + 2 * pad)
    lo = canvas.amin(dim=(1, 2, 3), keepdim=True)
    hi = canvas.amax(dim=(1, 2, 3), keepdim=True)
    canvas = ((canvas - lo) / (hi - lo)).permute(0, 2, 3, 1).numpy()
    n_obj = int(np.ceil(obj_frac * H * W / obj ** 2))
    tex = rng.random((N, n_obj, obj, obj, C), dtype=np.float32)
    pos = rng.uniform(0, [H - obj, W - obj], (N, n_obj, 2))
    vel = rng.uniform(2, 4, (N, n_obj, 2)) * rng.choice([-1, 1],
                                                         (N, n_obj, 2))
    ang = rng.uniform(0, 2 * np.pi, N)
    step = rng.uniform(1, 2, N)
    frames = []
    for t in range(n_frames):
        f = np.empty((N, H, W, C), np.float32)
        for n in range(N):
            dy = int(round(pad + t * step[n] * np.sin(ang[n])))
            dx = int(round(pad + t * step[n] * np.cos(ang[n])))
            f[n] = canvas[n, dy:dy + H, dx:dx + W]
            for j in range(n_obj):
                y, x = (pos[n, j] + t * vel[n, j]).astype(int)
                y = int(np.clip(y, 0, H - obj))
                x = int(np.clip(x, 0, W - obj))
                f[n, y:y + obj, x:x + obj] = tex[n, j]
        frames.append(to_storage(f, dtype))
    return frames


def multistream_video(seed: int = 7, n_frames: int = 8, N: int = 32,
                      H: int = 256, W: int = 256, C: int = 3,
                      dens=(0.01, 0.30), dtype: str = "bf16"):
    """N independent streams: stream s has its own seed (2000 + s) and a
    change density drawn uniformly from `dens` with the master seed; each
    stream is a driving-like video whose later frames re-draw rectangles
    (sides 16-64) until that density is covered.  Returns (frames,
    densities)."""
    rng = np.random.default_rng(seed)
    d = rng.uniform(dens[0], dens[1], N)
    per = [driving_video(seed=2000 + s, n_frames=n_frames, N=1, H=H, W=W,
                         C=C, density=float(d[s]), side=(16, 64),
                         dtype=dtype) for s in range(N)]
    frames = [np.concatenate([per[s][t] for s in range(N)], axis=0)
              for t in range(n_frames)]
    return frames, d
