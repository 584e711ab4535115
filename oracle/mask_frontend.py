"""Plain CPU oracle of Sphinx's spatial refinement mask (Sec. 5.3; Alg. 1
laplacian_var, otsu(norm(.)), the opacity mask 1[O < tau_o] and their union).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  It shares
no code with the HIP path and imports nothing from it.

Every step is integer-exact (numpy int64 and Python integers), so the GPU
result must match bit for bit:

* Sec. 5.3, opacity cue: pixels whose opacity is below the threshold (strict,
  0.5 in Sec. 6) are uncertain.
* Sec. 5.3, blur cue: the variance of the Laplacian of the image intensity is
  a reference-free sharpness measure; high variance means sharp.  Computed in
  a window around every pixel, it gives a blur map that is smoothed,
  normalised, inverted, and thresholded with Otsu's method (one threshold per
  frame); 1 marks blurry pixels.
* Alg. 1: the refinement mask is the union of the two masks.
* Sec. 5.3, block rule: a block is refined if any of its pixels is in the
  mask.  A latent token covers 16 x 16 image pixels (8x VAE, 2x2 patch).

Readings where the paper is silent (also listed in the design notes):
intensity is integer BT.601 luma Y = (77 R + 150 G + 29 B + 128) >> 8; the
Laplacian is the 4-neighbour stencil; windows are 9 x 9 for the variance and
5 x 5 box for the smoothing; every stencil reads its input map with
replicated borders; the variance is kept as the exact integer n^2 var =
n sum(L^2) - (sum L)^2 (n = 81); normalisation is per-frame min-max to
0..255 with floor division; Otsu maximises the between-class variance over
thresholds t = 0..254 (class 0 = values <= t), exact rational comparison,
the smallest t among equal maxima; blurry = inverted value > t.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence

import numpy as np

VAR_RADIUS = 4  # 9 x 9 window
SMOOTH_RADIUS = 2  # 5 x 5 box
PIXELS_PER_TOKEN = 16  # 8x VAE downsampling times the 2x2 patch


def luma(rgb: np.ndarray) -> np.ndarray:
    """Integer BT.601 luma of uint8 RGB [..., 3] -> int64 0..255."""
    c = rgb.astype(np.int64)
    return (77 * c[..., 0] + 150 * c[..., 1] + 29 * c[..., 2] + 128) >> 8


def window_sum(img: np.ndarray, radius: int) -> np.ndarray:
    """Sum over the (2r+1)^2 window around every pixel of a 2-D map, the map
    extended by replicating its border pixels."""
    H, W = img.shape
    p = np.pad(img, radius, mode="edge")
    out = np.zeros((H, W), dtype=np.int64)
    for dy in range(2 * radius + 1):
        for dx in range(2 * radius + 1):
            out += p[dy:dy + H, dx:dx + W]
    return out


def laplacian(gray: np.ndarray) -> np.ndarray:
    """4-neighbour Laplacian up + down + left + right - 4 centre, replicated border."""
    H, W = gray.shape
    p = np.pad(gray.astype(np.int64), 1, mode="edge")
    return p[0:H, 1:W + 1] + p[2:H + 2, 1:W + 1] + p[1:H + 1, 0:W] + p[1:H + 1, 2:W + 2] - 4 * p[1:H + 1, 1:W + 1]


def laplacian_variance(gray: np.ndarray) -> np.ndarray:
    """n^2 times the variance of the Laplacian in the 9 x 9 window of every pixel."""
    L = laplacian(gray)
    n = (2 * VAR_RADIUS + 1) ** 2
    s1 = window_sum(L, VAR_RADIUS)
    s2 = window_sum(L * L, VAR_RADIUS)
    return n * s2 - s1 * s1


def normalise_invert(w: np.ndarray) -> np.ndarray:
    """Min-max to 0..255 (floor), then inverted: 255 - q.  A constant map gives q = 0."""
    lo, hi = int(w.min()), int(w.max())
    q = np.zeros(w.shape, dtype=np.int64) if hi == lo else (255 * (w - lo)) // (hi - lo)
    return 255 - q


def otsu_threshold(values: np.ndarray) -> int:
    """Otsu's threshold of 8-bit values: the t in 0..254 maximising the
    between-class variance w0 w1 (mu0 - mu1)^2 (class 0 = values <= t),
    compared exactly; the smallest such t.  Scaled by W^2 the criterion is
    (S w0 - W s0)^2 / (w0 w1), with w0, s0 the count and sum of class 0 and
    W, S those of all values; an empty class scores 0."""
    hist = np.bincount(values.ravel().astype(np.int64), minlength=256)
    Wt = int(hist.sum())
    St = int((np.arange(256) * hist).sum())
    best, best_t = Fraction(-1), 0
    w0 = s0 = 0
    for t in range(255):
        w0 += int(hist[t])
        s0 += t * int(hist[t])
        w1 = Wt - w0
        score = Fraction(0) if w0 == 0 or w1 == 0 else Fraction((St * w0 - Wt * s0) ** 2, w0 * w1)
        if score > best:
            best, best_t = score, t
    return best_t


def blur_mask(rgb: np.ndarray) -> (np.ndarray, int):
    """Per-pixel blur mask of one frame (uint8 RGB [H][W][3]) and its Otsu threshold."""
    v = laplacian_variance(luma(rgb))
    w = window_sum(v, SMOOTH_RADIUS)
    inv = normalise_invert(w)
    t = otsu_threshold(inv)
    return inv > t, t


def frame_mask(rgb: np.ndarray, opacity: np.ndarray, tau_o: float = 0.5):
    """Alg. 1: M = M_op OR M_blur for one frame; returns (pixel mask, Otsu threshold)."""
    mb, t = blur_mask(rgb)
    mop = np.asarray(opacity, np.float32) < np.float32(tau_o)
    return mop | mb, t


def token_mask(pixel_mask: np.ndarray) -> np.ndarray:
    """Block rule of Sec. 5.3: a token (16 x 16 pixels) is selected iff any of its pixels is."""
    H, W = pixel_mask.shape
    P = PIXELS_PER_TOKEN
    out = np.zeros((H // P, W // P), dtype=bool)
    for y in range(H // P):
        for x in range(W // P):
            out[y, x] = pixel_mask[y * P:(y + 1) * P, x * P:(x + 1) * P].any()
    return out


def request_masks(requests: Sequence, rgb: Sequence[np.ndarray], opacity: Sequence[np.ndarray],
                  tau_o: float = 0.5):
    """Token mask of every request (concatenated in token order) and the Otsu
    threshold of every frame.  rgb[r]: uint8 [F][8h][8w][3]; opacity[r]:
    float32 [F][8h][8w]."""
    toks: List[np.ndarray] = []
    thr: List[int] = []
    for q, im, op in zip(requests, rgb, opacity):
        for f in range(q.frames):
            pm, t = frame_mask(im[f], op[f], tau_o)
            toks.append(token_mask(pm).ravel())
            thr.append(t)
    return np.concatenate(toks), np.array(thr, dtype=np.int64)
