"""Pins of the mask front-end oracle (Sec. 5.3; Alg. 1 laplacian_var, otsu,
opacity mask and union) and the mistakes they catch.

The pins check the oracle against scipy's Laplacian and integer convolution,
brute force on tiny inputs, the textbook within-class form of Otsu's method,
closed forms (a quadratic image, a two-spike histogram, a ramp) and the
behaviour the paper describes (blurry regions are selected, sharp ones not).
Each planted mistake is applied to a monkeypatched copy on the CPU."""
import math

import numpy as np
import pytest

import oracle.mask_frontend as M

_orig = {n: getattr(M, n) for n in dir(M) if callable(getattr(M, n))}


def pin_luma(M):
    px = np.array([[255, 255, 255], [0, 0, 0], [255, 0, 0], [0, 255, 0], [0, 0, 255], [10, 200, 30]], np.uint8)
    got = M.luma(px)
    assert list(got[:2]) == [255, 0]
    ref = 0.299 * px[:, 0] + 0.587 * px[:, 1] + 0.114 * px[:, 2]
    assert np.abs(got - ref).max() <= 1.0
    rng = np.random.default_rng(1)
    im = rng.integers(0, 256, (50, 3), dtype=np.uint8)
    assert np.abs(M.luma(im) - (0.299 * im[:, 0] + 0.587 * im[:, 1] + 0.114 * im[:, 2])).max() <= 1.0


def pin_laplacian(M):
    from scipy import ndimage

    rng = np.random.default_rng(2)
    g = rng.integers(0, 256, (23, 31)).astype(np.int64)
    assert np.array_equal(M.laplacian(g), ndimage.laplace(g, mode="nearest"))
    y = np.arange(12, dtype=np.int64)[:, None] * np.ones((1, 9), np.int64)
    lap = M.laplacian(y * y)
    assert (lap[1:-1] == 2).all()  # second difference of y^2


def pin_window_sums(M):
    from scipy import ndimage

    rng = np.random.default_rng(3)
    a = rng.integers(-1020, 1021, (19, 27)).astype(np.int64)
    for r in (1, 2, 4):
        ref = ndimage.convolve(a, np.ones((2 * r + 1, 2 * r + 1), np.int64), mode="nearest")
        assert np.array_equal(M.window_sum(a, r), ref)


def pin_local_variance(M):
    rng = np.random.default_rng(4)
    g = rng.integers(0, 256, (14, 17)).astype(np.int64)
    got = M.laplacian_variance(g)
    L = M.laplacian(g)
    H, W = g.shape
    r = 4
    n = (2 * r + 1) ** 2
    for y in range(H):
        for x in range(W):
            win = [L[min(max(y + dy, 0), H - 1), min(max(x + dx, 0), W - 1)] for dy in range(-r, r + 1)
                   for dx in range(-r, r + 1)]
            assert abs(got[y, x] - n * n * np.var(np.array(win, np.float64))) <= 1e-6 * max(1.0, got[y, x])


def pin_normalise(M):
    assert (M.normalise_invert(np.full((3, 4), 7, np.int64)) == 255).all()
    ramp = np.arange(0, 511, dtype=np.int64).reshape(1, -1)
    inv = M.normalise_invert(ramp)
    assert inv[0, 0] == 255 and inv[0, -1] == 0
    assert np.array_equal(inv[0], 255 - (255 * np.arange(511)) // 510)


def _otsu_within(values):
    """Textbook Otsu: the t minimising the within-class variance w0 var0 + w1 var1."""
    v = values.astype(np.float64).ravel()
    best, bt = math.inf, None
    for t in range(255):
        a, b = v[v <= t], v[v > t]
        if a.size == 0 or b.size == 0:
            continue
        s = a.size * a.var() + b.size * b.var()
        if bt is None or s < best - 1e-9 * max(1.0, best):
            best, bt = s, t
    return bt


def pin_otsu(M):
    two = np.array([30] * 50 + [200] * 70)
    assert M.otsu_threshold(two) == 30  # every t in [30, 199] is optimal: the smallest
    rng = np.random.default_rng(5)
    for _ in range(6):
        vals = np.concatenate([rng.normal(rng.uniform(40, 110), 15, 300), rng.normal(rng.uniform(140, 220), 20, 500)])
        vals = np.clip(np.rint(vals), 0, 255).astype(np.int64)
        assert M.otsu_threshold(vals) == _otsu_within(vals)
    assert M.otsu_threshold(np.full(10, 77)) == 0  # one class only: every score is 0


def pin_token_pool(M):
    m = np.zeros((32, 48), bool)
    m[17, 47] = True
    t = M.token_mask(m)
    assert t.shape == (2, 3) and t.sum() == 1 and t[1, 2]
    m[:] = False
    m[15, 16] = True
    assert M.token_mask(m)[0, 1] and M.token_mask(m).sum() == 1


def pin_opacity_strict(M):
    rgb = np.full((16, 16, 3), 128, np.uint8)  # flat: every pixel blurry
    rng = np.random.default_rng(6)
    sharp = rng.integers(0, 256, (16, 16, 3), dtype=np.uint8)
    op = np.full((16, 16), 0.5, np.float32)
    pm, _ = M.frame_mask(sharp, op)
    mb, _ = M.blur_mask(sharp)
    assert np.array_equal(pm, mb)  # O = 0.5 is not below 0.5
    op[3, 4] = np.nextafter(np.float32(0.5), np.float32(0))
    pm2, _ = M.frame_mask(sharp, op)
    assert pm2[3, 4] and (pm2 ^ pm).sum() <= 1
    assert M.frame_mask(rgb, np.ones((16, 16), np.float32))[0].all()


def pin_blur_selects_blurry_half(M):
    rng = np.random.default_rng(7)
    H, W = 64, 128
    img = rng.integers(0, 256, (H, W, 3)).astype(np.float64)
    img[:, W // 2:] = 120.0 + 0.2 * (np.arange(W // 2)[None, :, None])  # smooth ramp: no edges
    mb, _ = M.blur_mask(np.rint(img).astype(np.uint8))
    band = M.VAR_RADIUS + M.SMOOTH_RADIUS + 1
    assert mb[:, W // 2 + band:].all()
    # away from the seam and from the top and bottom rows (whose replicated
    # border lowers the local variance) the textured half stays unselected
    assert not mb[band:H - band, : W // 2 - band].any()


PINS = [pin_luma, pin_laplacian, pin_window_sums, pin_local_variance, pin_normalise, pin_otsu, pin_token_pool,
        pin_opacity_strict, pin_blur_selects_blurry_half]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_frontend_pin(pin):
    pin(M)


def _luma_rb_swapped(rgb):
    return _orig["luma"](rgb[..., ::-1])


def _lap_8(gray):
    H, W = gray.shape
    p = np.pad(gray.astype(np.int64), 1, mode="edge")
    s = sum(p[dy:dy + H, dx:dx + W] for dy in range(3) for dx in range(3))
    return s - 9 * p[1:H + 1, 1:W + 1]


def _window_zero_pad(img, radius):
    H, W = img.shape
    p = np.pad(img, radius)
    return sum(p[dy:dy + H, dx:dx + W] for dy in range(2 * radius + 1) for dx in range(2 * radius + 1))


def _lapvar_radius3(gray):
    L = M.laplacian(gray)
    s1, s2 = _orig["window_sum"](L, 3), _orig["window_sum"](L * L, 3)
    return 81 * s2 - s1 * s1


def _no_invert(w):
    return 255 - _orig["normalise_invert"](w)


def _otsu_strict_class(values):
    return max(_orig["otsu_threshold"](values) - 1, 0)


def _otsu_last_max(values):
    hist = np.bincount(values.ravel().astype(np.int64), minlength=256)
    Wt, St = int(hist.sum()), int((np.arange(256) * hist).sum())
    best, bt, w0, s0 = -1.0, 0, 0, 0
    for t in range(255):
        w0 += int(hist[t])
        s0 += t * int(hist[t])
        w1 = Wt - w0
        sc = 0.0 if w0 == 0 or w1 == 0 else (St * w0 - Wt * s0) ** 2 / (w0 * w1)
        if sc >= best:
            best, bt = sc, t
    return bt


def _pool_corner(pixel_mask):
    return pixel_mask[::16, ::16].copy()


def _frame_mask_le(rgb, opacity, tau_o=0.5):
    mb, t = M.blur_mask(rgb)
    return (np.asarray(opacity, np.float32) <= np.float32(tau_o)) | mb, t


MUTANTS = {
    "luma_rb_swapped": ("luma", _luma_rb_swapped),
    "laplacian_8_neighbour": ("laplacian", _lap_8),
    "window_zero_border": ("window_sum", _window_zero_pad),
    "variance_window_7x7": ("laplacian_variance", _lapvar_radius3),
    "normalise_not_inverted": ("normalise_invert", _no_invert),
    "otsu_class_boundary": ("otsu_threshold", _otsu_strict_class),
    "otsu_last_maximum": ("otsu_threshold", _otsu_last_max),
    "pool_one_pixel": ("token_mask", _pool_corner),
    "opacity_not_strict": ("frame_mask", _frame_mask_le),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_frontend_pins_catch_mutant(name, monkeypatch):
    attr, bad = MUTANTS[name]
    monkeypatch.setattr(M, attr, bad)
    caught = []
    for pin in PINS:
        try:
            pin(M)
        except Exception as e:
            caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught {name}"
    print(name, caught)
