"""Seeded synthetic workloads for the selective-refinement step.

Every input that the CPU oracle and the GPU path consume comes from here:
request shapes, latents ``z0``, injection noise ``eps``, the per-token
uncertainty map ``u``, per-frame thresholds ``thr``, per-frame start indices
``s_start``, per-request step counts and the random-init denoiser weights.
This module holds none of the method's arithmetic (no schedule, no mask, no
denoiser); it only draws numbers and applies the workload recipes.

The paper's own inputs (RE10K / DL3DV / ACID scenes encoded by a trained VAE,
regression outputs and opacity maps, Sec. 6) are not available; these seeded
arrays stand in for them with the paper's shapes: 576x1024 views give a
72x128 latent after the 8x VAE (Sec. 7.1 discussion of Sphinx-S), 21 frames
match two inputs plus 19 targets (Sec. 6).

Layouts (shared contract with the C-ABI):
  * token ``t`` of a request with ``F`` frames and latent ``h x w`` is
    ``t = f*(h/2)*(w/2) + y*(w/2) + x``; requests are concatenated, request
    ``r`` starting at global token ``tok_offset[r]``;
  * latents are NCHW per request, ``[F][4][h][w]``, request ``r`` starting at
    element ``16*tok_offset[r]``;
  * a token's 16 values are ordered ``c*4 + py*2 + px`` (patch 2x2, 4 ch);
  * weights are row-major ``[out][in]`` (``y = x @ W.T + b``).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

SEED_WEIGHTS, SEED_Z0, SEED_EPS, SEED_U, SEED_T = 0, 1, 2, 3, 4
LATENT_C = 4
PATCH = 2
TOKEN_DIM = LATENT_C * PATCH * PATCH  # 16
TEMB_DIM = 256
WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Request:
    frames: int
    h: int  # latent height (pixels of the latent grid)
    w: int  # latent width

    @property
    def hp(self) -> int:
        return self.h // PATCH

    @property
    def wp(self) -> int:
        return self.w // PATCH

    @property
    def tokens(self) -> int:
        return self.frames * self.hp * self.wp


@dataclass(frozen=True)
class ModelCfg:
    D: int
    heads: int
    head_dim: int
    mlp: int
    L: int
    dtype: str  # "f32" or "bf16": storage/operand type of weights, latents
    attention: str = "joint"  # "joint" or "factorised" (even blocks spatial, odd blocks temporal)

    def __post_init__(self):
        assert self.D == self.heads * self.head_dim
        assert self.dtype in ("f32", "bf16")
        assert self.attention in ("joint", "factorised")


@dataclass
class Workload:
    name: str
    model: ModelCfg
    requests: List[Request]
    u: np.ndarray  # float32 [N] per-token uncertainty
    thr: np.ndarray  # float32 [G] per-frame threshold (select iff u > thr)
    s_start: np.ndarray  # int32 [G] per-frame start timestep index
    nsteps: np.ndarray  # int32 [R] DDIM steps per request
    z0: np.ndarray  # float32 [16*N] (bf16-exact when model.dtype == "bf16")
    eps: np.ndarray  # float32 [16*N] (bf16-exact when model.dtype == "bf16")
    weights: Dict[str, np.ndarray] = field(default_factory=dict)
    notes: str = ""

    @property
    def R(self) -> int:
        return len(self.requests)

    @property
    def G(self) -> int:
        return sum(r.frames for r in self.requests)

    @property
    def N(self) -> int:
        return sum(r.tokens for r in self.requests)

    @property
    def tok_offset(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum([r.tokens for r in self.requests])]).astype(np.int64)

    @property
    def frame_offset(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum([r.frames for r in self.requests])]).astype(np.int64)

    @property
    def max_steps(self) -> int:
        return int(self.nsteps.max())


# ----------------------------------------------------------------------------
# number formats
# ----------------------------------------------------------------------------
def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), kept as float32."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _storage(a: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_values(a) if dtype == "bf16" else np.ascontiguousarray(a, dtype=np.float32)


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
def weight_shapes(m: ModelCfg) -> List[tuple]:
    """(name, shape) in draw order; per-block tensors are named ``b{l}.<name>``."""
    D, P = m.D, TOKEN_DIM
    out = [("pe_w", (D, P)), ("pe_b", (D,)),
           ("t1_w", (D, TEMB_DIM)), ("t1_b", (D,)),
           ("t2_w", (D, D)), ("t2_b", (D,))]
    for l in range(m.L):
        out += [(f"b{l}.ada_w", (6 * D, D)), (f"b{l}.ada_b", (6 * D,)),
                (f"b{l}.qkv_w", (3 * D, D)), (f"b{l}.qkv_b", (3 * D,)),
                (f"b{l}.o_w", (D, D)), (f"b{l}.o_b", (D,)),
                (f"b{l}.fc1_w", (m.mlp, D)), (f"b{l}.fc1_b", (m.mlp,)),
                (f"b{l}.fc2_w", (D, m.mlp)), (f"b{l}.fc2_b", (D,))]
    out += [("fada_w", (2 * D, D)), ("fada_b", (2 * D,)),
            ("out_w", (P, D)), ("out_b", (P,))]
    return out


def make_weights(m: ModelCfg, seed: int = SEED_WEIGHTS) -> Dict[str, np.ndarray]:
    """Random-init weights and biases, every value an N(0, 0.02^2) draw."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = {}
    for name, shape in weight_shapes(m):
        x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(WEIGHT_STD)
        w[name] = _storage(x, m.dtype).reshape(shape)
    return w


# ----------------------------------------------------------------------------
# uncertainty recipes (token grid of one request -> [F][hp][wp] float32)
# ----------------------------------------------------------------------------
def _u_uniform(rng, req: Request) -> np.ndarray:
    return rng.random(size=(req.frames, req.hp, req.wp), dtype=np.float64).astype(np.float32)


def _u_lognormal_box(rng, req: Request) -> np.ndarray:
    raw = rng.lognormal(0.0, 1.0, size=(req.frames, req.hp, req.wp))
    acc = np.zeros_like(raw)
    cnt = np.zeros_like(raw)
    for dy in (-1, 0, 1):
        for dx in (-1, 0, 1):
            ys = slice(max(0, dy), req.hp + min(0, dy))
            yd = slice(max(0, -dy), req.hp + min(0, -dy))
            xs = slice(max(0, dx), req.wp + min(0, dx))
            xd = slice(max(0, -dx), req.wp + min(0, -dx))
            acc[:, yd, xd] += raw[:, ys, xs]
            cnt[:, yd, xd] += 1.0
    return (acc / cnt).astype(np.float32)


def _u_blobs(rng, req: Request, centres: int = 20, sigma: float = 8.0, noise: float = 0.1) -> np.ndarray:
    out = np.empty((req.frames, req.hp, req.wp), dtype=np.float64)
    py = (2.0 * np.arange(req.hp) + 0.5)[:, None]
    px = (2.0 * np.arange(req.wp) + 0.5)[None, :]
    for f in range(req.frames):
        cy = rng.random(centres) * req.h
        cx = rng.random(centres) * req.w
        acc = np.zeros((req.hp, req.wp))
        for i in range(centres):
            acc += np.exp(-((py - cy[i]) ** 2 + (px - cx[i]) ** 2) / (2.0 * sigma * sigma))
        out[f] = acc + noise * rng.random((req.hp, req.wp))
    return out.astype(np.float32)


# ----------------------------------------------------------------------------
# threshold recipes
# ----------------------------------------------------------------------------
def rho_threshold(values: np.ndarray, rho: float) -> np.float32:
    """Threshold so that ``values > thr`` selects k = floor(rho*n + 0.5) of n.

    The threshold is one of the values themselves (or +-inf), so the strict
    comparison is exact; ties at the boundary select fewer than k.
    """
    v = np.sort(np.asarray(values, dtype=np.float32).ravel())
    n = v.size
    k = int(np.floor(rho * n + 0.5))
    if k >= n:
        return np.float32(-np.inf)
    if k <= 0:
        return np.float32(np.inf)
    return np.float32(v[n - k - 1])


def start_index(t_start: float) -> int:
    """Start timestep index of a normalised start time: round(1000 t) - 1."""
    return int(round(1000.0 * t_start)) - 1


# ----------------------------------------------------------------------------
# workload assembly
# ----------------------------------------------------------------------------
def _latents(requests: Sequence[Request], dtype: str):
    n = sum(r.tokens for r in requests) * TOKEN_DIM
    z0 = np.random.Generator(np.random.PCG64(SEED_Z0)).standard_normal(n, dtype=np.float32)
    eps = np.random.Generator(np.random.PCG64(SEED_EPS)).standard_normal(n, dtype=np.float32)
    return _storage(z0, dtype), _storage(eps, dtype)


def build(name: str, model: ModelCfg, requests: Sequence[Request], u_recipe: Sequence[str],
          thr_rule: Sequence, t_start: Sequence, nsteps: Sequence[int], with_weights: bool = True,
          notes: str = "") -> Workload:
    """Assemble a workload.

    u_recipe[r]  : "uniform" | "lognormal_box" | "blobs"
    thr_rule[r]  : ("value", x) | ("rho", rho) | ("frames_top_then_rho", n_full, rho)
    t_start[r]   : float (shared by the request's frames) or ("uniform", lo, hi) per frame
    """
    requests = list(requests)
    rng_u = np.random.Generator(np.random.PCG64(SEED_U))
    rng_t = np.random.Generator(np.random.PCG64(SEED_T))
    us, thrs, starts = [], [], []
    for r, req in enumerate(requests):
        rec = u_recipe[r]
        if rec == "uniform":
            u = _u_uniform(rng_u, req)
        elif rec == "lognormal_box":
            u = _u_lognormal_box(rng_u, req)
        elif rec == "blobs":
            u = _u_blobs(rng_u, req)
        else:
            raise ValueError(rec)
        rule = thr_rule[r]
        if rule[0] == "value":
            thr = np.full(req.frames, rule[1], dtype=np.float32)
        elif rule[0] == "rho":
            thr = np.full(req.frames, rho_threshold(u, rule[1]), dtype=np.float32)
        elif rule[0] == "frames_top_then_rho":
            n_full, rho = rule[1], rule[2]
            means = u.reshape(req.frames, -1).astype(np.float64).mean(axis=1)
            order = sorted(range(req.frames), key=lambda f: (-means[f], f))
            full = set(order[:n_full])
            thr = np.array([-np.inf if f in full else rho_threshold(u[f], rho)
                            for f in range(req.frames)], dtype=np.float32)
        else:
            raise ValueError(rule)
        ts = t_start[r]
        if isinstance(ts, tuple) and ts[0] == "uniform":
            t = rng_t.uniform(ts[1], ts[2], size=req.frames)
            s = np.array([start_index(x) for x in t], dtype=np.int32)
        else:
            s = np.full(req.frames, start_index(float(ts)), dtype=np.int32)
        us.append(u.ravel())
        thrs.append(thr)
        starts.append(s)
    z0, eps = _latents(requests, model.dtype)
    return Workload(name=name, model=model, requests=requests,
                    u=np.concatenate(us).astype(np.float32),
                    thr=np.concatenate(thrs).astype(np.float32),
                    s_start=np.concatenate(starts).astype(np.int32),
                    nsteps=np.asarray(nsteps, dtype=np.int32),
                    z0=z0, eps=eps,
                    weights=make_weights(model) if with_weights else {},
                    notes=notes)


TINY_MODEL = ModelCfg(D=64, heads=4, head_dim=16, mlp=256, L=1, dtype="f32")
SMALL_MODEL = ModelCfg(D=512, heads=8, head_dim=64, mlp=2048, L=4, dtype="bf16")
HEADLINE_MODEL = ModelCfg(D=1024, heads=16, head_dim=64, mlp=4096, L=12, dtype="bf16")
XL_MODEL = ModelCfg(D=1152, heads=16, head_dim=72, mlp=4608, L=28, dtype="bf16")


def tiny(**kw) -> Workload:
    """2 frames of a 4x8x8 fp32 latent, 32 tokens, U[0,1) uncertainty, thr 0.75, 1 step from 0.5."""
    return build("tiny", TINY_MODEL, [Request(2, 8, 8)], ["uniform"], [("value", 0.75)], [0.5], [1], **kw)


def small(**kw) -> Workload:
    """8 frames of 4x32x32 bf16, 2048 tokens, box-smoothed lognormal map, median threshold, 10 steps from 0.6."""
    return build("small", SMALL_MODEL, [Request(8, 32, 32)], ["lognormal_box"], [("rho", 0.5)], [0.6], [10], **kw)


def headline(model: Optional[ModelCfg] = None, rho: float = 0.3, **kw) -> Workload:
    """14 frames of 4x72x128 bf16 (576x1024 views), 32256 tokens, Gaussian-blob map, 30% selected, 25 steps from 0.5."""
    return build("headline", model or HEADLINE_MODEL, [Request(14, 72, 128)], ["blobs"], [("rho", rho)],
                 [0.5], [25], **kw)


def frame_region(model: Optional[ModelCfg] = None, **kw) -> Workload:
    """21 frames of 4x64x64; top-8 frames fully refined, the rest 15% region-masked; per-frame t_start ~ U[0.3,0.7]."""
    return build("frame_region", model or XL_MODEL, [Request(21, 64, 64)], ["blobs"],
                 [("frames_top_then_rho", 8, 0.15)], [("uniform", 0.3, 0.7)], [25], **kw)


def batched(model: Optional[ModelCfg] = None, **kw) -> Workload:
    """4 requests packed varlen: (6,32x32,10%), (14,72x128,30%), (21,64x64,60%), (8,64x64,100%)."""
    reqs = [Request(6, 32, 32), Request(14, 72, 128), Request(21, 64, 64), Request(8, 64, 64)]
    return build("batched", model or HEADLINE_MODEL, reqs, ["blobs"] * 4,
                 [("rho", 0.1), ("rho", 0.3), ("rho", 0.6), ("rho", 1.0)],
                 [0.3, 0.5, 0.7, 0.5], [10, 25, 25, 10], **kw)


def custom(name: str, model: ModelCfg, requests: Sequence[Request], rho: Sequence[float],
           t_start: Sequence, nsteps: Sequence[int], u_recipe: str = "blobs", **kw) -> Workload:
    """A test workload with the blob (or other) recipe and per-request selected fraction."""
    return build(name, model, requests, [u_recipe] * len(requests), [("rho", x) for x in rho],
                 t_start, nsteps, **kw)


CONFIGS = {"tiny": tiny, "small": small, "headline": headline,
           "frame_region": frame_region, "batched": batched}


# ----------------------------------------------------------------------------
# image-space inputs of the mask front-end (regression output frames and opacity)
# ----------------------------------------------------------------------------
SEED_IMAGES = 5
IMAGE_SCALE = 8  # image pixels per latent pixel (8x VAE)


def _box_blur(img: np.ndarray, r: int) -> np.ndarray:
    """(2r+1)^2 box mean of an [H][W][C] float image with clamped borders (input synthesis only)."""
    H, W = img.shape[:2]
    p = np.pad(img, ((r, r), (r, r), (0, 0)), mode="edge")
    c = np.cumsum(np.cumsum(p, axis=0), axis=1)
    c = np.pad(c, ((1, 0), (1, 0), (0, 0)))
    k = 2 * r + 1
    s = c[k:k + H, k:k + W] - c[0:H, k:k + W] - c[k:k + H, 0:W] + c[0:H, 0:W]
    return s / (k * k)


def frontend_frame(rng, H: int, W: int, blur_discs: int = 5, holes: int = 6):
    """One synthetic regression output: a textured RGB frame (uint8 [H][W][3])
    with `blur_discs` box-blurred discs standing in for motion blur, and an
    opacity map (float32 [H][W]) near 1 with `holes` low-opacity Gaussian
    holes standing in for disoccluded regions."""
    yy, xx = np.mgrid[0:H, 0:W].astype(np.float64)
    base = np.zeros((H, W, 3))
    for c in range(3):
        for _ in range(3):
            fy, fx, ph = rng.random(3) * np.array([6.0, 6.0, 6.28])
            base[..., c] += 40.0 * np.sin(2 * np.pi * (fy * yy / H + fx * xx / W) + ph)
    sharp = np.clip(128.0 + base + rng.uniform(-48.0, 48.0, size=(H, W, 3)), 0, 255)
    blurred = _box_blur(sharp, 3)
    inside = np.zeros((H, W), bool)
    for _ in range(blur_discs):
        cy, cx = rng.random() * H, rng.random() * W
        rad = (0.05 + 0.1 * rng.random()) * min(H, W)
        inside |= (yy - cy) ** 2 + (xx - cx) ** 2 < rad * rad
    img = np.where(inside[..., None], blurred, sharp)
    rgb = np.rint(img).astype(np.uint8)
    opac = np.ones((H, W))
    for _ in range(holes):
        cy, cx = rng.random() * H, rng.random() * W
        sig = (0.02 + 0.04 * rng.random()) * min(H, W)
        opac -= 0.95 * np.exp(-((yy - cy) ** 2 + (xx - cx) ** 2) / (2 * sig * sig))
    opac = np.clip(opac + 0.02 * rng.standard_normal((H, W)), 0.0, 1.0).astype(np.float32)
    return rgb, opac


def frontend_inputs(requests: Sequence[Request], seed: int = SEED_IMAGES):
    """Per request: RGB frames uint8 [F][8h][8w][3] and opacity float32 [F][8h][8w]."""
    rng = np.random.default_rng(seed)
    rgb, opac = [], []
    for q in requests:
        H, W = IMAGE_SCALE * q.h, IMAGE_SCALE * q.w
        frames = [frontend_frame(rng, H, W) for _ in range(q.frames)]
        rgb.append(np.stack([f[0] for f in frames]))
        opac.append(np.stack([f[1] for f in frames]))
    return rgb, opac


SEED_QUALITY = 6


def quality_scores(requests: Sequence[Request], seed: int = SEED_QUALITY):
    """Synthetic perceptual quality scores standing in for MUSIQ (Sec. 5.1):
    per request the two input views' scores U[40, 75) (float32 [R][2]) and per
    frame a regression output score U[0.7, 1.05) times the mean of the two."""
    rng = np.random.default_rng(seed)
    q_in = rng.uniform(40.0, 75.0, size=(len(requests), 2)).astype(np.float32)
    q_reg = np.concatenate([rng.uniform(0.7, 1.05, q.frames) * q_in[r].mean() for r, q in enumerate(requests)])
    return q_in, q_reg.astype(np.float32)
