"""Plain CPU oracle of Sphinx's selective partial-denoising step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  It shares
no code with the HIP path (``paper_2511_18672_amd``) and imports nothing from
it; the only module both sides use is ``workloads`` (seeded inputs, no method
arithmetic).

Everything is numpy in float64.  It is slow and meant to be checked by eye
against the paper (Sphinx, arXiv 2511.18672):

* Alg. 1 ("Sphinx Inference"), partial-denoising loop: noise is injected into
  the clean latents at the start step (``add_noise``), the frames whose start
  step has been reached form the active set ``A_u = 1[k <= u]``, and the
  denoiser updates only the active frames (``D.partial_step``) restricted to
  the mask ``M``.
* Sec. 5.3 (spatially selective refinement): only positions inside the binary
  mask are forwarded to the diffusion model; confident regions bypass the
  partial denoising entirely and keep their values.
* Sec. 5.2 (temporally consistent partial denoising) and Alg. 1's full_step /
  store_temporal: with a cache period T, every T-th step forwards every token
  and the keys and values of every block are cached; the steps in between
  forward the masked tokens only and attend to the rest through the cache.
  Tokens forwarded only as context enter as their clean latents noised to the
  step's level (Alg. 1 resamples inactive content from the clean latents).
* Sec. 3 (hybrid proposal): the regression output, with controlled noise
  injected, replaces Gaussian-noise initialisation and partial denoising
  removes the added noise.
* Sec. 6: 1000-step training schedule sampled with 50 inference steps; opacity
  threshold 0.5 with strict "below" comparison.

Where the paper is silent (sampler, beta schedule, timestep spacing, denoiser
architecture, threshold semantics, attention context), this module follows the
readings listed in the design notes (sampler DDIM eta=0 with eps-prediction,
linear betas 1e-4..2e-2, trailing grid from the start index, DiT-style adaLN
blocks with (1+gate) residuals, strict ``u > thr`` with NaN unselected,
attention over the selected tokens of one request).

Precision modes:
  ``precision="fp64"``  -- every value in float64 (the "truth").
  ``precision="model"`` -- float64 arithmetic, but for a bf16 model the
      operands that the model declares as bf16 are rounded to bf16
      (round-to-nearest-even) exactly where the model stores them: the
      adaLN-modulated LayerNorm outputs fed to the QKV and MLP1 GEMMs, the
      query scaled by log2(e)/sqrt(d) (the model keeps its queries in the
      units of a base-2 softmax, so the 1/sqrt(d) of the attention is applied
      before the query is stored, not after), k, v, the attention output, and
      the GELU output fed to MLP2.  Weights and
      latents are bf16 values already.  Residual stream, statistics, softmax,
      conditioning, noise prediction and the DDIM update stay float64.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

T_TRAIN = 1000
BETA_START = 1e-4
BETA_END = 2e-2
LN_EPS = 1e-6
TEMB_DIM = 256
TOKEN_DIM = 16


# ----------------------------------------------------------------------------
# number format: bfloat16 round-to-nearest-even on float64 data
# ----------------------------------------------------------------------------
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (ties to even) of each element, returned as float64.

    bfloat16 keeps the float32 exponent and the top 7 stored mantissa bits.
    The value is first rounded to float32 (RNE), then the low 16 bits of the
    float32 pattern are rounded away with ties to even.  NaN stays NaN.
    """
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    out = rounded.astype(np.uint32).view(np.float32).astype(np.float64)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.nan
    return out


# ----------------------------------------------------------------------------
# noise schedule and sampler (reading: linear betas, DDIM eta = 0)
# ----------------------------------------------------------------------------
def betas() -> np.ndarray:
    """Linear beta schedule over the 1000 training timesteps."""
    i = np.arange(T_TRAIN, dtype=np.float64)
    return BETA_START + (BETA_END - BETA_START) * i / (T_TRAIN - 1)


def alpha_bar() -> np.ndarray:
    """Cumulative product of (1 - beta_i), i <= t, for t = 0..999."""
    return np.cumprod(1.0 - betas())


def abar_at(t: int, ab: Optional[np.ndarray] = None) -> float:
    """alpha_bar at timestep t; t = -1 denotes the clean end point (alpha_bar = 1)."""
    if t < 0:
        return 1.0
    ab = alpha_bar() if ab is None else ab
    return float(ab[t])


def timestep_grid(s_max: int, n: int) -> List[int]:
    """The n+1 timesteps visited by n steps starting at index s_max.

    tau_i = floor((n - i)(s_max + 1) / n) - 1, so tau_0 = s_max and tau_n = -1.
    At s_max = 499, n = 25 this is the last 25 entries of a 50-step grid with
    spacing 20 (the paper's S = 50 with refinement starting at k = 25).
    """
    return [((n - i) * (s_max + 1)) // n - 1 for i in range(n + 1)]


def injection_coeffs(t: int, ab=None):
    """(a, b) with add_noise(z0, t) = a*z0 + b*eps: a = sqrt(abar_t), b = sqrt(1 - abar_t)."""
    a_t = abar_at(t, ab)
    return np.sqrt(a_t), np.sqrt(1.0 - a_t)


def ddim_coeffs(t: int, t_next: int, ab=None):
    """(c1, c2) of the deterministic DDIM update x' = c1*x + c2*eps_hat.

    x0_hat = (x - sqrt(1-abar)*eps_hat)/sqrt(abar);
    x'     = sqrt(abar')*x0_hat + sqrt(1-abar')*eps_hat.
    """
    a, an = abar_at(t, ab), abar_at(t_next, ab)
    c1 = np.sqrt(an / a)
    c2 = np.sqrt(1.0 - an) - np.sqrt(an * (1.0 - a) / a)
    return c1, c2


@dataclass
class StepPlan:
    active: np.ndarray  # bool [G]
    newly: np.ndarray  # bool [G]
    tau: np.ndarray  # int [G] (timestep of the frame's request at this step; -1 if idle)
    a: np.ndarray  # float64 [G]
    b: np.ndarray
    c1: np.ndarray
    c2: np.ndarray
    full: Optional[np.ndarray] = None  # bool [R]: the request takes a full step (latent cache only)
    a_ctx: Optional[np.ndarray] = None  # float64 [G]: add_noise(z0, tau_i) coefficients of context tokens
    b_ctx: Optional[np.ndarray] = None


def plan_steps(frames_per_req: Sequence[int], s_start: np.ndarray, nsteps: Sequence[int],
               period: int = 0, per_frame_grid: bool = False) -> List[StepPlan]:
    """Per-step, per-frame schedule (Alg. 1 loop with a per-frame start step).

    Each request walks its own grid from s_max = max of its frames' start
    indices.  Frame f is active at step i iff tau_i <= s_f (it has reached its
    own start); on its first active step it is newly active and receives
    add_noise at level tau_i.  A request takes part in global step i iff
    i < nsteps[r].

    With a cache period T = ``period`` > 0 (Alg. 1: a full step when the step
    counter is a multiple of T), a live request takes a full step at every i
    with i mod T = 0, counted from its first step so that the first step
    always fills the cache.  Every frame of a live request gets the context
    coefficients (a_ctx, b_ctx) = (sqrt(abar(tau_i)), sqrt(1 - abar(tau_i))):
    a token forwarded only as context enters as add_noise of its clean latent
    at the step's level (Alg. 1 resamples inactive content from the clean
    latents).

    per_frame_grid=True is the other reading of Alg. 1's per-frame start:
    every frame walks its own n-step grid from its own s_f, so all frames are
    active from the first step (newly active there) at their own timesteps.
    """
    ab = alpha_bar()
    G = int(sum(frames_per_req))
    total = int(max(nsteps))
    out = []
    R = len(frames_per_req)
    for i in range(total):
        p = StepPlan(np.zeros(G, bool), np.zeros(G, bool), np.full(G, -1, np.int64),
                     np.ones(G), np.zeros(G), np.ones(G), np.zeros(G),
                     np.zeros(R, bool), np.ones(G), np.zeros(G))
        g0 = 0
        for r, F in enumerate(frames_per_req):
            n = int(nsteps[r])
            if i < n:
                s = s_start[g0:g0 + F]
                grid = timestep_grid(int(max(s)), n)
                t, tn = grid[i], grid[i + 1]
                c1, c2 = ddim_coeffs(t, tn, ab)
                p.full[r] = period > 0 and i % period == 0
                for f in range(F):
                    g = g0 + f
                    if per_frame_grid:
                        own = timestep_grid(int(s[f]), n)
                        p.tau[g] = own[i]
                        p.active[g] = True
                        p.newly[g] = i == 0
                        p.c1[g], p.c2[g] = ddim_coeffs(own[i], own[i + 1], ab)
                        p.a_ctx[g], p.b_ctx[g] = injection_coeffs(own[i], ab)
                        if i == 0:
                            p.a[g], p.b[g] = injection_coeffs(own[0], ab)
                        continue
                    p.tau[g] = t
                    p.a_ctx[g], p.b_ctx[g] = injection_coeffs(t, ab)
                    if t <= s[f]:
                        p.active[g] = True
                        p.newly[g] = (i == 0) or (grid[i - 1] > s[f])
                        p.c1[g], p.c2[g] = c1, c2
                        if p.newly[g]:
                            p.a[g], p.b[g] = injection_coeffs(t, ab)
            g0 += F
        out.append(p)
    return out


# ----------------------------------------------------------------------------
# token geometry
# ----------------------------------------------------------------------------
@dataclass
class TokenInfo:
    req: np.ndarray  # request of each token
    gframe: np.ndarray  # global frame index
    f: np.ndarray  # frame index inside its request
    y: np.ndarray
    x: np.ndarray


def token_info(requests) -> TokenInfo:
    req, gfr, ff, yy, xx = [], [], [], [], []
    g0 = 0
    for r, q in enumerate(requests):
        hp, wp = q.h // 2, q.w // 2
        f, y, x = np.meshgrid(np.arange(q.frames), np.arange(hp), np.arange(wp), indexing="ij")
        req.append(np.full(f.size, r))
        gfr.append(g0 + f.ravel())
        ff.append(f.ravel())
        yy.append(y.ravel())
        xx.append(x.ravel())
        g0 += q.frames
    cat = lambda a: np.concatenate(a).astype(np.int64)
    return TokenInfo(cat(req), cat(gfr), cat(ff), cat(yy), cat(xx))


def patchify(latent: np.ndarray, requests) -> np.ndarray:
    """NCHW latents of all requests -> [N][16] token rows, value order c*4 + py*2 + px."""
    rows, e0 = [], 0
    for q in requests:
        n = q.frames * 4 * q.h * q.w
        z = np.asarray(latent[e0:e0 + n], dtype=np.float64).reshape(q.frames, 4, q.h // 2, 2, q.w // 2, 2)
        rows.append(z.transpose(0, 2, 4, 1, 3, 5).reshape(-1, TOKEN_DIM))
        e0 += n
    return np.concatenate(rows, axis=0)


def unpatchify(tokens: np.ndarray, requests) -> np.ndarray:
    """Inverse of patchify."""
    out, t0 = [], 0
    for q in requests:
        n = q.frames * (q.h // 2) * (q.w // 2)
        z = tokens[t0:t0 + n].reshape(q.frames, q.h // 2, q.w // 2, 4, 2, 2)
        out.append(z.transpose(0, 3, 1, 4, 2, 5).ravel())
        t0 += n
    return np.concatenate(out)


# ----------------------------------------------------------------------------
# mask and compaction (Sec. 5.3 mask; Alg. 1 opacity mask 1[O < tau_o])
# ----------------------------------------------------------------------------
def select(u: np.ndarray, thr_tok: np.ndarray, active_tok: np.ndarray, tok_offset: np.ndarray):
    """Selected-token mask and its stable compaction.

    mask[t] = active(t) and u[t] > thr(t)  (strict; NaN compares false).
    idx     = ascending positions with mask = 1.
    cu_sel  = number of selected tokens before each request boundary.
    """
    mask = np.logical_and(active_tok, np.asarray(u) > np.asarray(thr_tok))
    idx = np.flatnonzero(mask).astype(np.int64)
    cu = np.array([np.count_nonzero(mask[:o]) for o in tok_offset], dtype=np.int64)
    return mask, idx, cu, int(idx.size)


# ----------------------------------------------------------------------------
# denoiser pieces
# ----------------------------------------------------------------------------
def linear(x, w, b):
    """y = x W^T + b with W stored [out][in]."""
    return x @ np.asarray(w, np.float64).T + np.asarray(b, np.float64)


def silu(z):
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z):
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def layer_norm(h):
    """Normalise each row to zero mean and unit (biased) variance, eps 1e-6, no affine."""
    mu = h.mean(axis=-1, keepdims=True)
    var = ((h - mu) ** 2).mean(axis=-1, keepdims=True)
    return (h - mu) / np.sqrt(var + LN_EPS)


def timestep_embedding(tau: np.ndarray) -> np.ndarray:
    """[len(tau)][256]: cos(tau*w_k) for k < 128, then sin(tau*w_k); w_k = 10^4^(-k/128)."""
    half = TEMB_DIM // 2
    w = np.exp(-np.log(1e4) * np.arange(half) / half)
    arg = np.asarray(tau, np.float64)[:, None] * w[None, :]
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=1)


def position_embedding(f, y, x, D: int) -> np.ndarray:
    """[n][D]: [Ty(y) || Tx(x)] + Tf(f).

    Ty(y) = [sin(y v_k)]_{k<D/4} || [cos(y v_k)]_{k<D/4}, v_k = 10^4^(-k/(D/4)); Tx likewise
    over x; Tf(f) = [sin(f m_k)]_{k<D/2} || [cos(f m_k)]_{k<D/2}, m_k = 10^4^(-k/(D/2)).
    """
    q = D // 4
    nu = 1e4 ** (-np.arange(q) / q)
    mu = 1e4 ** (-np.arange(D // 2) / (D // 2))
    ay = np.asarray(y, np.float64)[:, None] * nu
    ax = np.asarray(x, np.float64)[:, None] * nu
    af = np.asarray(f, np.float64)[:, None] * mu
    spatial = np.concatenate([np.sin(ay), np.cos(ay), np.sin(ax), np.cos(ax)], axis=1)
    return spatial + np.concatenate([np.sin(af), np.cos(af)], axis=1)


def attention(q, k, v, heads: int, seg: np.ndarray, chunk: int = 2048, kv_seg: Optional[np.ndarray] = None,
              scale: Optional[float] = None):
    """Non-causal softmax(scale q k^T) v per head, scale = 1/sqrt(d) unless
    given, each query attending to the keys of its own segment only (segments
    = contiguous row ranges seg[r]..seg[r+1]).

    With kv_seg, the queries of segment r attend to the key/value rows
    kv_seg[r]..kv_seg[r+1] instead (k and v then have their own row count)."""
    n, D = q.shape
    d = D // heads
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.zeros((n, D))
    for r in range(len(seg) - 1):
        s0, s1 = int(seg[r]), int(seg[r + 1])
        k0, k1 = (s0, s1) if kv_seg is None else (int(kv_seg[r]), int(kv_seg[r + 1]))
        if s1 <= s0:
            continue
        for h in range(heads):
            cols = slice(h * d, (h + 1) * d)
            kh, vh = k[k0:k1, cols], v[k0:k1, cols]
            for c0 in range(s0, s1, chunk):
                c1 = min(s1, c0 + chunk)
                s = (q[c0:c1, cols] @ kh.T) * scale
                s -= s.max(axis=1, keepdims=True)
                p = np.exp(s)
                p /= p.sum(axis=1, keepdims=True)
                out[c0:c1, cols] = p @ vh
    return out


def attention_groups(q, k, v, heads: int, gq: np.ndarray, gk: np.ndarray, scale: Optional[float] = None):
    """Non-causal softmax(scale q k^T) v per head (scale = 1/sqrt(d) unless
    given) where query row i attends to the key rows j with gk[j] == gq[i]
    (groups need not be contiguous)."""
    n, D = q.shape
    d = D // heads
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.zeros((n, D))
    for g in np.unique(gq):
        qi = np.flatnonzero(gq == g)
        kj = np.flatnonzero(gk == g)
        for h in range(heads):
            cols = slice(h * d, (h + 1) * d)
            s = (q[qi, cols] @ k[kj, cols].T) * scale
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[qi, cols] = p @ v[kj, cols]
    return out


def block_attention(attn: str, l: int) -> str:
    """Attention of block l: 'joint' over the request, or for a factorised
    denoiser (the spatial / temporal split of the paper's denoisers, Sec. 4 and
    Sec. 5.2) 'spatial' (same frame) in even blocks and 'temporal' (same
    (y, x) position across the request's frames) in odd blocks."""
    if attn == "joint":
        return "joint"
    return "spatial" if l % 2 == 0 else "temporal"


def attention_group_ids(kind: str, req, f, y, x) -> np.ndarray:
    """Group of every token for a spatial or temporal block."""
    key = np.stack([req, f] if kind == "spatial" else [req, y, x], axis=1)
    return np.unique(key, axis=0, return_inverse=True)[1].ravel()


@dataclass
class Model:
    D: int
    heads: int
    mlp: int
    L: int
    dtype: str
    weights: Dict[str, np.ndarray]
    attention: str = "joint"


def model_from_workload(wl) -> Model:
    m = wl.model
    return Model(m.D, m.heads, m.mlp, m.L, m.dtype, wl.weights, getattr(m, "attention", "joint"))


def conditioning(model: Model, tau: np.ndarray) -> np.ndarray:
    """c = W_t2 SiLU(W_t1 temb(tau) + b_t1) + b_t2, one row per timestep."""
    w = model.weights
    return linear(silu(linear(timestep_embedding(tau), w["t1_w"], w["t1_b"])), w["t2_w"], w["t2_b"])


def denoise(model: Model, x: np.ndarray, f, y, xx, tau_tok: np.ndarray, seg: np.ndarray,
            precision: str = "model", cache: Optional[list] = None, rows: Optional[np.ndarray] = None,
            kv_seg: Optional[np.ndarray] = None, kv_pos: Optional[tuple] = None) -> np.ndarray:
    """Noise prediction eps_hat [n][16] for packed tokens x [n][16].

    Tokens carry their in-request frame f, grid position (y, xx) and their
    frame's timestep tau_tok; attention runs inside each segment.

    With a latent cache (Sec. 5.2), ``cache[l] = (K, V)`` holds block l's
    keys and values of every token of the batch (global token order).  Each
    block first stores the keys and values of the forwarded tokens at their
    global positions ``rows``, then the queries of segment r attend to cache
    rows kv_seg[r]..kv_seg[r+1] (all tokens of request r): fresh values for the
    forwarded tokens, the stored ones for the rest.

    A factorised denoiser (model.attention == "factorised") restricts block
    l's attention to the segment's tokens of the same frame (even l) or of the
    same (y, x) position (odd l); with the cache, kv_pos = (f, y, x) of every
    cached token gives the key groups.
    """
    w = model.weights
    D, H = model.D, model.heads
    rnd = round_bf16 if (precision == "model" and model.dtype == "bf16") else (lambda a: a)
    # queries are kept in base-2 softmax units: q' = q log2(e)/sqrt(d), and
    # softmax(q k^T / sqrt(d)) = softmax(ln(2) q' k^T)
    qscale, sscale = np.log2(np.e) / np.sqrt(D // H), np.log(2.0)
    # conditioning, per distinct timestep (identical for equal timesteps)
    taus, inv = np.unique(np.asarray(tau_tok), return_inverse=True)
    c = silu(conditioning(model, taus))
    h = linear(x, w["pe_w"], w["pe_b"]) + position_embedding(f, y, xx, D)
    for l in range(model.L):
        mod = linear(c, w[f"b{l}.ada_w"], w[f"b{l}.ada_b"])[inv]
        sh1, sc1, g1, sh2, sc2, g2 = (mod[:, i * D:(i + 1) * D] for i in range(6))
        a = rnd(layer_norm(h) * (1.0 + sc1) + sh1)
        qkv = linear(a, w[f"b{l}.qkv_w"], w[f"b{l}.qkv_b"])
        q, k, v = rnd(qkv[:, :D] * qscale), rnd(qkv[:, D:2 * D]), rnd(qkv[:, 2 * D:])
        kind = block_attention(model.attention, l)
        if cache is None:
            if kind == "joint":
                o = rnd(attention(q, k, v, H, seg, scale=sscale))
            else:
                req = np.searchsorted(seg, np.arange(x.shape[0]), side="right") - 1
                grp = attention_group_ids(kind, req, f, y, xx)
                o = rnd(attention_groups(q, k, v, H, grp, grp, scale=sscale))
        else:
            cache[l][0][rows] = k
            cache[l][1][rows] = v
            if kind == "joint":
                o = rnd(attention(q, cache[l][0], cache[l][1], H, seg, kv_seg=kv_seg, scale=sscale))
            else:
                n_all = cache[l][0].shape[0]
                req_q = np.searchsorted(seg, np.arange(x.shape[0]), side="right") - 1
                req_k = np.searchsorted(kv_seg, np.arange(n_all), side="right") - 1
                both = attention_group_ids(kind, np.concatenate([req_q, req_k]), np.concatenate([f, kv_pos[0]]),
                                           np.concatenate([y, kv_pos[1]]), np.concatenate([xx, kv_pos[2]]))
                gq, gk = both[:x.shape[0]], both[x.shape[0]:]
                o = rnd(attention_groups(q, cache[l][0], cache[l][1], H, gq, gk, scale=sscale))
        h = h + (1.0 + g1) * linear(o, w[f"b{l}.o_w"], w[f"b{l}.o_b"])
        a2 = rnd(layer_norm(h) * (1.0 + sc2) + sh2)
        m = rnd(gelu_tanh(linear(a2, w[f"b{l}.fc1_w"], w[f"b{l}.fc1_b"])))
        h = h + (1.0 + g2) * linear(m, w[f"b{l}.fc2_w"], w[f"b{l}.fc2_b"])
    fm = linear(c, w["fada_w"], w["fada_b"])[inv]
    shf, scf = fm[:, :D], fm[:, D:]
    return linear(layer_norm(h) * (1.0 + scf) + shf, w["out_w"], w["out_b"])


# ----------------------------------------------------------------------------
# one step and the whole refinement loop
# ----------------------------------------------------------------------------
@dataclass
class StepResult:
    mask: np.ndarray
    idx: np.ndarray
    cu_sel: np.ndarray
    n_sel: int
    x_in: np.ndarray  # gathered (and injected) token rows
    eps_hat: np.ndarray
    x_out: np.ndarray  # after the DDIM update
    state: np.ndarray  # NCHW state after scatter
    qidx: Optional[np.ndarray] = None  # forwarded tokens (latent cache: selected plus context)
    cu_q: Optional[np.ndarray] = None  # forwarded tokens before each request start


def per_token(values_per_frame: np.ndarray, info: TokenInfo) -> np.ndarray:
    return np.asarray(values_per_frame)[info.gframe]


def step(wl, model: Model, state: np.ndarray, plan: StepPlan, precision: str = "model",
         denoiser=None, info: Optional[TokenInfo] = None) -> StepResult:
    """One partial-denoising step: select, compact, gather(+inject), denoise, DDIM, scatter."""
    info = token_info(wl.requests) if info is None else info
    tok_off = wl.tok_offset[:-1]  # request starts
    mask, idx, cu, n = select(wl.u, per_token(wl.thr, info), per_token(plan.active, info), tok_off)
    state = np.array(state, dtype=np.float64, copy=True)
    if n == 0:
        z = np.zeros((0, TOKEN_DIM))
        return StepResult(mask, idx, cu, 0, z, z, z, state)
    P = patchify(state, wl.requests)
    E = patchify(wl.eps, wl.requests)
    g = info.gframe[idx]
    a, b = plan.a[g][:, None], plan.b[g][:, None]
    x = a * P[idx] + b * E[idx]
    seg = np.concatenate([cu, [n]])
    den = denoiser or denoise
    eps_hat = den(model, x, info.f[idx], info.y[idx], info.x[idx], plan.tau[g], seg, precision)
    x_out = plan.c1[g][:, None] * x + plan.c2[g][:, None] * eps_hat
    P[idx] = x_out
    return StepResult(mask, idx, cu, n, x, eps_hat, x_out, unpatchify(P, wl.requests))


def step_cached(wl, model: Model, state: np.ndarray, plan: StepPlan, cache: list, precision: str = "model",
                info: Optional[TokenInfo] = None) -> StepResult:
    """One step of Alg. 1 with the latent cache (Sec. 5.2, Alg. 1 full_step /
    store_temporal / partial_step with the cache).

    The write set is the selection of ``step`` (mask within the active
    frames).  A request taking a full step forwards every one of its tokens;
    otherwise only the write set is forwarded.  Write-set tokens enter as in
    ``step`` (the state, or add_noise on a frame's first active step); the
    other forwarded tokens (context: unselected tokens and inactive frames)
    enter as add_noise(z0, tau_i), their clean latent noised to the step's
    level -- the state still holds z0 there, since only write-set tokens are
    ever written.  The denoiser stores the keys and values of every forwarded
    token in the cache and attends over the whole request through it, so a
    partial step sees the context as it was at the last full step.  The DDIM
    update is applied to the forwarded tokens and written back for the write
    set only (unselected tokens keep their values, Sec. 5.3).
    """
    info = token_info(wl.requests) if info is None else info
    tok_off = wl.tok_offset[:-1]
    mask, idx, cu, n = select(wl.u, per_token(wl.thr, info), per_token(plan.active, info), tok_off)
    forward = mask | plan.full[info.req]
    qidx = np.flatnonzero(forward)
    cu_q = np.array([np.count_nonzero(forward[:o]) for o in tok_off])
    nq = int(qidx.size)
    state = np.array(state, dtype=np.float64, copy=True)
    if nq == 0:
        z = np.zeros((0, TOKEN_DIM))
        return StepResult(mask, idx, cu, n, z, z, z, state, qidx, cu_q)
    P = patchify(state, wl.requests)
    E = patchify(wl.eps, wl.requests)
    g = info.gframe[qidx]
    w = mask[qidx]
    a = np.where(w, plan.a[g], plan.a_ctx[g])[:, None]
    b = np.where(w, plan.b[g], plan.b_ctx[g])[:, None]
    x = a * P[qidx] + b * E[qidx]
    seg = np.concatenate([cu_q, [nq]])
    eps_hat = denoise(model, x, info.f[qidx], info.y[qidx], info.x[qidx], plan.tau[g], seg, precision,
                      cache=cache, rows=qidx, kv_seg=np.asarray(wl.tok_offset), kv_pos=(info.f, info.y, info.x))
    x_out = plan.c1[g][:, None] * x + plan.c2[g][:, None] * eps_hat
    P[qidx[w]] = x_out[w]
    return StepResult(mask, idx, cu, n, x, eps_hat, x_out, unpatchify(P, wl.requests), qidx, cu_q)


def new_cache(model: Model, n_tokens: int) -> list:
    """Per block, keys and values of every token (zeros until a full step writes them)."""
    return [(np.zeros((n_tokens, model.D)), np.zeros((n_tokens, model.D))) for _ in range(model.L)]


def refine(wl, precision: str = "model", denoiser=None, trace: bool = False, steps: Optional[int] = None,
           period: int = 0, per_frame_grid: bool = False):
    """Run the whole partial-denoising loop; returns the final NCHW state (float64)
    and, with trace=True, the list of per-step results.  period > 0 turns on
    the latent cache with a full step every ``period`` steps."""
    model = model_from_workload(wl)
    plans = plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps, period, per_frame_grid)
    info = token_info(wl.requests)
    state = np.asarray(wl.z0, dtype=np.float64).copy()
    cache = new_cache(model, wl.N) if period > 0 else None
    out = []
    for i, p in enumerate(plans[: steps if steps is not None else len(plans)]):
        if cache is not None:
            res = step_cached(wl, model, state, p, cache, precision, info)
        else:
            res = step(wl, model, state, p, precision, denoiser, info)
        state = res.state
        if trace:
            out.append(res)
    return (state, out) if trace else state


def refine_dense(wl, precision: str = "model", denoiser=None):
    """Dense partial denoising of every token of every frame, with no mask, no
    gather and no scatter: the whole latent is noised at the start step and the
    denoiser sees all tokens of each request.  Defined for workloads whose frames
    of a request share one start index."""
    model = model_from_workload(wl)
    info = token_info(wl.requests)
    ab = alpha_bar()
    P = patchify(wl.z0, wl.requests)
    E = patchify(wl.eps, wl.requests)
    seg = np.asarray(wl.tok_offset, dtype=np.int64)
    g0, t0 = 0, 0
    grids = []
    for r, q in enumerate(wl.requests):
        s = wl.s_start[g0:g0 + q.frames]
        assert (s == s[0]).all(), "dense path needs one start index per request"
        grids.append(timestep_grid(int(s[0]), int(wl.nsteps[r])))
        a, b = injection_coeffs(grids[-1][0], ab)
        P[t0:t0 + q.tokens] = a * P[t0:t0 + q.tokens] + b * E[t0:t0 + q.tokens]
        g0 += q.frames
        t0 += q.tokens
    den = denoiser or denoise
    for i in range(int(max(wl.nsteps))):
        live = [r for r in range(wl.R) if i < wl.nsteps[r]]
        rows = np.concatenate([np.arange(seg[r], seg[r + 1]) for r in live])
        tau = np.array([grids[r][i] for r in range(wl.R)])[info.req[rows]]
        sub = np.concatenate([[0], np.cumsum([seg[r + 1] - seg[r] for r in live])])
        eps_hat = den(model, P[rows], info.f[rows], info.y[rows], info.x[rows], tau, sub, precision)
        c = np.array([ddim_coeffs(grids[r][i], grids[r][i + 1], ab) if i < wl.nsteps[r] else (1.0, 0.0)
                      for r in range(wl.R)])
        c1, c2 = c[info.req[rows], 0][:, None], c[info.req[rows], 1][:, None]
        P[rows] = c1 * P[rows] + c2 * eps_hat
    return unpatchify(P, wl.requests)
