"""Pins of the CPU oracle: checks against facts fixed outside the oracle.

Each ``pin_*`` takes the oracle module ``O`` (so that the mutation tests can
hand in a copy with a planted mistake) and raises ``AssertionError`` when the
oracle disagrees with:

* exact rational arithmetic (the beta / alpha_bar schedule),
* closed forms (timestep grids of a 50-step schedule, DDIM run with the true
  noise returns the clean latent, eps_hat = 0 gives z0 + sqrt((1-a)/a) eps),
* brute force on tiny inputs (attention, mask + compaction, patch layout),
* library routines for special cases (torch LayerNorm, GELU-tanh, SiLU,
  scaled-dot-product attention, float32->bfloat16 conversion, a torch
  functional rebuild of the denoiser),
* invariants of the method (empty mask is the identity, all-selected equals
  dense partial denoising, unselected tokens never influence selected ones,
  packed requests equal separate runs, per-frame start counts of Alg. 1).
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

import workloads as W

MICRO_F32 = W.ModelCfg(D=32, heads=2, head_dim=16, mlp=64, L=2, dtype="f32")
MICRO_BF16 = W.ModelCfg(D=32, heads=2, head_dim=16, mlp=64, L=2, dtype="bf16")
MICRO_FACT = W.ModelCfg(D=32, heads=2, head_dim=16, mlp=64, L=3, dtype="f32", attention="factorised")


def micro(model=MICRO_F32, requests=None, rho=None, t_start=None, nsteps=None, name="micro"):
    requests = requests or [W.Request(2, 8, 8)]
    R = len(requests)
    return W.custom(name, model, requests, rho or [0.4] * R, t_start or [0.5] * R, nsteps or [3] * R)


# ----------------------------------------------------------------------------
# schedule
# ----------------------------------------------------------------------------
def pin_alpha_bar_exact(O):
    ab = O.alpha_bar()
    assert ab.shape == (1000,)
    prod = Fraction(1)
    checkpoints = {0, 1, 2, 299, 499, 599, 699, 998, 999}
    for i in range(1000):
        beta = Fraction(1, 10 ** 4) + Fraction(199, 10 ** 4) * Fraction(i, 999)
        prod *= 1 - beta
        if i in checkpoints:
            exact = float(prod)
            assert abs(exact - ab[i]) <= 1e-12 * exact, (i, exact, ab[i])
    assert O.abar_at(-1) == 1.0


def pin_grid(O):
    full = O.timestep_grid(999, 50)  # S = 50 inference steps over 1000 timesteps
    assert full == list(range(999, 18, -20)) + [-1], full
    assert O.timestep_grid(499, 25) == list(range(499, 18, -20)) + [-1]
    assert O.timestep_grid(599, 10) == list(range(599, 58, -60)) + [-1]
    assert O.timestep_grid(499, 1) == [499, -1]
    for k in range(5, 50, 5):  # refinement starting at step k of 50 runs the tail of the full grid
        assert O.timestep_grid(999 - 20 * k, 50 - k) == full[k:], k
    for s, n in [(3, 3), (17, 5), (998, 7), (0, 1)]:
        g = O.timestep_grid(s, n)
        assert g[0] == s and g[-1] == -1 and len(g) == n + 1
        assert all(a > b for a, b in zip(g, g[1:]))


def _true_noise_denoiser(O, wl):
    """A denoiser that returns exactly the noise injected into each token."""
    info = O.token_info(wl.requests)
    E = O.patchify(wl.eps, wl.requests)
    lookup = {(int(info.req[t]), int(info.f[t]), int(info.y[t]), int(info.x[t])): t for t in range(wl.N)}

    def den(model, x, f, y, xx, tau, seg, precision):
        rows = np.arange(x.shape[0])
        req = np.searchsorted(np.asarray(seg), rows, side="right") - 1
        t = np.array([lookup[(int(req[j]), int(f[j]), int(y[j]), int(xx[j]))] for j in rows])
        return E[t]

    return den


def pin_ddim_true_noise(O, wl=None):
    """DDIM (eta = 0) fed the true injected noise recovers z0 exactly, and after
    every step a refined token sits on the forward-process line
    sqrt(abar_next) z0 + sqrt(1 - abar_next) eps.  Checked with one start step
    for all frames and with per-frame start steps (frames joining late)."""
    cases = [wl] if wl is not None else [
        micro(nsteps=[4]),
        micro(requests=[W.Request(5, 4, 4), W.Request(2, 4, 8)], t_start=[("uniform", 0.2, 0.8), 0.4],
              nsteps=[6, 3], rho=[0.5, 0.3])]
    ab = O.alpha_bar()
    for wl in cases:
        den = _true_noise_denoiser(O, wl)
        final, trace = O.refine(wl, precision="fp64", denoiser=den, trace=True)
        assert np.abs(final - wl.z0).max() < 1e-9, np.abs(final - wl.z0).max()
        Z, E = O.patchify(wl.z0, wl.requests), O.patchify(wl.eps, wl.requests)
        info = O.token_info(wl.requests)
        smax = [int(wl.s_start[wl.frame_offset[q]:wl.frame_offset[q + 1]].max()) for q in range(wl.R)]
        for i, res in enumerate(trace):
            if res.n_sel == 0:
                continue
            tn = np.array([O.timestep_grid(smax[q], int(wl.nsteps[q]))[i + 1] for q in info.req[res.idx]])
            an = np.where(tn < 0, 1.0, ab[np.maximum(tn, 0)])[:, None]
            expect = np.sqrt(an) * Z[res.idx] + np.sqrt(1 - an) * E[res.idx]
            assert np.abs(res.x_out - expect).max() < 1e-9, i


def pin_ddim_zero_noise(O, wl=None):
    """With eps_hat = 0 every DDIM step multiplies by sqrt(abar'/abar); over the
    whole grid the product is 1/sqrt(abar_s), so a token injected at s ends at
    z0 + sqrt((1-abar_s)/abar_s) eps."""
    wl = wl or micro(nsteps=[5], t_start=[0.6])
    ab = O.alpha_bar()
    zero = lambda model, x, *a: np.zeros_like(x)
    final, trace = O.refine(wl, precision="fp64", denoiser=zero, trace=True)
    s = int(wl.s_start[0])
    idx = trace[0].idx
    Z, E = O.patchify(wl.z0, wl.requests), O.patchify(wl.eps, wl.requests)
    expect = Z[idx] + math.sqrt((1 - ab[s]) / ab[s]) * E[idx]
    got = O.patchify(final, wl.requests)[idx]
    assert np.abs(got - expect).max() < 1e-9


def pin_alg1_active_counts(O):
    """Alg. 1: frame f joins at the first step with tau_i <= s_f, is injected
    exactly once, and then takes part in every remaining step."""
    s_start = np.array([499, 300, 150, 0, 480], dtype=np.int32)
    plans = O.plan_steps([5], s_start, [25])
    grid = O.timestep_grid(499, 25)
    for f, s in enumerate(s_start):
        act = [p.active[f] for p in plans]
        new = [p.newly[f] for p in plans]
        n_expect = sum(1 for t in grid[:-1] if t <= s)
        assert sum(act) == n_expect, (f, sum(act), n_expect)
        assert sum(new) == (1 if n_expect else 0)
        if n_expect:
            first = act.index(True)
            assert all(act[first:]) and new[first]
            assert abs(plans[first].a[f] - math.sqrt(O.abar_at(grid[first]))) < 1e-15


# ----------------------------------------------------------------------------
# geometry, mask and compaction
# ----------------------------------------------------------------------------
def pin_patch_layout(O):
    reqs = [W.Request(2, 4, 6), W.Request(1, 2, 4)]
    n = sum(r.frames * 4 * r.h * r.w for r in reqs)
    lat = np.arange(n, dtype=np.float64)
    P = O.patchify(lat, reqs)
    t0 = e0 = 0
    for q in reqs:
        hp, wp = q.h // 2, q.w // 2
        for f in range(q.frames):
            for c in range(4):
                for yy in range(q.h):
                    for xx in range(q.w):
                        e = e0 + ((f * 4 + c) * q.h + yy) * q.w + xx
                        t = t0 + f * hp * wp + (yy // 2) * wp + xx // 2
                        assert P[t, c * 4 + (yy % 2) * 2 + xx % 2] == lat[e]
        t0 += q.frames * hp * wp
        e0 += q.frames * 4 * q.h * q.w
    assert np.array_equal(O.unpatchify(P, reqs), lat)


def pin_token_coordinates(O):
    """token_info against the token layout written out by loops (token t of a
    request = f (h/2)(w/2) + y (w/2) + x, requests concatenated, frames
    numbered globally), and against the NCHW element each token covers: the
    patch of token (f, y, x) holds latent rows 2y, 2y+1 and columns 2x, 2x+1
    of frame f.  Non-square latents (h != w) so that a y/x mix-up shows."""
    reqs = [W.Request(3, 4, 10), W.Request(2, 6, 2), W.Request(1, 8, 12)]
    info = O.token_info(reqs)
    t = g0 = 0
    for r, q in enumerate(reqs):
        hp, wp = q.h // 2, q.w // 2
        for f in range(q.frames):
            for y in range(hp):
                for x in range(wp):
                    assert (info.req[t], info.gframe[t], info.f[t], info.y[t], info.x[t]) == (r, g0 + f, f, y, x), t
                    t += 1
        g0 += q.frames
    assert t == len(info.req)
    # coordinates carried by the latent itself: each element holds its own
    # frame, row and column; the patch of every token must hold its own (f, y, x)
    n = sum(q.frames * 4 * q.h * q.w for q in reqs)
    lf, ly, lx = (np.zeros(n) for _ in range(3))
    e = 0
    for q in reqs:
        for f in range(q.frames):
            for c in range(4):
                for yy in range(q.h):
                    for xx in range(q.w):
                        lf[e], ly[e], lx[e] = f, yy // 2, xx // 2
                        e += 1
    for lat, want in ((lf, info.f), (ly, info.y), (lx, info.x)):
        P = O.patchify(lat, reqs)
        assert np.array_equal(P, np.repeat(want[:, None], 16, axis=1).astype(np.float64))


def brute_select(u, thr, active, tok_offset):
    mask = [bool(a) and (float(x) > float(t)) for x, t, a in zip(u, thr, active)]
    idx = [t for t, m in enumerate(mask) if m]
    cu = [sum(mask[:o]) for o in tok_offset]
    return mask, idx, cu


def pin_select_bruteforce(O, seed=7):
    rng = np.random.default_rng(seed)
    for n in [1, 5, 64, 257]:
        u = rng.choice(np.array([0.0, 0.25, 0.5, 0.75, 1.0, np.nan, np.inf, -np.inf], np.float32), n)
        thr = rng.choice(np.array([0.25, 0.5, -np.inf, np.inf], np.float32), n)
        act = rng.random(n) < 0.7
        offs = np.array(sorted({0, n // 3, n // 2}), dtype=np.int64)
        mask, idx, cu, k = O.select(u, thr, act, offs)
        bm, bi, bc = brute_select(u, thr, act, offs)
        assert list(map(bool, mask)) == bm
        assert list(map(int, idx)) == bi
        assert list(map(int, cu)) == bc
        assert k == len(bi)


def pin_select_threshold_count(O):
    """Without ties, the rho rule's threshold selects exactly floor(rho n + 0.5)."""
    rng = np.random.default_rng(3)
    u = rng.permutation(np.arange(1000, dtype=np.float32))
    for rho in [0.0, 0.1, 0.3, 0.5, 0.999, 1.0]:
        thr = W.rho_threshold(u, rho)
        _, _, _, k = O.select(u, np.full(u.size, thr), np.ones(u.size, bool), np.array([0]))
        assert k == int(math.floor(rho * 1000 + 0.5)), (rho, k)


# ----------------------------------------------------------------------------
# layers against library routines
# ----------------------------------------------------------------------------
def pin_round_bf16(O):
    import torch

    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(4000).astype(np.float32) * 10,
                        np.float32([0.0, -0.0, 1.0, np.inf, -np.inf, 1e-30, 3e38])])
    # exact ties: low 16 bits 0x8000 with even and odd kept bit
    ties = (np.arange(1, 200, dtype=np.uint32) << 16 | 0x8000) + (0x3F80 << 16)
    x = np.concatenate([x, ties.view(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(x.astype(np.float64))
    assert np.array_equal(got, ref)
    assert np.isnan(O.round_bf16(np.array([np.nan])))[0]


def pin_layer_norm(O):
    import torch
    import torch.nn.functional as F

    x = np.random.default_rng(1).standard_normal((7, 48)) * 3 + 1
    ref = F.layer_norm(torch.from_numpy(x), (48,), eps=1e-6).numpy()
    assert np.abs(O.layer_norm(x) - ref).max() < 1e-12


def pin_activations(O):
    import torch
    import torch.nn.functional as F

    z = np.linspace(-8, 8, 1001)
    t = torch.from_numpy(z)
    assert np.abs(O.gelu_tanh(z) - F.gelu(t, approximate="tanh").numpy()).max() < 1e-13
    assert np.abs(O.silu(z) - F.silu(t).numpy()).max() < 1e-13


def pin_linear(O):
    import torch
    import torch.nn.functional as F

    rng = np.random.default_rng(2)
    x, w, b = rng.standard_normal((5, 7)), rng.standard_normal((3, 7)), rng.standard_normal(3)
    ref = F.linear(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b)).numpy()
    assert np.abs(O.linear(x, w, b) - ref).max() < 1e-12


def pin_embeddings(O):
    """Sinusoid tables against complex exponentials (cos + i sin)."""
    tau = np.array([0, 1, 19, 499, 999])
    te = O.timestep_embedding(tau)
    w = np.exp(-np.log(1e4) * np.arange(128) / 128)
    z = np.exp(1j * tau[:, None] * w[None, :])
    assert np.abs(te[:, :128] - z.real).max() < 1e-12 and np.abs(te[:, 128:] - z.imag).max() < 1e-12
    assert np.array_equal(te[0], np.r_[np.ones(128), np.zeros(128)])
    D = 64
    f, y, x = np.array([0, 3, 0]), np.array([0, 0, 5]), np.array([0, 2, 7])
    pe = O.position_embedding(f, y, x, D)
    q = D // 4
    nu = np.exp(-np.log(1e4) * np.arange(q) / q)
    mu = np.exp(-np.log(1e4) * np.arange(D // 2) / (D // 2))
    zy, zx, zf = np.exp(1j * y[:, None] * nu), np.exp(1j * x[:, None] * nu), np.exp(1j * f[:, None] * mu)
    ref = np.concatenate([zy.imag, zy.real, zx.imag, zx.real], 1) + np.concatenate([zf.imag, zf.real], 1)
    assert np.abs(pe - ref).max() < 1e-12
    assert np.array_equal(pe[0], np.tile(np.r_[np.zeros(q), np.ones(q)], 2) + np.r_[np.zeros(D // 2), np.ones(D // 2)])


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------
def brute_attention(q, k, v, heads, seg):
    n, D = q.shape
    d = D // heads
    out = np.zeros((n, D))
    for r in range(len(seg) - 1):
        rows = range(int(seg[r]), int(seg[r + 1]))
        for h in range(heads):
            for i in rows:
                s = [sum(q[i, h * d + c] * k[j, h * d + c] for c in range(d)) / math.sqrt(d) for j in rows]
                m = max(s)
                e = [math.exp(x - m) for x in s]
                tot = sum(e)
                for c in range(d):
                    out[i, h * d + c] = sum(e[jj] * v[j, h * d + c] for jj, j in enumerate(rows)) / tot
    return out


def pin_attention_bruteforce(O):
    rng = np.random.default_rng(11)
    for n, heads, d, seg in [(9, 2, 3, [0, 4, 9]), (12, 3, 4, [0, 1, 1, 12]), (6, 1, 5, [0, 6])]:
        q, k, v = (rng.standard_normal((n, heads * d)) * 2 for _ in range(3))
        got = O.attention(q, k, v, heads, np.array(seg))
        assert np.abs(got - brute_attention(q, k, v, heads, seg)).max() < 1e-12


def pin_attention_sdpa(O):
    import torch
    import torch.nn.functional as F

    rng = np.random.default_rng(12)
    n, heads, d = 150, 4, 16
    seg = np.array([0, 40, 41, 150])
    q, k, v = (rng.standard_normal((n, heads * d)) for _ in range(3))
    allowed = np.zeros((n, n), bool)
    for r in range(len(seg) - 1):
        allowed[seg[r]:seg[r + 1], seg[r]:seg[r + 1]] = True
    T = lambda a: torch.from_numpy(a).reshape(n, heads, d).transpose(0, 1).contiguous()
    ref = F.scaled_dot_product_attention(T(q), T(k), T(v), attn_mask=torch.from_numpy(allowed))
    ref = ref.transpose(0, 1).reshape(n, heads * d).numpy()
    assert np.abs(O.attention(q, k, v, heads, seg, chunk=64) - ref).max() < 1e-12


def pin_attention_special(O):
    rng = np.random.default_rng(13)
    n, H, d = 20, 2, 8
    q, k, v = (rng.standard_normal((n, H * d)) for _ in range(3))
    seg = np.array([0, 1, 20])
    o = O.attention(q, k, v, H, seg)
    assert np.abs(o[0] - v[0]).max() < 1e-14  # a one-token segment returns its own value
    o0 = O.attention(np.zeros_like(q), k, v, H, seg)
    assert np.abs(o0[1:] - v[1:].mean(axis=0)).max() < 1e-13  # q = 0: uniform weights
    perm = np.r_[0, 1 + rng.permutation(19)]
    op = O.attention(q[perm], k[perm], v[perm], H, seg)
    assert np.abs(op - o[perm]).max() < 1e-12  # permutation equivariance inside a segment


# ----------------------------------------------------------------------------
# the denoiser against a torch functional rebuild
# ----------------------------------------------------------------------------
def torch_denoiser(O, model, x, f, y, xx, tau, seg, precision, attention="joint"):
    import torch
    import torch.nn.functional as F

    t = lambda a: torch.as_tensor(np.asarray(a, np.float64))
    wt = {k: t(v) for k, v in model.weights.items()}
    D, H = model.D, model.heads
    d = D // H
    n = x.shape[0]
    bf = precision == "model" and model.dtype == "bf16"
    rnd = (lambda a: a.to(torch.float32).to(torch.bfloat16).to(torch.float64)) if bf else (lambda a: a)
    ln = lambda a: F.layer_norm(a, (D,), eps=1e-6)
    c = F.silu(F.linear(F.silu(F.linear(t(O.timestep_embedding(tau)), wt["t1_w"], wt["t1_b"])), wt["t2_w"], wt["t2_b"]))
    h = F.linear(t(x), wt["pe_w"], wt["pe_b"]) + t(O.position_embedding(f, y, xx, D))
    allowed = torch.zeros((n, n), dtype=torch.bool)
    for r in range(len(seg) - 1):
        allowed[seg[r]:seg[r + 1], seg[r]:seg[r + 1]] = True
    f_, y_, x_ = (torch.as_tensor(np.asarray(a)) for a in (f, y, xx))
    same_frame = allowed & (f_[:, None] == f_[None, :])
    same_column = allowed & (y_[:, None] == y_[None, :]) & (x_[:, None] == x_[None, :])
    for l in range(model.L):
        mask = allowed if attention == "joint" else (same_frame if l % 2 == 0 else same_column)
        mod = F.linear(c, wt[f"b{l}.ada_w"], wt[f"b{l}.ada_b"]).chunk(6, dim=1)
        a = rnd(ln(h) * (1 + mod[1]) + mod[0])
        q, k, v = F.linear(a, wt[f"b{l}.qkv_w"], wt[f"b{l}.qkv_b"]).chunk(3, dim=1)
        # the model stores q already multiplied by log2(e)/sqrt(d) (rounded after
        # the scale) and runs the softmax in base 2: scale ln(2) on q' k^T
        q, k, v = rnd(q * (math.log2(math.e) / math.sqrt(d))), rnd(k), rnd(v)
        heads = lambda z: z.reshape(n, H, d).transpose(0, 1)
        o = F.scaled_dot_product_attention(heads(q), heads(k), heads(v), attn_mask=mask, scale=math.log(2.0))
        o = rnd(o.transpose(0, 1).reshape(n, D))
        h = h + (1 + mod[2]) * F.linear(o, wt[f"b{l}.o_w"], wt[f"b{l}.o_b"])
        a2 = rnd(ln(h) * (1 + mod[4]) + mod[3])
        m = rnd(F.gelu(F.linear(a2, wt[f"b{l}.fc1_w"], wt[f"b{l}.fc1_b"]), approximate="tanh"))
        h = h + (1 + mod[5]) * F.linear(m, wt[f"b{l}.fc2_w"], wt[f"b{l}.fc2_b"])
    sh, sc = F.linear(c, wt["fada_w"], wt["fada_b"]).chunk(2, dim=1)
    return F.linear(ln(h) * (1 + sc) + sh, wt["out_w"], wt["out_b"]).numpy()


def pin_denoiser_torch(O):
    for cfg in (MICRO_F32, MICRO_BF16):
        wl = micro(model=cfg, requests=[W.Request(2, 8, 8), W.Request(1, 4, 8)], rho=[0.5, 0.6])
        model = O.model_from_workload(wl)
        info = O.token_info(wl.requests)
        rng = np.random.default_rng(4)
        idx = np.sort(rng.choice(wl.N, 30, replace=False))
        seg = np.array([0, int((idx < wl.tok_offset[1]).sum()), 30])
        x = O.patchify(wl.z0, wl.requests)[idx]
        tau = np.where(info.req[idx] == 0, 479, 139)
        for precision in ("fp64", "model"):
            got = O.denoise(model, x, info.f[idx], info.y[idx], info.x[idx], tau, seg, precision)
            ref = torch_denoiser(O, model, x, info.f[idx], info.y[idx], info.x[idx], tau, seg, precision)
            tol = 1e-11 if precision == "fp64" or cfg.dtype == "f32" else 1e-6
            assert np.abs(got - ref).max() < tol, (cfg.dtype, precision, np.abs(got - ref).max())


# ----------------------------------------------------------------------------
# invariants of the whole step
# ----------------------------------------------------------------------------
def pin_empty_mask_identity(O):
    wl = micro(model=MICRO_BF16)
    wl.thr[:] = np.inf
    out = O.refine(wl)
    assert np.array_equal(out, wl.z0.astype(np.float64))


def pin_all_selected_dense(O):
    wl = micro(model=MICRO_F32, requests=[W.Request(2, 8, 8), W.Request(3, 4, 4)], nsteps=[3, 2],
               t_start=[0.5, 0.3])
    wl.thr[:] = -np.inf
    for precision in ("fp64", "model"):
        sparse = O.refine(wl, precision=precision)
        dense = O.refine_dense(wl, precision=precision)
        assert np.abs(sparse - dense).max() < 1e-11, np.abs(sparse - dense).max()


def pin_unselected_independence(O):
    wl = micro(model=MICRO_F32, nsteps=[2])
    base, tr = O.refine(wl, precision="fp64", trace=True)
    sel = tr[0].mask
    P = O.patchify(wl.z0, wl.requests)
    P[~sel] += 5.0
    wl.z0 = O.unpatchify(P, wl.requests).astype(np.float32)
    moved = O.refine(wl, precision="fp64")
    B, M = O.patchify(base, wl.requests), O.patchify(moved, wl.requests)
    assert np.array_equal(B[sel], M[sel])
    assert np.array_equal(M[~sel], P[~sel].astype(np.float32).astype(np.float64))


def pin_packed_equals_separate(O):
    reqs = [W.Request(2, 8, 8), W.Request(1, 8, 4)]
    both = micro(model=MICRO_F32, requests=reqs, rho=[0.4, 0.7], t_start=[0.5, 0.7], nsteps=[3, 2])
    out = O.refine(both, precision="fp64")
    for r in range(2):
        one = micro(model=MICRO_F32, requests=[reqs[r]], nsteps=[int(both.nsteps[r])])
        e0, e1 = 16 * both.tok_offset[r], 16 * both.tok_offset[r + 1]
        f0, f1 = both.frame_offset[r], both.frame_offset[r + 1]
        one.z0, one.eps = both.z0[e0:e1].copy(), both.eps[e0:e1].copy()
        one.u = both.u[both.tok_offset[r]:both.tok_offset[r + 1]].copy()
        one.thr, one.s_start = both.thr[f0:f1].copy(), both.s_start[f0:f1].copy()
        one.weights = both.weights
        sep = O.refine(one, precision="fp64")
        assert np.abs(sep - out[e0:e1]).max() < 1e-12, r


# ----------------------------------------------------------------------------
# latent cache (Sec. 5.2): full steps every T steps, partial steps through the cache
# ----------------------------------------------------------------------------
MICRO_F32_1BLOCK = W.ModelCfg(D=32, heads=2, head_dim=16, mlp=64, L=1, dtype="f32")


def _abar_direct(t):
    """alpha_bar(t) as the plain product of (1 - beta_i), beta linear 1e-4..2e-2 over 1000 steps."""
    if t < 0:
        return 1.0
    i = np.arange(t + 1, dtype=np.float64)
    return float(np.prod(1.0 - (1e-4 + (2e-2 - 1e-4) * i / 999.0)))


def pin_cache_all_selected_dense(O):
    """Every token selected: each step forwards (and re-stores) every token,
    so the cache holds this step's keys and values and the loop equals dense
    partial denoising whatever the period."""
    wl = micro(model=MICRO_F32, requests=[W.Request(2, 8, 8), W.Request(1, 4, 8)], nsteps=[3, 2],
               t_start=[0.5, 0.3])
    wl.thr[:] = -np.inf
    dense = O.refine_dense(wl, precision="fp64")
    for period in (1, 2, 5):
        got = O.refine(wl, precision="fp64", period=period)
        assert np.abs(got - dense).max() < 1e-11, (period, np.abs(got - dense).max())


def pin_cache_full_every_step(O):
    """Period 1: every step is a full step.  Rebuilt here without a cache: all
    tokens of the request go through the plain denoiser, selected ones from the
    state (noised on the first step), the others as their clean latent noised
    to the step's level, and only the selected tokens are written back."""
    for cfg in (MICRO_F32, MICRO_FACT):
        _cache_full_every_step(O, micro(model=cfg, nsteps=[3], rho=[0.35]))


def _cache_full_every_step(O, wl):
    got = O.refine(wl, precision="fp64", period=1)
    model = O.model_from_workload(wl)
    info = O.token_info(wl.requests)
    s = int(wl.s_start[0])
    n = int(wl.nsteps[0])
    grid = [((n - i) * (s + 1)) // n - 1 for i in range(n + 1)]
    Z0 = O.patchify(wl.z0, wl.requests)
    E = O.patchify(wl.eps, wl.requests)
    sel = np.asarray(wl.u) > np.repeat(wl.thr, wl.N // len(wl.thr))
    P = Z0.astype(np.float64).copy()
    for i in range(n):
        t, tn = grid[i], grid[i + 1]
        ab, abn = _abar_direct(t), _abar_direct(tn)
        noised = math.sqrt(ab) * Z0 + math.sqrt(1 - ab) * E
        x = np.where(sel[:, None], P if i > 0 else noised, noised)
        eps_hat = O.denoise(model, x, info.f, info.y, info.x, np.full(wl.N, t), np.array([0, wl.N]), "fp64")
        c1 = math.sqrt(abn / ab)
        c2 = math.sqrt(1 - abn) - math.sqrt(abn * (1 - ab) / ab)
        P[sel] = (c1 * x + c2 * eps_hat)[sel]
    ref = O.unpatchify(P, wl.requests)
    assert np.abs(got - ref).max() < 1e-11, np.abs(got - ref).max()
    assert np.array_equal(O.patchify(got, wl.requests)[~sel], Z0[~sel].astype(np.float64))


def pin_cache_partial_one_block(O):
    """One block, period 2, two steps: step 0 is full, step 1 partial.  In a
    one-block denoiser a token's key and value depend only on its own input and
    timestep, so the partial step equals the plain denoiser over the selected
    tokens at step 1 together with every other token as it entered step 0
    (clean latent noised to tau_0, timestep tau_0)."""
    wl = micro(model=MICRO_F32_1BLOCK, nsteps=[2], rho=[0.3])
    got = O.refine(wl, precision="fp64", period=2)
    model = O.model_from_workload(wl)
    info = O.token_info(wl.requests)
    s, n = int(wl.s_start[0]), 2
    t0, t1, t2 = [((n - i) * (s + 1)) // n - 1 for i in range(n + 1)]
    Z0 = O.patchify(wl.z0, wl.requests).astype(np.float64)
    E = O.patchify(wl.eps, wl.requests)
    sel = np.asarray(wl.u) > np.repeat(wl.thr, wl.N // len(wl.thr))
    a0, a1, a2 = _abar_direct(t0), _abar_direct(t1), _abar_direct(t2)
    ctx = math.sqrt(a0) * Z0 + math.sqrt(1 - a0) * E
    # step 0 (full): every token at tau_0; the selected ones are updated
    e0 = O.denoise(model, ctx, info.f, info.y, info.x, np.full(wl.N, t0), np.array([0, wl.N]), "fp64")
    x1 = math.sqrt(a1 / a0) * ctx + (math.sqrt(1 - a1) - math.sqrt(a1 * (1 - a0) / a0)) * e0
    # step 1 (partial): selected at tau_1 with their updated values, the rest frozen at step 0's input
    x = np.where(sel[:, None], x1, ctx)
    tau = np.where(sel, t1, t0)
    e1 = O.denoise(model, x, info.f, info.y, info.x, tau, np.array([0, wl.N]), "fp64")
    out = Z0.copy()
    out[sel] = (math.sqrt(a2 / a1) * x + (math.sqrt(1 - a2) - math.sqrt(a2 * (1 - a1) / a1)) * e1)[sel]
    ref = O.unpatchify(out, wl.requests)
    assert np.abs(got - ref).max() < 1e-11, np.abs(got - ref).max()


def pin_cache_context_matters(O):
    """With the cache, unselected tokens reach the selected ones through
    attention (without it they cannot): moving the clean latent of unselected
    tokens moves the selected outputs, and only those."""
    wl = micro(model=MICRO_F32, nsteps=[3])
    base, tr = O.refine(wl, precision="fp64", trace=True, period=2)
    sel = tr[0].mask
    P = O.patchify(wl.z0, wl.requests)
    P[~sel] += 1.0
    wl.z0 = O.unpatchify(P, wl.requests).astype(np.float32)
    moved = O.refine(wl, precision="fp64", period=2)
    B, M = O.patchify(base, wl.requests), O.patchify(moved, wl.requests)
    assert np.abs(B[sel] - M[sel]).max() > 1e-6
    assert np.array_equal(M[~sel], P[~sel].astype(np.float32).astype(np.float64))


# ----------------------------------------------------------------------------
# factorised spatial / temporal attention and the per-frame grid reading
# ----------------------------------------------------------------------------
def pin_attention_groups_bruteforce(O):
    rng = np.random.default_rng(14)
    n, H, d = 13, 2, 3
    q, k, v = (rng.standard_normal((n, H * d)) for _ in range(3))
    g = rng.integers(0, 4, n)
    got = O.attention_groups(q, k, v, H, g, g)
    for i in range(n):
        js = [j for j in range(n) if g[j] == g[i]]
        for h in range(H):
            c = slice(h * d, (h + 1) * d)
            s = [float(q[i, c] @ k[j, c]) / math.sqrt(d) for j in js]
            e = [math.exp(a - max(s)) for a in s]
            ref = sum(w * v[j, c] for w, j in zip(e, js)) / sum(e)
            assert np.abs(got[i, c] - ref).max() < 1e-12


def pin_factorised_torch(O):
    """A factorised denoiser (even blocks: same frame; odd blocks: same (y, x))
    against the torch rebuild with explicit boolean masks."""
    wl = micro(model=MICRO_FACT, requests=[W.Request(3, 8, 8), W.Request(2, 4, 8)], rho=[0.5, 0.6])
    model = O.model_from_workload(wl)
    assert model.attention == "factorised"
    info = O.token_info(wl.requests)
    rng = np.random.default_rng(5)
    idx = np.sort(rng.choice(wl.N, 40, replace=False))
    n0 = int((idx < wl.tok_offset[1]).sum())
    seg = np.array([0, n0, 40])
    x = O.patchify(wl.z0, wl.requests)[idx]
    tau = np.where(info.req[idx] == 0, 479, 139)
    got = O.denoise(model, x, info.f[idx], info.y[idx], info.x[idx], tau, seg, "fp64")
    ref = torch_denoiser(O, model, x, info.f[idx], info.y[idx], info.x[idx], tau, seg, "fp64", "factorised")
    assert np.abs(got - ref).max() < 1e-11, np.abs(got - ref).max()


def pin_factorised_special(O):
    """One frame: a spatial block is the joint block; a temporal block is a
    one-token segment per position, which returns the token's own value."""
    one_block = W.ModelCfg(D=32, heads=2, head_dim=16, mlp=64, L=1, dtype="f32", attention="factorised")
    joint = W.ModelCfg(D=32, heads=2, head_dim=16, mlp=64, L=1, dtype="f32")
    wl = micro(model=one_block, requests=[W.Request(1, 8, 8)])
    wj = micro(model=joint, requests=[W.Request(1, 8, 8)])
    info = O.token_info(wl.requests)
    x = O.patchify(wl.z0, wl.requests)
    tau = np.full(wl.N, 300)
    seg = np.array([0, wl.N])
    a = O.denoise(O.model_from_workload(wl), x, info.f, info.y, info.x, tau, seg, "fp64")
    b = O.denoise(O.model_from_workload(wj), x, info.f, info.y, info.x, tau, seg, "fp64")
    assert np.abs(a - b).max() < 1e-13
    rng = np.random.default_rng(15)
    q, k, v = (rng.standard_normal((wl.N, 32)) for _ in range(3))
    grp = O.attention_group_ids("temporal", np.zeros(wl.N, int), info.f, info.y, info.x)
    assert len(np.unique(grp)) == wl.N
    assert np.abs(O.attention_groups(q, k, v, 2, grp, grp) - v).max() < 1e-14


def pin_per_frame_grid(O):
    """The per-frame-grid reading: every frame walks its own grid from its own
    start, is injected once at its start, and with the true injected noise
    returns z0."""
    wl = micro(requests=[W.Request(4, 4, 4)], t_start=[("uniform", 0.2, 0.8)], nsteps=[5], rho=[0.6])
    plans = O.plan_steps([4], wl.s_start, wl.nsteps, per_frame_grid=True)
    for f in range(4):
        own = [((5 - i) * (int(wl.s_start[f]) + 1)) // 5 - 1 for i in range(6)]
        assert [int(p.tau[f]) for p in plans] == own[:5]
        assert all(p.active[f] for p in plans) and [bool(p.newly[f]) for p in plans] == [True] + [False] * 4
        assert abs(plans[0].a[f] - math.sqrt(_abar_direct(own[0]))) < 1e-15
    den = _true_noise_denoiser(O, wl)
    final = O.refine(wl, precision="fp64", denoiser=den, per_frame_grid=True)
    assert np.abs(final - wl.z0).max() < 1e-9
    same = micro(requests=[W.Request(3, 4, 4)], nsteps=[4])
    a = O.plan_steps([3], same.s_start, same.nsteps, per_frame_grid=True)
    b = O.plan_steps([3], same.s_start, same.nsteps)
    for pa, pb in zip(a, b):  # one start for all frames: the two readings agree
        for fld in ("active", "newly", "tau", "a", "b", "c1", "c2"):
            assert np.array_equal(getattr(pa, fld), getattr(pb, fld)), fld


ALL_PINS = [pin_alpha_bar_exact, pin_grid, pin_ddim_true_noise, pin_ddim_zero_noise, pin_alg1_active_counts,
            pin_patch_layout, pin_token_coordinates, pin_select_bruteforce, pin_select_threshold_count, pin_round_bf16,
            pin_layer_norm, pin_activations, pin_linear, pin_embeddings, pin_attention_bruteforce,
            pin_attention_sdpa, pin_attention_special, pin_denoiser_torch, pin_empty_mask_identity,
            pin_all_selected_dense, pin_unselected_independence, pin_packed_equals_separate,
            pin_cache_all_selected_dense, pin_cache_full_every_step, pin_cache_partial_one_block,
            pin_cache_context_matters, pin_attention_groups_bruteforce, pin_factorised_torch,
            pin_factorised_special, pin_per_frame_grid]
