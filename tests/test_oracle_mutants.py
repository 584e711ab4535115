"""Plant plausible mistakes in the CPU oracle and check that the pins catch
each one.  The mistakes are planted only here, on the CPU, in a monkeypatched
copy of the oracle's functions; the product path is not involved."""
import numpy as np
import pytest

import oracle.sphinx_oracle as O
from pins import ALL_PINS

_orig = {name: getattr(O, name) for name in dir(O) if callable(getattr(O, name))}


def _ddim_c2_sign(t, tn, ab=None):
    c1, c2 = _orig["ddim_coeffs"](t, tn, ab)
    return c1, -c2


def _ddim_no_sqrt(t, tn, ab=None):
    a, an = O.abar_at(t, ab), O.abar_at(tn, ab)
    return an / a, _orig["ddim_coeffs"](t, tn, ab)[1]


def _inject_swapped(t, ab=None):
    a, b = _orig["injection_coeffs"](t, ab)
    return b, a


def _grid_no_end(s, n):
    return [((n - i) * (s + 1)) // n for i in range(n + 1)]


def _grid_span_s(s, n):
    return [((n - i) * s) // n - 1 for i in range(n + 1)]


def _alpha_bar_off(*_):
    i = np.arange(1000, dtype=np.float64)
    return np.cumprod(1.0 - (1e-4 + (2e-2 - 1e-4) * i / 1000))


def _attention_no_scale(q, k, v, heads, seg, chunk=2048, kv_seg=None, scale=None):
    return _orig["attention"](q, k, v, heads, seg, chunk, kv_seg, 1.0)


def _attention_no_segments(q, k, v, heads, seg, chunk=2048, kv_seg=None, scale=None):
    kv = None if kv_seg is None else np.array([kv_seg[0], kv_seg[-1]])
    return _orig["attention"](q, k, v, heads, np.array([seg[0], seg[-1]]), chunk, kv, scale)


def _attention_wrong_axis(q, k, v, heads, seg, chunk=2048, kv_seg=None, scale=None):
    if kv_seg is not None:
        raise NotImplementedError
    n, D = q.shape
    d = D // heads
    sc = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.zeros((n, D))
    for r in range(len(seg) - 1):
        s0, s1 = int(seg[r]), int(seg[r + 1])
        for h in range(heads):
            c = slice(h * d, (h + 1) * d)
            s = q[s0:s1, c] @ k[s0:s1, c].T * sc
            p = np.exp(s - s.max(axis=0, keepdims=True))
            p /= p.sum(axis=0, keepdims=True)
            out[s0:s1, c] = p @ v[s0:s1, c]
    return out


def _ln_unbiased(h):
    mu = h.mean(axis=-1, keepdims=True)
    return (h - mu) / np.sqrt(h.var(axis=-1, ddof=1, keepdims=True) + O.LN_EPS)


def _gelu_erf(z):
    from scipy.special import erf
    return 0.5 * z * (1 + erf(z / np.sqrt(2)))


def _select_ge(u, thr, act, offs):
    mask = np.logical_and(act, np.asarray(u) >= np.asarray(thr))
    idx = np.flatnonzero(mask)
    return mask, idx, np.array([np.count_nonzero(mask[:o]) for o in offs]), int(idx.size)


def _select_cu_inclusive(u, thr, act, offs):
    mask, idx, cu, n = _orig["select"](u, thr, act, offs)
    return mask, idx, np.array([np.count_nonzero(mask[:o + 1]) for o in offs]), n


def _linear_transposed(x, w, b):
    w = np.asarray(w, np.float64)
    return x @ (w.reshape(w.shape[1], w.shape[0]).T if w.shape[0] != w.shape[1] else w) + b


def _round_truncate(x):
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return ((f.view(np.uint32) >> 16) << 16).astype(np.uint32).view(np.float32).astype(np.float64)


def _patchify_swapped(latent, requests):
    P = _orig["patchify"](latent, requests)
    return P.reshape(-1, 4, 2, 2).transpose(0, 1, 3, 2).reshape(-1, 16)


def _temb_swapped(tau):
    t = _orig["timestep_embedding"](tau)
    return np.concatenate([t[:, 128:], t[:, :128]], axis=1)


def _pos_x_uses_y(f, y, x, D):
    return _orig["position_embedding"](f, y, y, D)


def _token_info_yx_swapped(requests):
    ti = _orig["token_info"](requests)
    return O.TokenInfo(ti.req, ti.gframe, ti.f, ti.x, ti.y)


def _token_info_local_frames(requests):
    ti = _orig["token_info"](requests)
    return O.TokenInfo(ti.req, ti.f, ti.f, ti.y, ti.x)


def _denoise_raw_gate(model, x, f, y, xx, tau, seg, precision="model", **kw):
    w = dict(model.weights)
    D = model.D
    for l in range(model.L):
        b = w[f"b{l}.ada_b"].copy()
        b[2 * D:3 * D] -= 1.0
        b[5 * D:6 * D] -= 1.0
        w[f"b{l}.ada_b"] = b
    m = O.Model(model.D, model.heads, model.mlp, model.L, model.dtype, w)
    return _orig["denoise"](m, x, f, y, xx, tau, seg, precision, **kw)


def _plan_always_new(frames, s_start, nsteps, period=0, per_frame_grid=False):
    plans = _orig["plan_steps"](frames, s_start, nsteps, period, per_frame_grid)
    ab = O.alpha_bar()
    for p in plans:
        for g in np.flatnonzero(p.active):
            p.newly[g] = True
            p.a[g], p.b[g] = np.sqrt(ab[p.tau[g]]), np.sqrt(1 - ab[p.tau[g]])
    return plans


def _step_skips_update(wl, model, state, plan, precision="model", denoiser=None, info=None):
    res = _orig["step"](wl, model, state, plan, precision, denoiser, info)
    P = O.patchify(res.state, wl.requests)
    P[res.idx] = res.x_in
    res.state = O.unpatchify(P, wl.requests)
    return res


def _denoise_stale_entry(model, x, f, y, xx, tau, seg, precision="model", cache=None, rows=None, kv_seg=None):
    """Attends over the cache as it was before the block stored the fresh rows."""
    if cache is None:
        return _orig["denoise"](model, x, f, y, xx, tau, seg, precision)
    return _denoise_stale(model, x, f, y, xx, tau, seg, precision, cache, rows, kv_seg)


def _denoise_stale(model, x, f, y, xx, tau, seg, precision, cache, rows, kv_seg):
    before = [(k.copy(), v.copy()) for k, v in cache]
    orig_attention = O.attention
    calls = {"l": 0}

    def attention_on_old(q, k, v, heads, seg_, chunk=2048, kv_seg=None, scale=None):
        l = calls["l"]
        calls["l"] += 1
        return orig_attention(q, before[l][0], before[l][1], heads, seg_, chunk, kv_seg, scale)

    O.attention = attention_on_old
    try:
        return _orig["denoise"](model, x, f, y, xx, tau, seg, precision, cache, rows, kv_seg)
    finally:
        O.attention = orig_attention


def _plan_no_full_after_first(frames, s_start, nsteps, period=0, per_frame_grid=False):
    plans = _orig["plan_steps"](frames, s_start, nsteps, period, per_frame_grid)
    for p in plans[1:]:
        p.full[:] = False
    return plans


def _plan_context_unnoised(frames, s_start, nsteps, period=0, per_frame_grid=False):
    plans = _orig["plan_steps"](frames, s_start, nsteps, period, per_frame_grid)
    for p in plans:
        p.a_ctx[:] = 1.0
        p.b_ctx[:] = 0.0
    return plans


def _step_cached_writes_context(wl, model, state, plan, cache, precision="model", info=None):
    res = _orig["step_cached"](wl, model, state, plan, cache, precision, info)
    if res.qidx.size:
        P = O.patchify(res.state, wl.requests)
        P[res.qidx] = res.x_out
        res.state = O.unpatchify(P, wl.requests)
    return res


def _plan_full_at_odd_steps(frames, s_start, nsteps, period=0, per_frame_grid=False):
    plans = _orig["plan_steps"](frames, s_start, nsteps, period, per_frame_grid)
    for i, p in enumerate(plans):
        live = p.full | (p.tau[np.cumsum([0] + list(frames))[:-1]] >= 0)
        p.full[:] = live & (period > 0) & ((i + 1) % max(period, 1) == 0)
    return plans


def _groups_temporal_by_frame(kind, req, f, y, x):
    return _orig["attention_group_ids"]("spatial", req, f, y, x)


def _groups_spatial_no_request(kind, req, f, y, x):
    if kind == "spatial":
        return _orig["attention_group_ids"](kind, np.zeros_like(req), f, y, x)
    return _orig["attention_group_ids"](kind, req, f, y, x)


def _block_order_swapped(attn, l):
    kind = _orig["block_attention"](attn, l)
    return {"spatial": "temporal", "temporal": "spatial"}.get(kind, kind)


def _plan_grid_shared(frames, s_start, nsteps, period=0, per_frame_grid=False):
    return _orig["plan_steps"](frames, s_start, nsteps, period, False)


MUTANTS = {
    "ddim_c2_sign": ("ddim_coeffs", _ddim_c2_sign),
    "ddim_c1_no_sqrt": ("ddim_coeffs", _ddim_no_sqrt),
    "injection_swapped": ("injection_coeffs", _inject_swapped),
    "grid_no_clean_end": ("timestep_grid", _grid_no_end),
    "grid_span_off_by_one": ("timestep_grid", _grid_span_s),
    "beta_denominator_1000": ("alpha_bar", _alpha_bar_off),
    "attention_no_scale": ("attention", _attention_no_scale),
    "attention_ignores_segments": ("attention", _attention_no_segments),
    "softmax_wrong_axis": ("attention", _attention_wrong_axis),
    "layernorm_unbiased": ("layer_norm", _ln_unbiased),
    "gelu_erf": ("gelu_tanh", _gelu_erf),
    "select_ge": ("select", _select_ge),
    "cu_sel_inclusive": ("select", _select_cu_inclusive),
    "linear_transposed": ("linear", _linear_transposed),
    "bf16_truncate": ("round_bf16", _round_truncate),
    "patch_order_swapped": ("patchify", _patchify_swapped),
    "temb_sin_cos_swapped": ("timestep_embedding", _temb_swapped),
    "pos_x_uses_y": ("position_embedding", _pos_x_uses_y),
    "token_info_yx_swapped": ("token_info", _token_info_yx_swapped),
    "token_info_frames_not_global": ("token_info", _token_info_local_frames),
    "gate_without_one": ("denoise", _denoise_raw_gate),
    "reinject_every_step": ("plan_steps", _plan_always_new),
    "scatter_without_update": ("step", _step_skips_update),
    "cache_read_before_store": ("denoise", _denoise_stale_entry),
    "cache_never_refreshed": ("plan_steps", _plan_no_full_after_first),
    "context_not_noised": ("plan_steps", _plan_context_unnoised),
    "context_written_back": ("step_cached", _step_cached_writes_context),
    "full_step_misplaced": ("plan_steps", _plan_full_at_odd_steps),
    "temporal_groups_by_frame": ("attention_group_ids", _groups_temporal_by_frame),
    "spatial_groups_ignore_request": ("attention_group_ids", _groups_spatial_no_request),
    "factorised_order_swapped": ("block_attention", _block_order_swapped),
    "per_frame_grid_ignored": ("plan_steps", _plan_grid_shared),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    attr, bad = MUTANTS[name]
    monkeypatch.setattr(O, attr, bad)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(O)
        except Exception as e:  # an assertion or a crash both expose the mistake
            caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught mutant {name}"
