"""GPU parity of the latent cache with periodic full steps (Sec. 5.2; Alg. 1
full_step / store_temporal / partial_step with the cache) against the CPU
oracle, through the C ABI.

* end to end and teacher-forced per step (state and cache of the oracle
  loaded before each step), fp32 / bf16 head_dim 64 / bf16 head_dim 72;
* the cache contents after every step against the oracle's;
* every token selected equals dense partial denoising whatever the period;
* a reduced headline shape (14 frames, D 1024, 16 heads) one block deep, and
  the full-depth headline with the cache: deterministic, unselected tokens
  untouched.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2511_18672_amd")

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
F32_MODEL = W.ModelCfg(D=64, heads=4, head_dim=16, mlp=256, L=2, dtype="f32")
MID_BF16 = W.ModelCfg(D=128, heads=2, head_dim=64, mlp=512, L=2, dtype="bf16")
D72_BF16 = W.ModelCfg(D=1152, heads=16, head_dim=72, mlp=1152, L=1, dtype="bf16")


def _cache_view(R):
    tdt = torch.bfloat16 if R.cfg.dtype == "bf16" else torch.float32
    return R.kv_cache.view(tdt).view(R.cfg.L, R.N, 2, R.cfg.D)


def _load(R, state_nchw, cache):
    """Oracle state (NCHW) and cache into the Refiner (token-major state)."""
    P = O.patchify(state_nchw, R.shapes).astype(np.float32)
    R.z.copy_(torch.from_numpy(np.ascontiguousarray(P.ravel())).cuda())
    cv = _cache_view(R)
    for l, (K, V) in enumerate(cache):
        cv[l, :, 0].copy_(torch.from_numpy(K.astype(np.float32)).to(cv.dtype).cuda())
        cv[l, :, 1].copy_(torch.from_numpy(V.astype(np.float32)).to(cv.dtype).cuda())


def check_cached(wl, period, teacher_forced=True):
    model = O.model_from_workload(wl)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps, period)
    info = O.token_info(wl.requests)
    # free-running GPU run against the free-running oracle
    R = S.from_workload(wl, cache_period=period)
    R.reset()
    for i in range(R.total_steps):
        R.step(i)
    got = R.state.cpu().numpy().astype(np.float64)
    ref = O.refine(wl, precision="model", period=period)
    err = np.abs(got - ref).max()
    print(f"[cache {wl.name} T={period}] end-to-end {len(plans)} steps max_abs = {err:.3e}")
    assert err <= TOL[wl.model.dtype] and np.isfinite(got).all()
    if not teacher_forced:
        return
    # teacher forcing: before each step the GPU gets the oracle's state and cache
    R.reset()
    state = np.asarray(wl.z0, np.float64)
    cache = O.new_cache(model, wl.N)
    worst = worst_cache = 0.0
    for i, p in enumerate(plans):
        _load(R, state, cache)
        n = R.step(i, force_select=True)
        res = O.step_cached(wl, model, state, p, cache, "model", info)
        assert n == res.n_sel and np.array_equal(R.idx[:n].cpu().numpy(), res.idx), i
        assert R.n_fwd == res.qidx.size, i
        gs = R.state.cpu().numpy().astype(np.float64)
        worst = max(worst, np.abs(gs - res.state).max())
        cv = _cache_view(R).float().cpu().numpy()
        rows = res.qidx
        for l, (K, V) in enumerate(cache):
            worst_cache = max(worst_cache, np.abs(cv[l, rows, 0] - K[rows]).max(), np.abs(cv[l, rows, 1] - V[rows]).max())
        state = res.state
    print(f"[cache {wl.name} T={period}] teacher-forced per-step max_abs = {worst:.3e}, "
          f"stored keys/values max_abs = {worst_cache:.3e}")
    assert worst <= TOL[wl.model.dtype]
    assert worst_cache <= (1e-4 if wl.model.dtype == "f32" else 3e-2)


def test_cache_f32_end_to_end():
    wl = W.custom("cache_f32", F32_MODEL, [W.Request(3, 8, 12)], [0.35], [0.6], [5])
    check_cached(wl, 2)


@pytest.mark.parametrize("period", [1, 3])
def test_cache_bf16_ragged_staggered(period):
    wl = W.custom("cache_ragged", MID_BF16, [W.Request(3, 24, 20), W.Request(2, 10, 14), W.Request(1, 4, 4)],
                  [0.4, 0.7, 0.5], [("uniform", 0.3, 0.7), 0.5, 0.2], [6, 4, 3])
    check_cached(wl, period)


def test_cache_d72():
    wl = W.custom("cache_d72", D72_BF16, [W.Request(4, 16, 16)], [0.25], [("uniform", 0.3, 0.7)], [4])
    check_cached(wl, 2)


def test_cache_all_selected_equals_dense():
    wl = W.custom("cache_dense", MID_BF16, [W.Request(2, 16, 16), W.Request(1, 12, 8)], [1.0, 1.0], [0.5, 0.3],
                  [3, 2])
    R = S.from_workload(wl, cache_period=2)
    got = R.run().cpu().numpy().astype(np.float64)
    dense = O.refine_dense(wl, precision="model")
    err = np.abs(got - dense).max()
    print(f"[cache all-selected vs dense oracle] max_abs = {err:.3e}")
    assert err <= TOL["bf16"]


def test_cache_reduced_headline_one_block():
    """14 frames of 4x32x64 (7168 tokens, 30 % selected), D 1024, 16 heads of
    64, MLP 4096, one block: a full step over every token, then two partial
    steps of ~2150 queries against all 7168 keys through the cache."""
    model = W.ModelCfg(D=1024, heads=16, head_dim=64, mlp=4096, L=1, dtype="bf16")
    wl = W.custom("cache_headline_reduced", model, [W.Request(14, 32, 64)], [0.3], [0.5], [3])
    check_cached(wl, 3, teacher_forced=False)


def test_cache_headline_full_depth_properties():
    """12-block headline with the cache (T = 5): a full step then a partial
    step; two runs agree bit for bit and unselected tokens keep z0."""
    wl = W.headline()
    outs = []
    for _ in range(2):
        R = S.from_workload(wl, cache_period=5)
        R.reset()
        n0 = R.step(0)
        assert R.n_fwd == wl.N
        n1 = R.step(1)
        assert R.n_fwd == n1 == n0 == 9677
        outs.append(R.state.cpu().numpy())
        idx = R.idx[:n1].cpu().numpy()
        del R
        torch.cuda.empty_cache()
    assert np.array_equal(outs[0], outs[1]), "two runs differ"
    P = O.patchify(outs[0], wl.requests)
    keep = np.ones(wl.N, bool)
    keep[idx] = False
    assert np.array_equal(P[keep], O.patchify(wl.z0, wl.requests)[keep].astype(np.float32))
    assert np.isfinite(P).all()
