"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

* masks, indices and compaction: bit-exact;
* latents: max-abs error <= 1e-4 (fp32 model) / 2e-2 (bf16 model) against the
  oracle in its model precision (bf16 operands where the model stores bf16);
* full-size shapes: every kernel at the headline launch configuration against
  the oracle (one block deep), plus properties that hold at any size for the
  12-block headline and the packed four-request batch.
Each test prints the errors it measured.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from golden_states import forward_state
from pins import MICRO_BF16

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2511_18672_amd")

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
MID_BF16 = W.ModelCfg(D=128, heads=2, head_dim=64, mlp=512, L=2, dtype="bf16")


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def gpu_select(wl, active):
    N = wl.N
    reqs = S.make_requests(wl.requests)
    mask = torch.empty(N, dtype=torch.uint8, device="cuda")
    idx = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    cu = torch.empty(wl.R + 1, dtype=torch.int32, device="cuda")
    ws = torch.empty(S.sphinx_select_workspace_bytes(N), dtype=torch.uint8, device="cuda")
    act = None if active is None else _dev(np.asarray(active, np.uint8))
    cu_host = S.sphinx_select_mask(reqs, _dev(wl.u), _dev(wl.thr), act, mask, idx, cu, ws)
    n = int(cu_host[-1])
    return mask.cpu().numpy().astype(bool), idx[:n].cpu().numpy(), cu_host, cu.cpu().numpy()


def check_select(wl, active):
    info = O.token_info(wl.requests)
    act_tok = np.ones(wl.N, bool) if active is None else np.asarray(active, bool)[info.gframe]
    mask, idx, cu, n = O.select(wl.u, wl.thr[info.gframe], act_tok, wl.tok_offset[:-1])
    gm, gi, gcu, gcu_dev = gpu_select(wl, active)
    assert np.array_equal(gm, mask)
    assert np.array_equal(gi, idx)
    assert list(gcu) == list(cu) + [n]
    assert np.array_equal(gcu, gcu_dev)
    return n


@pytest.mark.parametrize("name", ["tiny", "small", "headline", "frame_region", "batched"])
def test_select_bitexact_configs(name):
    wl = W.CONFIGS[name](with_weights=False)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    seen = set()
    for p in plans:
        key = tuple(p.active)
        if key in seen:
            continue
        seen.add(key)
        n = check_select(wl, p.active.astype(np.uint8))
        print(f"[select] {name} active={int(p.active.sum())}/{wl.G} n_sel={n}")
    check_select(wl, None)


def test_select_edge_cases():
    rng = np.random.default_rng(21)
    shapes = [W.Request(3, 6, 10), W.Request(1, 2, 2), W.Request(5, 18, 6), W.Request(2, 64, 66)]
    wl = W.custom("edge", MICRO_BF16, shapes, [0.5] * 4, [0.5] * 4, [1] * 4, with_weights=False)
    specials = np.array([np.nan, np.inf, -np.inf, 0.5, 0.5, 0.25], np.float32)
    wl.u = np.where(rng.random(wl.N) < 0.2, rng.choice(specials, wl.N), wl.u).astype(np.float32)
    wl.thr = rng.choice(np.array([0.5, 0.25, -np.inf, np.inf, np.nan], np.float32), wl.G)
    for active in [None, (rng.random(wl.G) < 0.5).astype(np.uint8), np.zeros(wl.G, np.uint8)]:
        n = check_select(wl, active)
        print(f"[select] edge N={wl.N} n_sel={n}")
    # large ragged input spanning many 4096-token chunks
    big = W.custom("big", MICRO_BF16, [W.Request(37, 130, 98), W.Request(3, 10, 2)], [0.3, 0.9], [0.5, 0.5],
                   [1, 1], u_recipe="uniform", with_weights=False)
    n = check_select(big, None)
    print(f"[select] big N={big.N} n_sel={n}")


def test_select_stale_workspace_many_chunks():
    """Selection on a workspace full of stale bytes, three calls in a row on
    it: 150 chunks of 4096 tokens, a 3-chunk input, then 2301 chunks."""
    big = W.custom("lookback", MICRO_BF16, [W.Request(150, 128, 128), W.Request(2, 6, 4)], [0.3, 0.6], [0.5, 0.5],
                   [1, 1], u_recipe="uniform", with_weights=False)
    small = W.custom("lookback2", MICRO_BF16, [W.Request(9, 64, 66)], [0.5], [0.5], [1], u_recipe="uniform",
                     with_weights=False)
    huge = W.custom("lookback3", MICRO_BF16, [W.Request(3, 6, 10), W.Request(1150, 128, 128),
                                              W.Request(1150, 128, 128)], [0.5, 0.3, 0.6], [0.5] * 3, [1] * 3,
                    u_recipe="uniform", with_weights=False)
    ws = torch.full((S.sphinx_select_workspace_bytes(huge.N),), 0xAB, dtype=torch.uint8, device="cuda")
    for wl in (big, small, huge):
        info = O.token_info(wl.requests)
        mask, idx, cu, n = O.select(wl.u, wl.thr[info.gframe], np.ones(wl.N, bool), wl.tok_offset[:-1])
        gm = torch.empty(wl.N, dtype=torch.uint8, device="cuda")
        gi = torch.full((wl.N,), -7, dtype=torch.int32, device="cuda")
        gc = torch.empty(wl.R + 1, dtype=torch.int32, device="cuda")
        cu_host = S.sphinx_select_mask(S.make_requests(wl.requests), _dev(wl.u), _dev(wl.thr), None, gm, gi, gc, ws)
        assert np.array_equal(gm.cpu().numpy().astype(bool), mask)
        assert np.array_equal(gi[:n].cpu().numpy(), idx)
        assert list(cu_host) == list(cu) + [n]
        print(f"[select] stale-workspace N={wl.N} chunks={(wl.N + 4095) // 4096} n_sel={n}")


@pytest.mark.parametrize("case", ["two_scan_blocks", "ragged_requests"])
def test_select_large(case):
    """Large selections: 2^26 + 2^16 tokens (16 400 chunks of 4096 tokens, so
    the chunk-count scan runs two of its 16 384-count blocks and carries
    between them), and 21.3 M tokens in four requests (requests starting
    inside chunks, a ragged last chunk).  Per-frame thresholds and active
    flags, uniform-random u; the workspace (full of stale bytes) and the static
    entry point, both against the oracle."""
    if case == "two_scan_blocks":
        shapes = [W.Request(1025, 512, 512)]
    else:
        shapes = [W.Request(3, 6, 10), W.Request(325, 512, 512), W.Request(1, 2, 2), W.Request(3, 130, 98)]
    rng = np.random.default_rng(31)
    info = O.token_info(shapes)
    N, G = len(info.gframe), sum(r.frames for r in shapes)
    tok_off = np.concatenate([[0], np.cumsum([r.frames * (r.h // 2) * (r.w // 2) for r in shapes])])
    u = rng.random(N, dtype=np.float32)
    thr = (0.5 + 0.4 * rng.random(G)).astype(np.float32)
    active = (rng.random(G) < 0.7).astype(np.uint8)
    mask, idx, cu, n = O.select(u, thr[info.gframe], active.astype(bool)[info.gframe], tok_off[:-1])
    print(f"[select large] {case} N={N} chunks={(N + 4095) // 4096} n_sel={n}", flush=True)
    reqs = S.make_requests(shapes)
    ud, td, ad = _dev(u), _dev(thr), _dev(active)
    ws = torch.full((S.sphinx_select_workspace_bytes(N),), 0xAB, dtype=torch.uint8, device="cuda")
    for static in (False, True):
        gm = torch.empty(N, dtype=torch.uint8, device="cuda")
        gi = torch.full((N,), -7, dtype=torch.int32, device="cuda")
        gc = torch.empty(len(shapes) + 1, dtype=torch.int32, device="cuda")
        if static:
            cu_host = S.sphinx_select_mask_static(reqs, ud, td, ad, gm, gi, gc)
        else:
            cu_host = S.sphinx_select_mask(reqs, ud, td, ad, gm, gi, gc, ws)
        assert list(cu_host) == list(cu) + [n]
        assert np.array_equal(gm.cpu().numpy().astype(bool), mask)
        assert np.array_equal(gi[:n].cpu().numpy(), idx)
        assert (gi[n:] == -7).all().item()


def _in_layout(nchw, tokens_2d, layout):
    """The same latents in `layout` (tokens_2d: [N][16] in patch order)."""
    return nchw if layout == S.NCHW else np.ascontiguousarray(tokens_2d).ravel()


@pytest.mark.parametrize("layout", [S.NCHW, S.TOKENS], ids=["nchw", "tokens"])
def test_gather_scatter(layout):
    wl = W.custom("gs", MICRO_BF16, [W.Request(3, 8, 12), W.Request(2, 6, 4)], [0.5, 0.3], [0.5, 0.5], [1, 1],
                  with_weights=False)
    rng = np.random.default_rng(3)
    state = rng.standard_normal(16 * wl.N).astype(np.float32)
    a = rng.random(wl.G).astype(np.float32)
    b = (rng.random(wl.G) * (rng.random(wl.G) < 0.6)).astype(np.float32)
    _, idx, cu, _ = gpu_select(wl, None)
    n = len(idx)
    print(f"[gather_scatter] layout={layout} n={n} N={wl.N}", flush=True)
    reqs = S.make_requests(wl.requests)
    P, E = O.patchify(state, wl.requests), O.patchify(wl.eps, wl.requests)
    state_l = _in_layout(state, P.astype(np.float32), layout)
    eps_l = _in_layout(wl.eps, E.astype(np.float32), layout)
    x = torch.empty(16 * n, dtype=torch.float32, device="cuda")
    S.sphinx_gather(reqs, layout, _dev(state_l), S.F32, _dev(eps_l, torch.bfloat16), S.BF16,
                    _dev(idx.astype(np.int32)), n, _dev(a), _dev(b), x)
    info = O.token_info(wl.requests)
    Eb = torch.from_numpy(E.astype(np.float32)).to(torch.bfloat16).double().numpy()
    g = info.gframe[idx]
    ref = a[g].astype(np.float64)[:, None] * P[idx] + b[g].astype(np.float64)[:, None] * Eb[idx]
    err = np.abs(x.cpu().numpy().reshape(n, 16) - ref).max()
    print(f"[gather] n={n} max_abs={err:.3e}")
    assert err <= 1e-6 * max(1.0, np.abs(ref).max())
    # eps = NULL drops the noise term
    S.sphinx_gather(reqs, layout, _dev(state_l), S.F32, None, S.BF16, _dev(idx.astype(np.int32)), n, _dev(a),
                    _dev(b), x)
    assert np.array_equal(x.cpu().numpy().reshape(n, 16), (a[g][:, None] * P[idx].astype(np.float32)))
    # scatter in place: selected tokens replaced exactly, the rest untouched
    xs = rng.standard_normal(16 * n).astype(np.float32)
    st = _dev(state_l)
    S.sphinx_scatter_blend(reqs, _dev(xs), _dev(idx.astype(np.int32)), n, st, S.F32, layout, st, S.F32, layout)
    Pexp = P.copy()
    Pexp[idx] = xs.reshape(n, 16)
    exp_nchw = O.unpatchify(Pexp, wl.requests).astype(np.float32)
    assert np.array_equal(st.cpu().numpy(), _in_layout(exp_nchw, Pexp.astype(np.float32), layout))
    # out of place into the other layout with conversion to bf16 (round to nearest even)
    other = S.TOKENS if layout == S.NCHW else S.NCHW
    out = torch.empty(16 * wl.N, dtype=torch.bfloat16, device="cuda")
    S.sphinx_scatter_blend(reqs, _dev(xs), _dev(idx.astype(np.int32)), n, _dev(state_l), S.F32, layout, out, S.BF16,
                           other)
    expect = torch.from_numpy(_in_layout(exp_nchw, Pexp.astype(np.float32), other)).to(torch.bfloat16)
    assert torch.equal(out.cpu(), expect)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_layout_conversion_roundtrip(dt):
    """NCHW -> tokens -> NCHW with n_sel = 0 is a bit-exact permutation."""
    reqs_w = [W.Request(3, 10, 6), W.Request(1, 64, 66), W.Request(2, 2, 2)]
    reqs = S.make_requests(reqs_w)
    N = sum(r.frames * (r.h // 2) * (r.w // 2) for r in reqs_w)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    code = S.F32 if dt == "f32" else S.BF16
    z = torch.from_numpy(np.random.default_rng(5).standard_normal(16 * N).astype(np.float32)).to(tdt)
    zt = torch.empty_like(z, device="cuda")
    back = torch.empty_like(z, device="cuda")
    S.sphinx_scatter_blend(reqs, None, None, 0, z.cuda(), code, S.NCHW, zt, code, S.TOKENS)
    S.sphinx_scatter_blend(reqs, None, None, 0, zt, code, S.TOKENS, back, code, S.NCHW)
    expect_t = O.patchify(z.float().numpy(), reqs_w).astype(np.float32).ravel()
    assert np.array_equal(zt.float().cpu().numpy(), expect_t)
    assert torch.equal(back.cpu(), z)


def run_gpu(wl, trace=False, steps=None):
    R = S.from_workload(wl)
    R.reset()
    states = [R.state.cpu().numpy().astype(np.float64)] if trace else None
    sels = []
    for i in range(steps or R.total_steps):
        R.step(i)
        sels.append((R.n_sel, R.idx[:R.n_sel].cpu().numpy().copy(), R.cu_host.copy()))
        if trace:
            states.append(R.state.cpu().numpy().astype(np.float64))
    torch.cuda.synchronize()
    return R, states, sels


def _report(tag, got, ref, truth=None):
    err = np.abs(got - ref).max()
    msg = f"[{tag}] max_abs vs oracle(model precision) = {err:.3e}"
    if truth is not None:
        msg += f"; vs oracle(fp64) = {np.abs(got - truth).max():.3e}"
    print(msg)
    return err


def check_end_to_end(wl, teacher_forced=True):
    R, _, sels = run_gpu(wl)
    got = R.state.cpu().numpy().astype(np.float64)
    ref, trace = O.refine(wl, precision="model", trace=True)
    for i, (res, (n, idx, cu)) in enumerate(zip(trace, sels)):
        assert n == res.n_sel and np.array_equal(idx, res.idx), i
        assert list(cu) == list(res.cu_sel) + [res.n_sel], i
    truth = O.refine(wl, precision="fp64") if wl.model.dtype == "bf16" and wl.N <= 4096 else None
    err = _report(f"{wl.name} end-to-end {len(trace)} steps", got, ref, truth)
    assert err <= TOL[wl.model.dtype]
    assert np.isfinite(got).all()
    if teacher_forced:
        worst = teacher_forced_steps(R, wl, trace)
        print(f"[{wl.name}] teacher-forced per-step max_abs = {worst:.3e}")
        assert worst <= TOL[wl.model.dtype]
    return R


def teacher_forced_steps(R, wl, trace):
    """Every step once more from the oracle's state before it (loaded into the
    GPU state), against the oracle's state after it; returns the worst error."""
    worst = 0.0
    before = np.asarray(wl.z0, np.float64)
    R.reset()
    for i, res in enumerate(trace):
        R.load_state(before)
        n = R.step(i, force_select=True)
        assert n == res.n_sel and np.array_equal(R.idx[:n].cpu().numpy(), res.idx), i
        worst = max(worst, float(np.abs(R.state.cpu().numpy() - res.state).max()))
        before = res.state
    return worst


def test_tiny_end_to_end():
    R = check_end_to_end(W.tiny())
    f32 = R.output("f32")
    assert torch.equal(R.output("bf16"), f32.to(torch.bfloat16))
    # the NCHW state of record runs the same arithmetic: bit-identical result
    Rn = S.from_workload(W.tiny(), layout=S.NCHW)
    assert Rn.layout == S.NCHW
    Rn.run()
    assert torch.equal(Rn.state, f32)


def test_layouts_bit_identical_bf16():
    wl = W.custom("layouts", MID_BF16, [W.Request(2, 16, 12), W.Request(1, 10, 10)], [0.6, 0.4], [0.5, 0.3], [3, 2])
    Rt, Rn = S.from_workload(wl), S.from_workload(wl, layout=S.NCHW)
    assert torch.equal(Rt.run(), Rn.run())


def test_small_end_to_end():
    check_end_to_end(W.small())


def test_multi_request_ragged_staggered():
    wl = W.custom("ragged", MID_BF16, [W.Request(3, 24, 20), W.Request(2, 10, 14), W.Request(1, 4, 4)],
                  [0.6, 0.9, 0.5], [("uniform", 0.3, 0.7), 0.5, 0.2], [6, 4, 3])
    check_end_to_end(wl)


def test_max_requests_end_to_end():
    """The request limit of the ABI (64 requests in one call, the C header's
    SPHINX_MAX_REQUESTS): ragged shapes of 1-3 frames and 2-12 latent rows and
    columns, start times 0.2-0.9, selected fractions 0.1-0.9 and 1-4 steps,
    end to end and teacher-forced per step."""
    rng = np.random.default_rng(64)
    R = 64
    shapes = [W.Request(int(rng.integers(1, 4)), 2 * int(rng.integers(1, 7)), 2 * int(rng.integers(1, 7)))
              for _ in range(R)]
    wl = W.custom("max_requests", MID_BF16, shapes, [float(x) for x in rng.uniform(0.2, 0.9, R)],
                  [float(x) for x in rng.uniform(0.1, 0.9, R)], [int(x) for x in rng.integers(1, 5, R)])
    assert wl.R == 64
    check_end_to_end(wl)


def test_empty_mask_is_identity():
    wl = W.custom("empty", MID_BF16, [W.Request(2, 16, 16)], [0.3], [0.5], [3])
    wl.thr[:] = np.inf
    R, _, sels = run_gpu(wl)
    assert all(n == 0 for n, _, _ in sels)
    assert np.array_equal(R.state.cpu().numpy(), wl.z0)
    # one empty request next to a refined one: the empty one stays bit-exact
    wl2 = W.custom("half_empty", MID_BF16, [W.Request(2, 16, 16), W.Request(1, 8, 8)], [0.3, 0.5], [0.5, 0.5],
                   [3, 3])
    wl2.thr[2:] = np.inf
    R2 = check_end_to_end(wl2, teacher_forced=False)
    e0 = 16 * wl2.tok_offset[1]
    assert np.array_equal(R2.state.cpu().numpy()[e0:], wl2.z0[e0:])


def test_all_selected_equals_dense():
    wl = W.custom("dense", MID_BF16, [W.Request(2, 16, 16), W.Request(1, 12, 8)], [1.0, 1.0], [0.5, 0.3], [3, 2])
    assert np.isneginf(wl.thr).all()
    R, _, _ = run_gpu(wl)
    got = R.state.cpu().numpy().astype(np.float64)
    dense = O.refine_dense(wl, precision="model")
    assert _report("all-selected vs dense oracle", got, dense) <= TOL["bf16"]


def test_headline_shape_one_block_step():
    """Every kernel at the headline launch configuration (9677 of 32256 tokens,
    D 1024, 16 heads, MLP 4096), one block deep so the oracle can follow."""
    model = W.ModelCfg(D=1024, heads=16, head_dim=64, mlp=4096, L=1, dtype="bf16")
    wl = W.headline(model=model)
    R, states, sels = run_gpu(wl, trace=True, steps=1)
    assert sels[0][0] == 9677
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    res = O.step(wl, O.model_from_workload(wl), wl.z0, plans[0], "model")
    assert np.array_equal(sels[0][1], res.idx)
    assert _report("headline L=1 step 0", states[1], res.state) <= TOL["bf16"]


@pytest.mark.parametrize("rho", [0.05, 0.07, 0.15, 0.2])
def test_headline_width_few_tile_gemms(rho):
    """One block of the headline width (D 1024, MLP 4096) at selections whose
    GEMMs have at most one tile per CU, so that they run one workgroup per CU
    with a deeper operand ring: on a 256-CU device 1613 and 2258 selected
    tokens put the QKV projection on 192- and 256-row tiles and MLP1 on
    256-row ones, 4838 and 6451 tokens the out-projection and MLP2 on 192- and
    256-row ones (K = 1024 and 4096, so the rings end with a partial trip)."""
    model = W.ModelCfg(D=1024, heads=16, head_dim=64, mlp=4096, L=1, dtype="bf16")
    wl = W.headline(model=model, rho=rho)
    R, states, sels = run_gpu(wl, trace=True, steps=1)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    res = O.step(wl, O.model_from_workload(wl), wl.z0, plans[0], "model")
    assert sels[0][0] == res.n_sel and np.array_equal(sels[0][1], res.idx)
    assert _report(f"headline width L=1, {res.n_sel} selected", states[1], res.state) <= TOL["bf16"]


def test_few_tile_gemms_match_packed():
    """The deep-ring GEMM tiles give bit-identical results to the two-workgroup
    tiles: three headline-shape requests (1613, 4838 and 6451 selected tokens)
    each alone run on the deep-ring kernels, and packed into one launch (12902
    rows) on the two-workgroup kernels."""
    model = W.ModelCfg(D=1024, heads=16, head_dim=64, mlp=4096, L=1, dtype="bf16")
    req = W.Request(14, 72, 128)
    wl = W.custom("few_tile_packed", model, [req, req, req], [0.05, 0.15, 0.2], [0.5, 0.5, 0.5], [25, 25, 25])
    worst = _packed_vs_separate(wl)
    print(f"[few-tile GEMMs] packed vs separate max_abs = {worst:.3e}")
    assert worst == 0.0


def test_headline_full_depth_properties():
    """12-block headline step: deterministic, unselected tokens untouched,
    finite, and only selected tokens move."""
    wl = W.headline()
    R, states, sels = run_gpu(wl, trace=True, steps=2)
    R2, states2, _ = run_gpu(wl, trace=True, steps=2)
    assert np.array_equal(states[2], states2[2]), "two runs differ"
    idx = sels[0][1]
    P0 = O.patchify(states[0], wl.requests)
    P2 = O.patchify(states[2], wl.requests)
    keep = np.ones(wl.N, bool)
    keep[idx] = False
    assert np.array_equal(P2[keep], P0[keep])
    assert np.isfinite(P2).all()
    print(f"[headline] 12 blocks, n_sel={len(idx)}, mean |dx| selected={np.abs(P2[idx] - P0[idx]).mean():.3f}")


def _packed_vs_separate(wl):
    R, _, _ = run_gpu(wl, steps=1)
    packed = R.state.cpu().numpy()
    del R
    worst = 0.0
    for r, q in enumerate(wl.requests):
        one = W.Workload(name=f"r{r}", model=wl.model, requests=[q],
                         u=wl.u[wl.tok_offset[r]:wl.tok_offset[r + 1]],
                         thr=wl.thr[wl.frame_offset[r]:wl.frame_offset[r + 1]],
                         s_start=wl.s_start[wl.frame_offset[r]:wl.frame_offset[r + 1]],
                         nsteps=wl.nsteps[r:r + 1], z0=wl.z0[16 * wl.tok_offset[r]:16 * wl.tok_offset[r + 1]],
                         eps=wl.eps[16 * wl.tok_offset[r]:16 * wl.tok_offset[r + 1]], weights=wl.weights)
        Rr, _, _ = run_gpu(one, steps=1)
        sep = Rr.state.cpu().numpy()
        worst = max(worst, float(np.abs(sep - packed[16 * wl.tok_offset[r]:16 * wl.tok_offset[r + 1]]).max()))
        del Rr
    return worst


def test_batched_packed_equals_separate():
    """Four requests packed varlen into one launch give the same result as each
    request alone (segment isolation), for a small batch and at the full
    batched shape: every row's arithmetic is independent of the packing."""
    small = W.custom("batched_small", W.HEADLINE_MODEL, [W.Request(6, 32, 32), W.Request(4, 24, 32),
                                                         W.Request(2, 16, 16)], [0.1, 0.6, 1.0], [0.3, 0.5, 0.7],
                     [10, 25, 25])
    exact = _packed_vs_separate(small)
    full = _packed_vs_separate(W.batched())
    print(f"[batched] packed vs separate max_abs: small batch {exact:.3e}, full batched shape {full:.3e}")
    assert exact <= 1e-5
    assert full <= 1e-5


XL1 = W.ModelCfg(D=1152, heads=16, head_dim=72, mlp=4608, L=1, dtype="bf16")


def test_frame_region_small_end_to_end_d72():
    """head_dim 72 (the DiT-XL-like denoiser) end to end on a reduced
    frame+region workload: 21 frames, top-8 fully refined, the rest 15 %,
    per-frame start times, 25 steps on one shared grid."""
    wl = W.build("frame_region_small", W.ModelCfg(D=1152, heads=16, head_dim=72, mlp=4608, L=2, dtype="bf16"),
                 [W.Request(21, 16, 16)], ["blobs"], [("frames_top_then_rho", 8, 0.15)],
                 [("uniform", 0.3, 0.7)], [25])
    check_end_to_end(wl, teacher_forced=False)


MID72 = W.ModelCfg(D=1152, heads=16, head_dim=72, mlp=1152, L=1, dtype="bf16")


def test_ragged_d72_tile_edges():
    """The pipelined head_dim-72 attention at its tile edges: four requests
    whose segments hold one partial key tile, exactly the two-tile path (one
    loop iteration and the last tile), and longer ragged tails, with staggered
    starts; every step teacher-forced against the oracle."""
    wl = W.custom("ragged72", MID72, [W.Request(3, 24, 20), W.Request(2, 16, 16), W.Request(2, 10, 14),
                                      W.Request(1, 4, 4)],
                  [0.6, 0.75, 0.9, 0.5], [("uniform", 0.3, 0.7), 0.5, 0.5, 0.2], [4, 3, 3, 2])
    R, _, sels = run_gpu(wl)
    lens = sorted({int(x) for _, _, cu in sels for x in np.diff(cu) if x > 0})
    print(f"[ragged72] segment lengths seen: {lens}")
    assert any(x < 64 for x in lens) and any(64 < x <= 128 for x in lens) and any(x > 128 for x in lens)
    _, trace = O.refine(wl, precision="model", trace=True)
    worst = teacher_forced_steps(R, wl, trace)
    print(f"[ragged72] teacher-forced per-step max_abs = {worst:.3e}")
    assert worst <= TOL["bf16"]


@pytest.mark.parametrize("width", ["d128", "d1152_h72"])
@pytest.mark.parametrize("n", [1, 3, 17, 33])
def test_few_selected_tokens(width, n):
    """Selections smaller than one row block of the matrix-core embedding (32
    rows) and final projection (16 rows): 1, 3, 17 and 33 tokens, at D 128 and
    at D 1152 with heads of 72, end to end and teacher-forced per step."""
    model = MID_BF16 if width == "d128" else MID72
    req = W.Request(1, 8, 8) if n < 16 else W.Request(1, 16, 16)
    tokens = (req.h // 2) * (req.w // 2) * req.frames
    wl = W.custom(f"few{n}_{width}", model, [req], [n / tokens], [0.5], [2])
    R = check_end_to_end(wl)
    assert R.n_sel == n


def test_frame_region_full_shape_one_block_step():
    """Frame+region at its full shape (21 x 64x64 latent) with a one-block
    head_dim-72 denoiser, at the first step with every frame active, from the
    oracle's forward-process state before it (its loop run with the true
    injected noise as the denoiser output)."""
    wl = W.frame_region(model=XL1)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    k = next(i for i, p in enumerate(plans) if p.active.all())
    before = forward_state(wl, k)
    R = S.from_workload(wl)
    R.reset()
    R.load_state(before)
    assert R.step(k, force_select=True) == 10194
    res = O.step(wl, O.model_from_workload(wl), before, plans[k], "model")
    assert np.array_equal(R.idx[:10194].cpu().numpy(), res.idx)
    got = R.state.cpu().numpy().astype(np.float64)
    assert _report(f"frame_region L=1 step {k} (teacher-forced)", got, res.state) <= TOL["bf16"]


def test_frame_region_full_depth_properties():
    """28-block head_dim-72 denoiser at the full frame+region shape: two
    steps, deterministic, unselected tokens untouched, finite."""
    wl = W.frame_region()
    _, s1, sel1 = run_gpu(wl, trace=True, steps=2)
    _, s2, _ = run_gpu(wl, trace=True, steps=2)
    assert np.array_equal(s1[2], s2[2])
    P0, P2 = O.patchify(s1[0], wl.requests), O.patchify(s1[2], wl.requests)
    moved = np.zeros(wl.N, bool)
    for n, idx, _ in sel1:
        moved[idx] = True
    assert np.array_equal(P2[~moved], P0[~moved])
    assert np.isfinite(P2).all()
    print(f"[frame_region] 28 blocks, n_sel per step {[n for n, _, _ in sel1]}")


def test_batched_full_shape_one_block_step():
    """The four-request batch at its full shape (30 925 selected tokens in four
    segments of 154 .. 12 902) with a one-block denoiser, against the oracle."""
    model = W.ModelCfg(D=1024, heads=16, head_dim=64, mlp=4096, L=1, dtype="bf16")
    wl = W.batched(model=model)
    R, states, sels = run_gpu(wl, trace=True, steps=1)
    assert sels[0][0] == 30925 and list(np.diff(sels[0][2])) == [154, 9677, 12902, 8192]
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    res = O.step(wl, O.model_from_workload(wl), wl.z0, plans[0], "model")
    assert _report("batched L=1 step 0", states[1], res.state) <= TOL["bf16"]
