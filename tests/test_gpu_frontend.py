"""GPU parity of the mask front-end (Sec. 5.3; Alg. 1 laplacian_var, otsu,
opacity mask, union, block rule) against the integer-exact CPU oracle:
token masks and per-frame Otsu thresholds bit for bit, through the C ABI."""
import numpy as np
import pytest

import oracle.mask_frontend as M
import workloads as W

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2511_18672_amd")

pytestmark = pytest.mark.gpu


def run_frontend(requests, rgb, opac, tau=0.5):
    reqs = S.make_requests(requests)
    N = sum(q.tokens for q in requests)
    G = sum(q.frames for q in requests)
    d_rgb = torch.from_numpy(np.concatenate([a.ravel() for a in rgb])).cuda()
    d_op = torch.from_numpy(np.concatenate([a.ravel() for a in opac]).astype(np.float32)).cuda()
    mask = torch.full((N,), 7, dtype=torch.uint8, device="cuda")
    u = torch.full((N,), -1.0, dtype=torch.float32, device="cuda")
    thr = torch.full((G,), -1, dtype=torch.int32, device="cuda")
    ws = torch.empty(S.sphinx_mask_frontend_workspace_bytes(reqs), dtype=torch.uint8, device="cuda")
    S.sphinx_mask_frontend(reqs, d_rgb, d_op, tau, mask, u, thr, ws)
    torch.cuda.synchronize()
    return mask.cpu().numpy(), u.cpu().numpy(), thr.cpu().numpy()


def check(requests, rgb, opac, tau=0.5, tag=""):
    mask, u, thr = run_frontend(requests, rgb, opac, tau)
    ref_mask, ref_thr = M.request_masks(requests, rgb, opac, tau)
    assert np.array_equal(thr, ref_thr), (thr, ref_thr)
    assert np.array_equal(mask.astype(bool), ref_mask)
    assert set(np.unique(mask)) <= {0, 1}
    assert np.array_equal(u, ref_mask.astype(np.float32))
    print(f"[frontend {tag}] {len(ref_thr)} frames, {ref_mask.size} tokens, {int(ref_mask.sum())} masked, "
          f"otsu t = {list(ref_thr[:6])}")
    return mask


def test_frontend_ragged_requests():
    """Image widths that are not multiples of the 64-pixel tile, several requests."""
    reqs = [W.Request(2, 8, 12), W.Request(1, 6, 4), W.Request(3, 4, 18)]
    rgb, opac = W.frontend_inputs(reqs, seed=11)
    check(reqs, rgb, opac, tag="ragged")


def test_frontend_special_frames():
    """A constant frame (every pixel blurry), a saturated checkerboard (the
    largest Laplacian), opacity exactly at the threshold, and no opacity cue."""
    req = [W.Request(4, 8, 16)]
    H, Wd = 64, 128
    rng = np.random.default_rng(3)
    rgb = np.empty((4, H, Wd, 3), np.uint8)
    rgb[0] = 90
    yy, xx = np.mgrid[0:H, 0:Wd]
    rgb[1] = (255 * ((yy + xx) % 2))[..., None].astype(np.uint8)
    rgb[2] = rng.integers(0, 256, (H, Wd, 3), dtype=np.uint8)
    rgb[3] = rng.integers(0, 256, (H, Wd, 3), dtype=np.uint8)
    rgb[3, :, :40] = 17
    opac = np.ones((4, H, Wd), np.float32)
    opac[2] = 0.5
    opac[2, 5, 70] = np.nextafter(np.float32(0.5), np.float32(0))
    opac[3, 33:40, 100:110] = 0.1
    check(req, [rgb], [opac], tag="special")


def test_frontend_opacity_threshold_values():
    reqs = [W.Request(2, 8, 8)]
    rgb, opac = W.frontend_inputs(reqs, seed=12)
    for tau in (0.0, 0.3, 1.0, 1.5):
        check(reqs, rgb, opac, tau, tag=f"tau={tau}")


def test_frontend_headline_shape():
    """14 frames of 576 x 1024 (the headline views): every token and every
    Otsu threshold bit for bit, and the uncertainty output selects exactly the
    mask through sphinx_select_mask at thr = 0.5."""
    reqs = [W.Request(14, 72, 128)]
    rgb, opac = W.frontend_inputs(reqs)
    mask = check(reqs, rgb, opac, tag="headline")
    N = reqs[0].tokens
    r = S.make_requests(reqs)
    _, u, _ = run_frontend(reqs, rgb, opac)
    m2 = torch.empty(N, dtype=torch.uint8, device="cuda")
    idx = torch.empty(N, dtype=torch.int32, device="cuda")
    cu = torch.empty(2, dtype=torch.int32, device="cuda")
    ws = torch.empty(S.sphinx_select_workspace_bytes(N), dtype=torch.uint8, device="cuda")
    thr = torch.full((14,), 0.5, dtype=torch.float32, device="cuda")
    cu_h = S.sphinx_select_mask(r, torch.from_numpy(u).cuda(), thr, None, m2, idx, cu, ws)
    assert np.array_equal(m2.cpu().numpy(), mask)
    assert int(cu_h[-1]) == int(mask.sum())


def test_pipeline_frontend_adaptive_refine():
    """Alg. 1 from the regression output on: the front-end mask (as the 0/1
    uncertainty map at thr 0.5), adaptive per-frame start steps from synthetic
    quality scores, then the partial-denoising loop, against the oracle's
    composition of the same three parts."""
    import oracle as O
    import oracle.adaptive_start as A

    model = W.ModelCfg(D=128, heads=2, head_dim=64, mlp=512, L=2, dtype="bf16")
    reqs_py = [W.Request(3, 16, 16), W.Request(2, 8, 24)]
    rgb, opac = W.frontend_inputs(reqs_py, seed=21)
    _, u_gpu, _ = run_frontend(reqs_py, rgb, opac)
    ref_mask, _ = M.request_masks(reqs_py, rgb, opac)
    assert np.array_equal(u_gpu, ref_mask.astype(np.float32))
    q_in, q_reg = W.quality_scores(reqs_py, seed=22)
    table = ([0.8, 0.9, 1.0], [40, 43, 45, 47])
    got = S.sphinx_adaptive_start(S.make_requests(reqs_py), q_in, q_reg, 0.5, [S.make_klogic(*table)],
                                  np.zeros(2, np.int32), 50)
    ks, ss, ns, _ = A.adaptive_start([q.frames for q in reqs_py], q_in.astype(np.float64), q_reg.astype(np.float64),
                                     0.5, [A.KLogic([float(np.float32(x)) for x in table[0]], table[1])], [0, 0], 50)
    assert np.array_equal(got["s_start"], ss) and np.array_equal(got["nsteps"], ns)
    wl = W.custom("pipeline", model, reqs_py, [0.5, 0.5], [0.5, 0.5], [3, 3])
    wl.u = u_gpu
    wl.thr = np.full(wl.G, 0.5, np.float32)
    wl.s_start = got["s_start"].astype(np.int32)
    wl.nsteps = got["nsteps"].astype(np.int32)
    R = S.from_workload(wl)
    out = R.run().cpu().numpy().astype(np.float64)
    ref = O.refine(wl, precision="model")
    err = np.abs(out - ref).max()
    print(f"[pipeline] k = {list(ks)}, steps = {list(ns)}, masked = {int(ref_mask.sum())}/{wl.N}, "
          f"max_abs = {err:.3e}")
    assert err <= 2e-2
