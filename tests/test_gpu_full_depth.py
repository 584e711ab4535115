"""Full-depth parity at the paper-sized workloads, through the C ABI, against
oracle states stored by ``tests/golden/make_golden.py`` (which calls only the
CPU oracle):

* headline (14 x 72x128 latent, 9677 of 32256 tokens, 12 blocks D 1024):
  steps 0, 1 and 24 teacher-forced (the oracle's state before the step loaded
  into the GPU state) and the free-running 25-step result;
* frame+region (21 x 64x64, 28 blocks D 1152, head_dim 72, per-frame starts):
  step 0 (one frame active) and step 14 (the first with every frame active);
* batched (four requests packed into one launch, 12 blocks D 1024): step 0
  (all four requests live, 30925 tokens) and step 10 (the two 10-step
  requests finished).

For frame+region and batched the state before a late step is the oracle's
loop run with the true injected noise as denoiser output, recomputed here.
Masks and indices are compared bit-exact, latents element by element at the
bf16 bar (2e-2 max-abs); tokens outside the step's selection must keep the
state they had before it bit for bit, i.e. the oracle's state as loaded (rounded
once to the GPU state's storage type: requests that finished earlier hold fp64
values there).  Runs in the launch configuration the benchmark times (Refiner,
token-major state).
"""
import os

import numpy as np
import pytest

import oracle as O
import workloads as W
from golden_states import forward_state, input_digest, state_from_rows

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2511_18672_amd")

pytestmark = pytest.mark.gpu

TOL = 2e-2
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
_WL = {}


def workload(name):
    if name not in _WL:
        _WL.clear()
        _WL[name] = W.CONFIGS[name]()
    return _WL[name]


def golden(wl, *steps):
    path = os.path.join(GOLDEN, f"{wl.name}_L{wl.model.L}.npz")
    if not os.path.exists(path):
        pytest.skip(f"{path} not written yet (tests/golden/make_golden.py {wl.name})")
    g = np.load(path, allow_pickle=False)
    assert str(g["digest"]) == input_digest(wl), f"{path} was written for other inputs: regenerate it"
    missing = [k for k in steps if f"x{k}" not in g.files]
    if missing:
        pytest.skip(f"{path} holds no state after step(s) {missing} yet")
    return g


def _refiner(wl):
    torch.cuda.empty_cache()
    R = S.from_workload(wl)
    R.reset()
    return R


def _compare(tag, R, wl, before, idx, x):
    """GPU state after the step vs `before` with the oracle's rows idx <- x."""
    got = R.state.cpu().numpy().astype(np.float64)
    loaded = torch.from_numpy(np.ascontiguousarray(before)).to(R.state.dtype).double().numpy()
    expect = state_from_rows(wl, loaded, idx, x)
    Pg, Pe = O.patchify(got, wl.requests), O.patchify(expect, wl.requests)
    keep = np.ones(wl.N, bool)
    keep[idx] = False
    assert np.array_equal(Pg[keep], Pe[keep]), f"{tag}: tokens outside the selection changed"
    err = float(np.abs(Pg[idx] - Pe[idx]).max())
    print(f"[{tag}] {len(idx)} refined tokens, max_abs vs oracle = {err:.3e}", flush=True)
    assert np.isfinite(Pg).all()
    return err


def _teacher_forced(name, k, before):
    wl = workload(name)
    g = golden(wl, k)
    R = _refiner(wl)
    R.load_state(before)
    print(f"[{name} L={wl.model.L}] step {k}", flush=True)
    n = R.step(k, force_select=True)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    info = O.token_info(wl.requests)
    act = plans[k].active[info.gframe]
    _, idx, cu, n_ref = O.select(wl.u, wl.thr[info.gframe], act, wl.tok_offset[:-1])
    assert n == n_ref and np.array_equal(R.idx[:n].cpu().numpy(), idx)
    assert list(R.cu_host) == list(cu) + [n_ref]
    # stored rows: the step's selection (headline: every token refined so far,
    # which is the same selection at every step)
    gi, gx = g[f"idx{k}"], g[f"x{k}"]
    assert np.array_equal(gi, idx)
    err = _compare(f"{name} L={wl.model.L} step {k} teacher-forced", R, wl, before, gi, gx)
    assert err <= TOL
    del R


def _headline_state(g, wl, k):
    return state_from_rows(wl, wl.z0, g[f"idx{k}"], g[f"x{k}"])


@pytest.mark.parametrize("k", [0, 1, 24])
def test_headline_teacher_forced(k):
    wl = workload("headline")
    g = golden(wl, *([k] if k == 0 else [k - 1, k]))
    before = np.asarray(wl.z0, np.float64) if k == 0 else _headline_state(g, wl, k - 1)
    _teacher_forced("headline", k, before)


def test_headline_free_running_25_steps():
    wl = workload("headline")
    g = golden(wl, 24)
    R = _refiner(wl)
    for i in range(R.total_steps):
        R.step(i)
    err = _compare("headline L=12 free-running 25 steps", R, wl, np.asarray(wl.z0, np.float64), g["idx24"],
                   g["x24"])
    assert err <= TOL


@pytest.mark.parametrize("k", [0, 14])
def test_frame_region_teacher_forced(k):
    wl = workload("frame_region")
    golden(wl, k)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    if k == 14:
        assert plans[k].active.all() and not plans[k - 1].active.all()
    _teacher_forced("frame_region", k, forward_state(wl, k))


@pytest.mark.parametrize("k", [0, 10])
def test_batched_teacher_forced(k):
    wl = workload("batched")
    golden(wl, k)
    _teacher_forced("batched", k, forward_state(wl, k))
