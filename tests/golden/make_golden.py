"""Writes the stored expected states of the full-depth parity tests
(``tests/test_gpu_full_depth.py``).  Calls only the CPU oracle (``oracle/``)
on the seeded inputs of ``workloads/``; nothing here runs on or reads from
the GPU path.

    python tests/golden/make_golden.py headline       # ~2-3 h on 8 cores
    python tests/golden/make_golden.py frame_region   # ~30 min
    python tests/golden/make_golden.py batched        # ~40 min

headline: the oracle's free-running 25-step trajectory (Alg. 1 loop, model
precision) with the 12-block denoiser; the state after steps 0, 1, 23 and 24
is stored (24 is the final state).
frame_region / batched: for each step k listed in GOLDEN_STEPS, the state
before step k is the oracle's loop run with the true-noise denoiser
(``golden_states.forward_state``); one oracle step with the full-depth
denoiser (28 / 12 blocks) from it is stored.
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path[:0] = [os.path.dirname(HERE), os.path.dirname(os.path.dirname(HERE))]

import oracle as O  # noqa: E402
import workloads as W  # noqa: E402
from golden_states import GOLDEN_STEPS, forward_state, input_digest, rows_from_state  # noqa: E402


def save(path, meta, arrays):
    tmp = path + ".tmp.npz"
    np.savez_compressed(tmp, **meta, **arrays)
    os.replace(tmp, path)


def main(name: str):
    wl = W.CONFIGS[name]()
    model = O.model_from_workload(wl)
    plans = O.plan_steps([r.frames for r in wl.requests], wl.s_start, wl.nsteps)
    info = O.token_info(wl.requests)
    path = os.path.join(HERE, f"{name}_L{wl.model.L}.npz")
    meta = {"digest": np.array(input_digest(wl)), "precision": np.array("model")}
    arrays = {}
    z0 = np.asarray(wl.z0, np.float64)
    t_all = time.time()
    if name == "headline":
        keep = {k for k in GOLDEN_STEPS[name]}
        state = z0.copy()
        for i, p in enumerate(plans):
            t0 = time.time()
            res = O.step(wl, model, state, p, "model", info=info)
            state = res.state
            print(f"{name} step {i}: n_sel {res.n_sel}, {time.time() - t0:.0f} s", flush=True)
            if i in keep:
                idx, x = rows_from_state(wl, state, z0)
                arrays[f"idx{i}"], arrays[f"x{i}"] = idx, x
                save(path, meta, arrays)
    else:
        for k in GOLDEN_STEPS[name]:
            t0 = time.time()
            before = forward_state(wl, k)
            res = O.step(wl, model, before, plans[k], "model", info=info)
            arrays[f"idx{k}"] = res.idx.astype(np.int32)
            arrays[f"x{k}"] = O.patchify(res.state, wl.requests)[res.idx].astype(np.float32)
            save(path, meta, arrays)
            print(f"{name} step {k}: n_sel {res.n_sel}, {time.time() - t0:.0f} s", flush=True)
    print(f"{name}: wrote {path} in {time.time() - t_all:.0f} s", flush=True)


if __name__ == "__main__":
    for n in sys.argv[1:] or ["headline", "frame_region", "batched"]:
        main(n)
