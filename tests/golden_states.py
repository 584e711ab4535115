"""Helpers shared by the full-depth parity tests and the script that writes
their stored expected states (``tests/golden/make_golden.py``).

Teacher-forced full-depth steps need the state *before* a late step.  For the
headline workload that is the oracle's own free-running trajectory (stored).
For the frame+region and batched workloads the state before step k is the one
the oracle's loop reaches when its denoiser returns exactly the noise that was
injected: every refined token then sits on the forward-process line
sqrt(abar(tau_k)) z0 + sqrt(1 - abar(tau_k)) eps (Alg. 1 loop with the DDIM
update; the exactness of this is itself a pin of the oracle).  That state is
recomputed here, by the oracle, in seconds.

Stored states hold only the token rows that differ from z0: ``idx{i}`` (int32,
ascending token ids) and ``x{i}`` (float32 [n][16], value order c*4+py*2+px).
"""
from __future__ import annotations

import hashlib

import numpy as np

import oracle as O

GOLDEN_STEPS = {
    # workload: {step: how its before-state is made}
    "headline": {0: "z0", 1: "stored", 23: None, 24: "stored"},
    "frame_region": {0: "z0", 14: "forward"},
    "batched": {0: "z0", 10: "forward"},
}


def true_noise_denoiser(wl):
    """A denoiser that returns, for every forwarded token, the noise injected into it."""
    info = O.token_info(wl.requests)
    E = O.patchify(wl.eps, wl.requests)
    key = {(int(info.req[t]), int(info.f[t]), int(info.y[t]), int(info.x[t])): t for t in range(wl.N)}

    def den(model, x, f, y, xx, tau, seg, precision):
        req = np.searchsorted(np.asarray(seg), np.arange(x.shape[0]), side="right") - 1
        rows = [key[(int(req[j]), int(f[j]), int(y[j]), int(xx[j]))] for j in range(x.shape[0])]
        return E[np.asarray(rows, dtype=np.int64)]

    return den


def forward_state(wl, k: int) -> np.ndarray:
    """NCHW state (float64) before step k of the oracle's loop run with the true-noise denoiser."""
    if k == 0:
        return np.asarray(wl.z0, np.float64).copy()
    return O.refine(wl, precision="fp64", denoiser=true_noise_denoiser(wl), steps=k)


def input_digest(wl) -> str:
    """Digest of the seeded inputs a stored state depends on (latents, noise,
    map, thresholds, schedule and a sample of the weights)."""
    h = hashlib.sha256()
    for a in (wl.z0, wl.eps, wl.u, wl.thr, wl.s_start, wl.nsteps):
        h.update(np.ascontiguousarray(a).tobytes())
    L = wl.model.L
    for name in ("pe_w", "t2_w", "b0.qkv_w", f"b{L - 1}.fc2_w", "fada_w", "out_w"):
        h.update(np.ascontiguousarray(wl.weights[name]).tobytes())
    return h.hexdigest()[:32]


def rows_from_state(wl, state: np.ndarray, base: np.ndarray):
    """Token rows of `state` that differ from `base` (both NCHW)."""
    P, B = O.patchify(state, wl.requests), O.patchify(base, wl.requests)
    idx = np.flatnonzero((P != B).any(axis=1)).astype(np.int32)
    return idx, P[idx].astype(np.float32)


def state_from_rows(wl, base: np.ndarray, idx: np.ndarray, x: np.ndarray) -> np.ndarray:
    """NCHW state (float64): `base` with token rows idx replaced by x."""
    P = O.patchify(base, wl.requests)
    P[np.asarray(idx, np.int64)] = np.asarray(x, np.float64)
    return O.unpatchify(P, wl.requests)
