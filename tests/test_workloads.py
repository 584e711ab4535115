"""Seeded workload recipes: shapes, selected counts and determinism."""
import numpy as np
import pytest

import workloads as W


def _selected(wl):
    per = np.concatenate([[r.hp * r.wp] * r.frames for r in wl.requests])
    return wl.u > np.repeat(wl.thr, per)


@pytest.mark.parametrize("name,counts", [
    ("small", [1024]), ("headline", [9677]), ("frame_region", [10194]),
    ("batched", [154, 9677, 12902, 8192])])
def test_selected_counts(name, counts):
    wl = W.CONFIGS[name](with_weights=False)
    sel = _selected(wl)
    off = wl.tok_offset
    assert [int(sel[off[r]:off[r + 1]].sum()) for r in range(wl.R)] == counts


def test_tiny_shapes_and_determinism():
    a, b = W.tiny(), W.tiny()
    assert a.N == 32 and a.G == 2 and a.z0.shape == (512,)
    assert np.array_equal(a.z0, b.z0) and np.array_equal(a.u, b.u)
    for k in a.weights:
        assert np.array_equal(a.weights[k], b.weights[k])
    assert list(a.s_start) == [499, 499]


def test_bf16_storage_is_exact():
    wl = W.small()
    for arr in [wl.z0, wl.eps, wl.weights["b0.qkv_w"]]:
        bits = arr.view(np.uint32)
        assert np.all((bits & 0xFFFF) == 0)


def test_frame_region_frames():
    wl = W.frame_region(with_weights=False)
    assert int(np.isneginf(wl.thr).sum()) == 8
    assert wl.s_start.min() >= 299 and wl.s_start.max() <= 699


def test_rho_threshold_edges():
    u = np.arange(10, dtype=np.float32)
    assert W.rho_threshold(u, 1.0) == -np.inf
    assert W.rho_threshold(u, 0.0) == np.inf
    assert W.rho_threshold(u, 0.3) == 6.0
