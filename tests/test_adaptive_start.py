"""The library's adaptive start-step selection (host code behind the C ABI)
against the oracle (Sec. 5.1, Eq. 2, k-decision logic; Alg. 1 k_min), bit for
bit in the integers, plus argument validation.  No GPU needed."""
import ctypes
import os

import numpy as np
import pytest

import oracle.adaptive_start as A
import workloads as W

S = pytest.importorskip("paper_2511_18672_amd")

TABLES = [([0.80, 0.85, 0.90, 0.95, 1.00], [5, 15, 20, 25, 30, 40]),
          ([0.7, 0.9], [10, 25, 40]),
          ([], [25])]


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(S.binding.LIB_PATH):
        pytest.skip("libsphinx.so not built")
    return S.lib()


def _oracle_tables():
    # the library's breakpoints are float32: give the oracle the same values
    return [A.KLogic([float(np.float32(x)) for x in r], k) for r, k in TABLES]


@pytest.mark.parametrize("gamma", [1.0, 0.5, 0.625, 0.3])
def test_adaptive_start_matches_oracle(L, gamma):
    rng = np.random.default_rng(int(gamma * 1000))
    reqs_py = [W.Request(6, 8, 8), W.Request(14, 72, 128), W.Request(21, 64, 64), W.Request(1, 4, 4)]
    q_in, q_reg = W.quality_scores(reqs_py, seed=int(gamma * 100))
    cluster = rng.integers(0, len(TABLES), len(reqs_py)).astype(np.int32)
    g = np.float32(gamma)
    got = S.sphinx_adaptive_start(S.make_requests(reqs_py), q_in, q_reg, float(g),
                                  [S.make_klogic(r, k) for r, k in TABLES], cluster, 50)
    ks, ss, ns, rs = A.adaptive_start([q.frames for q in reqs_py], q_in.astype(np.float64),
                                      q_reg.astype(np.float64), float(g), _oracle_tables(), cluster, 50)
    assert np.array_equal(got["k"], ks)
    assert np.array_equal(got["s_start"], ss)
    assert np.array_equal(got["nsteps"], ns)
    assert np.abs(got["ratio"] - rs).max() <= 1e-15 * np.abs(rs).max()
    print(f"[adaptive gamma={gamma}] k = {np.bincount(ks, minlength=41)[[5, 10, 15, 20, 25, 30, 40]]}, "
          f"steps = {list(ns)}")


def test_adaptive_start_other_schedules(L):
    reqs_py = [W.Request(5, 8, 8)]
    q_in, q_reg = W.quality_scores(reqs_py, seed=3)
    for steps in (3, 8, 25, 7):
        tab = ([0.8, 0.9], [0, steps // 3, steps - 1])
        got = S.sphinx_adaptive_start(S.make_requests(reqs_py), q_in, q_reg, 0.5, [S.make_klogic(*tab)],
                                      np.zeros(1, np.int32), steps)
        ref = A.adaptive_start([5], q_in.astype(np.float64), q_reg.astype(np.float64), 0.5,
                               [A.KLogic([float(np.float32(x)) for x in tab[0]], tab[1])], [0], steps)
        assert np.array_equal(got["s_start"], ref[1]) and np.array_equal(got["nsteps"], ref[2])


def test_adaptive_start_validation(L):
    reqs = S.make_requests([W.Request(2, 8, 8)])
    P = ctypes.c_void_p
    qi = np.array([50.0, 60.0], np.float32)
    qr = np.array([45.0, 55.0], np.float32)
    cl = np.zeros(1, np.int32)
    outs = [np.zeros(2, np.int32), np.zeros(2, np.int32), np.zeros(1, np.int32)]
    good = S.make_klogic([0.9], [10, 40])

    def call(gamma=0.5, tab=good, n_tables=1, cluster=cl, steps=50, q_in=qi, q_reg=qr):
        arr = (S.KLogic * 1)(tab)
        return L.sphinx_adaptive_start(reqs, 1, P(q_in.ctypes.data), P(q_reg.ctypes.data), ctypes.c_float(gamma),
                                       arr, n_tables, P(cluster.ctypes.data), steps,
                                       *[P(o.ctypes.data) for o in outs], None)

    assert call() == 0
    assert call(gamma=0.0) == 1 and call(gamma=1.5) == 1
    assert call(steps=0) == 1 and call(steps=40) == 1  # k = 40 outside [0, S-1]
    assert call(tab=S.make_klogic([0.9, 0.8], [10, 20, 30])) == 1  # breakpoints not increasing
    assert call(tab=S.make_klogic([0.9], [40, 10])) == 1  # k decreasing
    assert call(cluster=np.array([1], np.int32)) == 1
    assert call(q_in=np.array([0.0, 60.0], np.float32)) == 1
    assert call(q_reg=np.array([np.nan, 55.0], np.float32)) == 1
