"""Pins of the adaptive start-step oracle (Sec. 5.1, Eq. 2, k-decision logic;
Alg. 1 k_min and the active rule) and the mistakes they catch: closed forms of
Eq. 2, a brute-force table lookup, monotonicity, and agreement of the start
indices with the partial-denoising plan's active rule (A_u = 1[k <= u])."""
import math

import numpy as np
import pytest

import oracle.adaptive_start as A
import oracle.sphinx_oracle as O

TABLE = A.KLogic(ratio=[0.80, 0.85, 0.90, 0.95, 1.00], k=[5, 15, 20, 25, 30, 40])


def pin_eq2_closed_forms(A):
    assert A.reference_quality(40.0, 60.0, 0.25, 1.0) == pytest.approx(45.0, abs=1e-12)  # gamma 1: linear
    assert A.reference_quality(60.0, 40.0, 0.25, 1.0) == pytest.approx(55.0, abs=1e-12)
    for c0, c1 in ((40.0, 60.0), (60.0, 40.0)):
        assert A.reference_quality(c0, c1, 0.0, 0.5) == pytest.approx(c0, abs=1e-12)
        assert A.reference_quality(c0, c1, 1.0, 0.5) == pytest.approx(c1, abs=1e-12)
    # rising: t^gamma; falling: 1 - (1 - t)^gamma, both concave for gamma < 1
    assert A.reference_quality(40.0, 60.0, 0.25, 0.5) == pytest.approx(40.0 + 20.0 * 0.5, abs=1e-12)
    assert A.reference_quality(60.0, 40.0, 0.25, 0.5) == pytest.approx(60.0 - 20.0 * (1 - math.sqrt(0.75)),
                                                                     abs=1e-12)
    ts = np.linspace(0, 1, 11)
    up = [A.reference_quality(40.0, 60.0, t, 0.6) for t in ts]
    dn = [A.reference_quality(60.0, 40.0, t, 0.6) for t in ts]
    assert all(a <= b for a, b in zip(up, up[1:])) and all(a >= b for a, b in zip(dn, dn[1:]))


def pin_table_lookup(A):
    for r, k in [(0.5, 5), (0.8, 15), (0.8499, 15), (0.85, 20), (0.97, 30), (1.0, 40), (7.0, 40)]:
        assert A.k_decision(TABLE, r) == k
    rng = np.random.default_rng(1)
    rs = np.sort(rng.uniform(0.6, 1.2, 200))
    ks = [A.k_decision(TABLE, r) for r in rs]
    assert all(a <= b for a, b in zip(ks, ks[1:]))
    for r, k in zip(rs, ks):  # brute force: the k of the last breakpoint not above r
        assert k == ([5] + [TABLE.k[i + 1] for i in range(5) if TABLE.ratio[i] <= r])[-1]


def pin_start_index(A):
    assert A.start_index_of_k(25, 50) == 499  # t_start 0.5
    assert A.start_index_of_k(0, 50) == 999 and A.start_index_of_k(40, 50) == 199
    assert A.start_index_of_k(1, 3) == 666  # 666.67 rounds to 667, minus 1
    assert A.start_index_of_k(1, 8) == 874  # 875 exactly, minus 1


def pin_alg1_active_rule(A):
    """Frame f joins at step u = k_f of the 50-step loop that starts at k_min."""
    rng = np.random.default_rng(2)
    frames = [5, 3]
    q_in = np.array([[45.0, 62.0], [70.0, 50.0]])
    q_reg = rng.uniform(35.0, 70.0, sum(frames))
    ks, ss, nsteps, _ = A.adaptive_start(frames, q_in, q_reg, 0.7, [TABLE], [0, 0], 50)
    plans = O.plan_steps(frames, ss, nsteps)
    g0 = 0
    for r, F in enumerate(frames):
        kmin = int(ks[g0:g0 + F].min())
        assert nsteps[r] == 50 - kmin
        for f in range(F):
            g = g0 + f
            active = [i for i in range(len(plans)) if plans[i].active[g]]
            assert active == list(range(int(ks[g]) - kmin, int(nsteps[r]))), (r, f)
        g0 += F


def pin_quality_monotone(A):
    """Better regression output (higher score) never starts earlier."""
    frames = [6]
    q_in = np.array([[50.0, 55.0]])
    lo = np.full(6, 40.0)
    ks_lo = A.adaptive_start(frames, q_in, lo, 0.5, [TABLE], [0])[0]
    ks_hi = A.adaptive_start(frames, q_in, lo + 8.0, 0.5, [TABLE], [0])[0]
    assert (ks_hi >= ks_lo).all() and (ks_hi > ks_lo).any()


PINS = [pin_eq2_closed_forms, pin_table_lookup, pin_start_index, pin_alg1_active_rule, pin_quality_monotone]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_adaptive_pin(pin):
    pin(A)


_orig = {n: getattr(A, n) for n in dir(A) if callable(getattr(A, n))}


def _eq2_no_branch(c0, c1, t, gamma):
    return c0 + (c1 - c0) * t ** gamma


def _lookup_strict(table, r):
    i = 0
    while i < len(table.ratio) and r > table.ratio[i]:
        i += 1
    return int(table.k[i])


def _s_truncate(k, S):
    return (1000 * (S - k)) // S - 1


def _steps_from_max(frames, q_in, q_reg, gamma, tables, cluster, S=50):
    ks, ss, ns, rs = _orig["adaptive_start"](frames, q_in, q_reg, gamma, tables, cluster, S)
    g0, out = 0, []
    for F in frames:
        out.append(S - int(ks[g0:g0 + F].max()))
        g0 += F
    return ks, ss, np.array(out), rs


def _inverse_ratio(c0, c1, t, gamma):
    return 1.0 / _orig["reference_quality"](c0, c1, t, gamma)


MUTANTS = {"eq2_single_branch": ("reference_quality", _eq2_no_branch),
           "lookup_strict_breakpoint": ("k_decision", _lookup_strict),
           "start_index_truncated": ("start_index_of_k", _s_truncate),
           "steps_from_k_max": ("adaptive_start", _steps_from_max),
           "reference_inverted": ("reference_quality", _inverse_ratio)}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_adaptive_pins_catch_mutant(name, monkeypatch):
    attr, bad = MUTANTS[name]
    monkeypatch.setattr(A, attr, bad)
    caught = []
    for pin in PINS:
        try:
            pin(A)
        except Exception as e:
            caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught {name}"
