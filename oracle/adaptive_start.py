"""Plain CPU oracle of Sphinx's adaptive start-step selection (Sec. 5.1, Eq. 2,
the k-decision logic; Alg. 1 k <- K_c(r), k_min <- min(k)).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  It shares
no code with the library and imports nothing from it.

* Eq. 2: the reference quality of a target frame is interpolated between the
  quality scores c0, c1 of the two input views with a power law in the
  target's normalised position t (t^gamma when c1 >= c0, 1 - (1-t)^gamma
  otherwise).
* Sec. 5.1: the ratio r = (regression output quality) / (reference quality)
  is mapped by a monotone k-decision table of the request's scene cluster to
  the start step k of a 50-step schedule (the largest k is 40 in the paper).
* Alg. 1: the request starts at k_min = min over its frames of k; frame f
  joins when the step counter reaches k_f.  With t_start = 1 - k/S and start
  index s = round(1000 t_start) - 1, and n = S - k_min steps on the grid from
  s_max, this is exactly the active rule of the partial-denoising plan.

Readings (also in the design notes): target j of n (1-based) sits at
t = j / (n + 1), so no target coincides with an input view; the k table is a
parameter (the paper's figure gives no numbers); rounding of 1000 (S - k) / S
is half up.
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction
from typing import List, Sequence

import numpy as np


@dataclass
class KLogic:
    ratio: Sequence[float]  # strictly increasing breakpoints
    k: Sequence[int]  # len(ratio) + 1 non-decreasing start steps


def reference_quality(c0: float, c1: float, t: float, gamma: float) -> float:
    """Eq. 2: Q* = c0 + (c1 - c0) f(t)."""
    f = t ** gamma if c1 >= c0 else 1.0 - (1.0 - t) ** gamma
    return c0 + (c1 - c0) * f


def k_decision(table: KLogic, r: float) -> int:
    """Start step of ratio r: k[i] with i the number of breakpoints <= r."""
    i = 0
    while i < len(table.ratio) and r >= table.ratio[i]:
        i += 1
    return int(table.k[i])


def start_index_of_k(k: int, S: int) -> int:
    """s = round(1000 (1 - k/S)) - 1, rounded half up, exactly."""
    x = Fraction(1000 * (S - k), S)
    return int(x + Fraction(1, 2)) - 1 if x.denominator != 1 else int(x) - 1


def adaptive_start(frames: Sequence[int], q_in: np.ndarray, q_reg: np.ndarray, gamma: float,
                   tables: Sequence[KLogic], cluster: Sequence[int], S: int = 50):
    """Per frame k, start index s and ratio r; per request the step count S - k_min."""
    ks: List[int] = []
    ss: List[int] = []
    rs: List[float] = []
    nsteps: List[int] = []
    g = 0
    for r_i, F in enumerate(frames):
        c0, c1 = float(q_in[r_i][0]), float(q_in[r_i][1])
        kk = []
        for f in range(F):
            t = (f + 1) / (F + 1)
            ratio = float(q_reg[g]) / reference_quality(c0, c1, t, gamma)
            k = k_decision(tables[cluster[r_i]], ratio)
            kk.append(k)
            rs.append(ratio)
            ss.append(start_index_of_k(k, S))
            g += 1
        ks.extend(kk)
        nsteps.append(S - min(kk))
    return np.array(ks), np.array(ss), np.array(nsteps), np.array(rs)
