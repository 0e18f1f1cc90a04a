"""Oracle of the draft-configuration search objective and selection (Sec. 4.1; App. C, Eq. 21-22).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).

  Sim(phi) = 1 - mean over the calibration prompts of the distance between y_phi(x) and y_base(x)
             (the paper's distance is LPIPS; the harness substitutes a latent-space distance),
  J(phi)   = lambda * T_base / T(phi) + (1 - lambda) * Sim(phi),
  Pareto front over (speedup, Sim), both maximised; phi* = the largest speedup with Sim >= 0.6
  (ties: larger Sim, then the smaller phi tuple).

Readings: the stand-in distance is d(a, b) = ||a - b||_2 / (||a||_2 + ||b||_2), in [0, 1]; a point is
on the front if no other point is at least as good in both coordinates and better in one.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def latent_distance(a, b) -> float:
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    den = np.linalg.norm(a) + np.linalg.norm(b)
    return 0.0 if den == 0.0 else float(np.linalg.norm(a - b) / den)


def similarity(distances: Sequence[float]) -> float:
    """Eq. 21 with the per-prompt distances given."""
    return 1.0 - float(np.mean(np.asarray(distances, np.float64)))


def objective(speedup: float, sim: float, lam: float) -> float:
    """Eq. 22."""
    return lam * speedup + (1.0 - lam) * sim


def pareto_front(points: Sequence[Tuple[tuple, float, float]]) -> List[int]:
    """Indices of (phi, speedup, sim) points that no other point dominates (brute force)."""
    out = []
    for i, (_, si, mi) in enumerate(points):
        dominated = False
        for j, (_, sj, mj) in enumerate(points):
            if j != i and sj >= si and mj >= mi and (sj > si or mj > mi):
                dominated = True
                break
        if not dominated:
            out.append(i)
    return out


def select_star(points: Sequence[Tuple[tuple, float, float]], min_sim: float = 0.6):
    """Index of phi*: the largest speedup among points with Sim >= min_sim, or None."""
    ok = [i for i, p in enumerate(points) if p[2] >= min_sim]
    if not ok:
        return None
    return min(ok, key=lambda i: (-points[i][1], -points[i][2], tuple(points[i][0])))
