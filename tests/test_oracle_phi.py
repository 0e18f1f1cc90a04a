"""Pins of the configuration-search oracle (App. C, Eq. 21-22): closed forms of the stand-in distance,
the objective's end points, and the Pareto front against an independent sweep algorithm."""
import numpy as np
import pytest

from oracle import phi as ophi


def test_latent_distance_closed_forms():
    a = np.random.default_rng(0).standard_normal((4, 6, 6))
    assert ophi.latent_distance(a, a) == 0.0
    assert ophi.latent_distance(a, -a) == pytest.approx(1.0)
    assert ophi.latent_distance(a, np.zeros_like(a)) == pytest.approx(1.0)
    assert ophi.latent_distance(a, 2 * a) == pytest.approx(1.0 / 3.0)
    assert ophi.latent_distance(np.zeros(3), np.zeros(3)) == 0.0


def test_similarity_and_objective():
    assert ophi.similarity([0.0, 0.0]) == 1.0
    assert ophi.similarity([0.2, 0.4]) == pytest.approx(0.7)
    assert ophi.objective(3.0, 0.7, 0.0) == 0.7
    assert ophi.objective(3.0, 0.7, 1.0) == 3.0
    assert ophi.objective(3.0, 0.7, 0.25) == pytest.approx(0.75 + 0.525)


def _front_by_sweep(points):
    # independent method: sort by speedup (desc), then Sim (desc); keep points whose Sim beats every
    # point of strictly larger speedup, and drop exact duplicates of a kept point's coordinates
    order = sorted(range(len(points)), key=lambda i: (-points[i][1], -points[i][2]))
    keep, best = [], -np.inf
    i = 0
    while i < len(order):
        j = i
        while j < len(order) and points[order[j]][1] == points[order[i]][1]:
            j += 1
        group = order[i:j]
        top = max(points[g][2] for g in group)
        if top > best:
            keep += [g for g in group if points[g][2] == top]
            best = top
        i = j
    return sorted(keep)


def test_pareto_front_hand_example():
    pts = [((1,), 1.0, 0.9), ((2,), 2.0, 0.8), ((3,), 2.0, 0.7), ((4,), 3.0, 0.5), ((5,), 1.5, 0.85),
           ((6,), 0.5, 0.95), ((7,), 3.0, 0.5)]
    assert ophi.pareto_front(pts) == [0, 1, 3, 4, 5, 6]
    assert ophi.select_star(pts, 0.6) == 1                    # speedup 2.0 at Sim 0.8
    assert ophi.select_star(pts, 0.96) is None
    assert ophi.select_star(pts, 0.5) == 3                    # tie at 3.0 / 0.5: smaller phi tuple


def test_pareto_front_matches_sweep_on_random_sets():
    rng = np.random.default_rng(3)
    for _ in range(50):
        n = int(rng.integers(1, 40))
        pts = [((i,), float(rng.integers(1, 8)) / 2, float(rng.integers(0, 10)) / 10) for i in range(n)]
        assert ophi.pareto_front(pts) == _front_by_sweep(pts)
