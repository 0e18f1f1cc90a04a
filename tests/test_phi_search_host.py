"""Host logic of the configuration search (Sec. 4.1; App. C) against the oracle: masks of phi, the
stand-in distance, the Pareto front and phi* selection (exact), and a dual-annealing run over an
analytic evaluator."""
import json
import os

import numpy as np
import pytest

from oracle import dispatch as odisp
from oracle import phi as ophi
from paper_2607_04461_amd import phi_search as ps

GOLD = os.path.join(os.path.dirname(__file__), "golden", "phi_star.json")


def _random_phis(rng, n, steps=50, L=30):
    out = []
    for _ in range(n):
        out.append(ps.decode(rng.random(5), steps, L, 8))
    return out


def test_masks_match_dispatcher_reading():
    cases = json.load(open(GOLD))["cases"]
    phis = [ps.Phi(*c["phi"]) for c in cases]
    phis += _random_phis(np.random.default_rng(1), 200)
    for phi in phis:
        L = 40 if phi.l_end > 30 else 30
        for k in range(phi.s_draft):
            s1, p1 = ps.phi_masks(phi, L, k)
            s2, p2 = odisp.masks_from_phi(phi.astuple(), L, k)
            assert np.array_equal(s1, s2) and np.array_equal(p1, p2)


def test_decode_is_always_valid_and_covers_the_corners():
    rng = np.random.default_rng(2)
    for x in list(rng.random((2000, 5))) + [np.zeros(5), np.ones(5)]:
        phi = ps.decode(x, 50, 30, 8)
        assert 1 <= phi.s_draft <= 50 and 0 <= phi.n_skip <= phi.s_draft
        assert 1 <= phi.l_start <= phi.l_end <= 30 and 1 <= phi.f_full <= 8
    assert ps.decode(np.zeros(5), 50, 30, 8) == ps.Phi(1, 0, 1, 1, 1)
    assert ps.decode(np.ones(5), 50, 30, 8) == ps.Phi(50, 50, 30, 30, 8)


def test_distance_front_and_selection_match_oracle():
    rng = np.random.default_rng(4)
    for _ in range(30):
        a, b = rng.standard_normal((2, 3, 8, 8))
        assert ps.latent_distance(a, b) == pytest.approx(ophi.latent_distance(a, b), rel=1e-12)
    for _ in range(100):
        n = int(rng.integers(1, 30))
        phis = _random_phis(rng, n)
        ev = [ps.Evaluation(phis[i], float(rng.integers(1, 8)) / 2, float(rng.integers(0, 10)) / 10, 0.0)
              for i in range(n)]
        pts = [(e.phi.astuple(), e.speedup, e.sim) for e in ev]
        assert ps.pareto_front(ev) == ophi.pareto_front(pts)
        assert ps.select_star(ev, 0.6) == ophi.select_star(pts, 0.6)


def _analytic_evaluator(L=30, steps=50):
    """Speedup = full block evaluations / the configuration's computed block evaluations (proxies and
    skips cost nothing); Sim falls with every knob.  Deterministic."""
    def evaluate(phi):
        work = 0
        for k in range(phi.s_draft):
            skip, proxy = ps.phi_masks(phi, L, k)
            if not proxy.any():
                work += int(L - skip.sum())
        speedup = steps * L / max(work, 1)
        n_skipped = phi.l_end - phi.l_start + 1
        sim = (phi.s_draft / steps) ** 0.5 * (1 - 0.02 * n_skipped) * (1 - 0.05 * (phi.f_full - 1))
        return speedup, max(sim, 0.0)
    return evaluate


def test_search_runs_and_selects_by_the_rule():
    evals, star, best = ps.search(_analytic_evaluator(), 50, 30, lam=0.1, maxiter=60, seed=5)
    phis = [e.phi for e in evals]
    assert len(set(phis)) == len(phis) >= 20
    pts = [(e.phi.astuple(), e.speedup, e.sim) for e in evals]
    assert star == ophi.select_star(pts, 0.6)
    assert best == max(range(len(evals)), key=lambda i: ophi.objective(pts[i][1], pts[i][2], 0.1))
    if star is not None:
        assert evals[star].sim >= 0.6 and star in ps.pareto_front(evals)
    again, star2, best2 = ps.search(_analytic_evaluator(), 50, 30, lam=0.1, maxiter=60, seed=5)
    assert [e.phi for e in again] == phis and (star2, best2) == (star, best)
