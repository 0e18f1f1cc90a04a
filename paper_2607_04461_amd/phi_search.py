"""Search for the draft configuration phi = (S', n_skip, l_start, l_end, f_full) (Sec. 4.1
Configuration Space; App. C).

The search maximises J(phi) = lambda T_base / T(phi) + (1 - lambda) Sim(phi) (Eq. 22) with dual
annealing (scipy's generalized simulated annealing without its local search; each iteration proposes
a chain of moves, and a configuration is evaluated once however often it is proposed),
then takes phi* = the fastest configuration with Sim >= 0.6 from the evaluated set (App. C, Pareto
selection).  T is wall-clock time measured on the GPU through the library; Sim is 1 - the mean
distance of the draft's preview to the full-compute output over a calibration pool (Eq. 21).  The
paper measures that distance with LPIPS on decoded images; without a VAE or LPIPS weights the
harness uses the normalised latent distance ||a - b|| / (||a|| + ||b||) in [0, 1].

The preview of a draft is its clean-latent estimate at t_S': x0 = z - t v with the last step's
velocity v (rectified flow, App. A.1), i.e. one Euler jump from t_S' to 0; for S' = S it is z itself.

Masks follow the dispatcher's reading of phi: blocks l_start..l_end (1-based) are skipped from step
n_skip on; steps with k mod f_full == 0 compute every other block, the rest proxy them.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True, order=True)
class Phi:
    s_draft: int
    n_skip: int
    l_start: int
    l_end: int
    f_full: int

    def astuple(self) -> tuple:
        return dataclasses.astuple(self)


def phi_masks(phi: Phi, num_blocks: int, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """(skip, proxy) uint8 masks of draft step k (0-based, k < S')."""
    if not 0 <= k < phi.s_draft:
        raise ValueError("step outside the draft")
    skip = np.zeros(num_blocks, np.uint8)
    proxy = np.zeros(num_blocks, np.uint8)
    if k >= phi.n_skip:
        skip[phi.l_start - 1:phi.l_end] = 1
    if phi.f_full > 1 and k % phi.f_full:
        proxy[:] = 1
    return skip, proxy


def decode(x: Sequence[float], steps: int, num_blocks: int, f_max: int) -> Phi:
    """Point of the annealer's box [0, 1)^5 -> a valid configuration (every coordinate is a fraction of
    its own range, so every point is valid): S' in 1..S, n_skip in 0..S', 1 <= l_start <= l_end <= L,
    f_full in 1..f_max."""
    u = [min(max(float(v), 0.0), 1.0 - 1e-12) for v in x]
    s_draft = 1 + int(u[0] * steps)
    n_skip = int(u[1] * (s_draft + 1))
    l_start = 1 + int(u[2] * num_blocks)
    l_end = l_start + int(u[3] * (num_blocks - l_start + 1))
    f_full = 1 + int(u[4] * f_max)
    return Phi(s_draft, n_skip, l_start, l_end, f_full)


def latent_distance(a, b) -> float:
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    den = float(np.sqrt(a @ a) + np.sqrt(b @ b))
    return 0.0 if den == 0.0 else float(np.sqrt((a - b) @ (a - b)) / den)


def objective(speedup: float, sim: float, lam: float) -> float:
    return lam * speedup + (1.0 - lam) * sim


@dataclasses.dataclass
class Evaluation:
    phi: Phi
    speedup: float
    sim: float
    seconds: float


def pareto_front(evals: Sequence[Evaluation]) -> List[int]:
    """Indices of the evaluations no other one beats in both speedup and Sim (sweep by speedup)."""
    order = sorted(range(len(evals)), key=lambda i: (-evals[i].speedup, -evals[i].sim))
    front, best_sim, i = [], -math.inf, 0
    while i < len(order):
        j = i
        while j < len(order) and evals[order[j]].speedup == evals[order[i]].speedup:
            j += 1
        top = max(evals[g].sim for g in order[i:j])
        if top > best_sim:
            front += [g for g in order[i:j] if evals[g].sim == top]
            best_sim = top
        i = j
    return sorted(front)


def select_star(evals: Sequence[Evaluation], min_sim: float = 0.6) -> Optional[int]:
    ok = [i for i, e in enumerate(evals) if e.sim >= min_sim]
    if not ok:
        return None
    return min(ok, key=lambda i: (-evals[i].speedup, -evals[i].sim, evals[i].phi.astuple()))


def search(evaluate: Callable[[Phi], Tuple[float, float]], steps: int, num_blocks: int, lam: float = 0.5,
           maxiter: int = 200, seed: int = 0, f_max: int = 8, min_sim: float = 0.6):
    """Dual annealing on -J over the decoded box for ``maxiter`` iterations.  ``evaluate(phi) ->
    (speedup, sim)`` is called once per distinct configuration (results are cached).  Returns (evaluations, index of phi* or None,
    index of the best J)."""
    from scipy.optimize import dual_annealing
    import time

    cache: Dict[Phi, int] = {}
    evals: List[Evaluation] = []

    def neg_j(x):
        phi = decode(x, steps, num_blocks, f_max)
        if phi not in cache:
            t0 = time.time()
            sp, sim = evaluate(phi)
            cache[phi] = len(evals)
            evals.append(Evaluation(phi, float(sp), float(sim), time.time() - t0))
        e = evals[cache[phi]]
        return -objective(e.speedup, e.sim, lam)

    dual_annealing(neg_j, bounds=[(0.0, 1.0)] * 5, maxiter=maxiter, seed=seed, no_local_search=True)
    best = max(range(len(evals)), key=lambda i: objective(evals[i].speedup, evals[i].sim, lam))
    return evals, select_star(evals, min_sim), best


class GpuEvaluator:
    """T(phi) and Sim(phi) of a draft pool on the GPU.  The pool's candidates (one or more per prompt)
    form the calibration set; T_base is the full schedule with every knob off, timed once."""

    def __init__(self, pool, reps: int = 1):
        import torch
        self.torch, self.pool, self.reps = torch, pool, reps
        self.z0 = pool.latents.detach().clone()
        self.sched = pool.schedule
        self.steps = len(self.sched) - 1
        self.t_base, self.y_base = self._run_base()

    def _time(self, fn) -> float:
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        best = math.inf
        for _ in range(self.reps):
            self._reset()
            torch.cuda.synchronize()
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        return best

    def _reset(self):
        import ctypes
        self.pool.latents.copy_(self.z0)
        ctypes.memset(self.pool.meta, 0, ctypes.sizeof(self.pool.meta))

    def _run_base(self):
        def run():
            for k in range(self.steps):
                self.pool.refine_step(k)
        t = self._time(run)
        return t, self.pool.latents.detach().double().cpu().numpy()

    def __call__(self, phi: Phi) -> Tuple[float, float]:
        L = self.pool.L
        prev = {}

        def run():
            for k in range(phi.s_draft):
                if k == phi.s_draft - 1:
                    prev["z"] = self.pool.latents.detach().clone()
                skip, proxy = phi_masks(phi, L, k)
                self.pool.draft_step(k, skip=skip, proxy=proxy)
        t = self._time(run)
        z = self.pool.latents.detach().double().cpu().numpy()
        t_s = float(self.sched[phi.s_draft])
        if t_s > 0.0:
            z_prev = prev["z"].double().cpu().numpy()
            v = (z - z_prev) / (t_s - float(self.sched[phi.s_draft - 1]))
            preview = z - t_s * v
        else:
            preview = z
        dist = [latent_distance(preview[i], self.y_base[i]) for i in range(z.shape[0])]
        return self.t_base / t, 1.0 - float(np.mean(dist))


def main(argv=None) -> int:
    """Measure T_base / T(phi) and Sim(phi) of given configurations on a workload's pool, and
    optionally run the search.  One JSON line per configuration, then one for the search."""
    import argparse
    import json
    import sys

    from . import synth
    from .pool import DraftPool

    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--workload", default="wan1.3b_pool16")
    ap.add_argument("--dtype", default=None)
    ap.add_argument("--phi", action="append", default=[], help="S',n_skip,l_start,l_end,f_full (repeatable)")
    ap.add_argument("--search-iters", type=int, default=0)
    ap.add_argument("--lam", type=float, default=0.5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--f-max", type=int, default=8)
    ap.add_argument("--reps", type=int, default=1)
    args = ap.parse_args(argv)
    wl = synth.WORKLOADS[args.workload]
    pool = DraftPool(wl, dtype=args.dtype)
    pool.reset()
    ev = GpuEvaluator(pool, reps=args.reps)
    print(json.dumps({"workload": wl.name, "t_base_ms": round(ev.t_base, 2), "steps": ev.steps}), flush=True)
    for s in args.phi:
        phi = Phi(*(int(v) for v in s.split(",")))
        sp, sim = ev(phi)
        print(json.dumps({"phi": phi.astuple(), "speedup": round(sp, 3), "sim": round(sim, 5),
                          "t_ms": round(ev.t_base / sp, 2)}), flush=True)
    if args.search_iters:
        evals, star, best = search(ev, ev.steps, pool.L, lam=args.lam, maxiter=args.search_iters,
                                   seed=args.seed, f_max=args.f_max)
        front = pareto_front(evals)
        print(json.dumps({"evaluated": len(evals), "lambda": args.lam,
                          "best_J": evals[best].phi.astuple(),
                          "phi_star": None if star is None else evals[star].phi.astuple(),
                          "phi_star_speedup": None if star is None else round(evals[star].speedup, 3),
                          "phi_star_sim": None if star is None else round(evals[star].sim, 5),
                          "front": [(evals[i].phi.astuple(), round(evals[i].speedup, 3), round(evals[i].sim, 5))
                                    for i in front]}), flush=True)
    pool.close()
    return 0


if __name__ == "__main__":
    import sys
    sys.exit(main())
