"""Oracle of the multi-stage selection with Elo ranking (Sec. 4.2 Stage 2, Eq. 9-12).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).  Plain Python floats (IEEE double).

Stage 1: every candidate j has an integer pointwise score s_j in 1..10 (Eq. 9); its Elo rating starts
at 1500 + 100 (s_j - 5); the top ceil(rho1 M) ratings survive (Eq. 10).
Stage 2: ceil(kappa M1) pairwise matches between neighbours in the rating order, each an Elo update
with K scaled by the verifier's confidence (high 1.2, medium 1.0, low 0.7; footnote of Stage 2); the
top ceil(rho2 M1) survive (Eq. 11).
Stage 3: every pair of survivors plays once; the winner is the highest rating (Eq. 12).

Readings (the paper leaves these open):
  * Elo: expected score E_a = 1 / (1 + 10^((r_b - r_a) / 400)), base K = 32; a win scores 1, a loss 0;
    the update r_a += K c (S_a - E_a), r_b -= the same amount (zero-sum).
  * "Top" orders by rating, larger first, equal ratings by smaller candidate index.
  * ceil(x) of a product with rho or kappa is taken as ceil(x - 1e-9), at least 1 for the survivor
    counts, so that a product that is an integer in exact arithmetic (0.3 x 10) is not rounded up.
  * Stage 2 sweeps the neighbour pairs (L[0], L[1]), (L[1], L[2]), ... of the list L of survivors in
    rating order, updating as it goes; when a sweep ends before ceil(kappa M1) matches, the survivors
    are re-ordered by their current ratings and the next sweep starts.  M1 < 2 plays no match.
  * Stage 3 orders the survivors by rating once, then plays positions (i, j), i < j, in lexicographic
    order.
  * The verifier is called as judge(a, b) with a ranked above b; it returns the winner (a or b) and a
    confidence 0 (high), 1 (medium) or 2 (low).
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Sequence, Tuple

K_BASE = 32.0
ELO_SCALE = 400.0
CONFIDENCE_K = (1.2, 1.0, 0.7)


def expected_score(r_a: float, r_b: float) -> float:
    return 1.0 / (1.0 + 10.0 ** ((r_b - r_a) / ELO_SCALE))


def elo_update(r: Dict[int, float], a: int, b: int, winner: int, confidence: int) -> None:
    s_a = 1.0 if winner == a else 0.0
    delta = K_BASE * CONFIDENCE_K[confidence] * (s_a - expected_score(r[a], r[b]))
    r[a] = r[a] + delta
    r[b] = r[b] - delta


def _ceil(x: float) -> int:
    return math.ceil(x - 1e-9)


def ranked(ids: Sequence[int], r: Dict[int, float]) -> List[int]:
    return sorted(ids, key=lambda j: (-r[j], j))


def select(scores: Sequence[int], judge: Callable[[int, int], Tuple[int, int]],
           rho1: float = 0.5, rho2: float = 0.5, kappa: float = 1.5):
    """Returns (winner, ratings [M], stages {"S1", "S2", "matches"}) ."""
    M = len(scores)
    r = {j: 1500.0 + 100.0 * (int(scores[j]) - 5) for j in range(M)}
    # Stage 1: pointwise pruning + Elo seeding (Eq. 10)
    S1 = ranked(range(M), r)[:max(1, _ceil(rho1 * M))]
    M1 = len(S1)
    matches = []
    # Stage 2: sparse pairwise between neighbours in rating order (Eq. 11)
    C2 = _ceil(kappa * M1) if M1 >= 2 else 0
    played = 0
    while played < C2:
        L = ranked(S1, r)
        for i in range(M1 - 1):
            if played == C2:
                break
            a, b = L[i], L[i + 1]
            w, c = judge(a, b)
            matches.append((a, b, w, c))
            elo_update(r, a, b, w, c)
            played += 1
    S2 = ranked(S1, r)[:max(1, _ceil(rho2 * M1))]
    # Stage 3: dense round robin, then argmax (Eq. 12)
    L2 = ranked(S2, r)
    for i in range(len(L2)):
        for j in range(i + 1, len(L2)):
            a, b = L2[i], L2[j]
            w, c = judge(a, b)
            matches.append((a, b, w, c))
            elo_update(r, a, b, w, c)
    winner = ranked(S2, r)[0]
    return winner, [r[j] for j in range(M)], {"S1": S1, "S2": S2, "matches": matches}


def pairwise_calls(M: int, rho1: float = 0.5, rho2: float = 0.5, kappa: float = 1.5) -> int:
    """Closed-form count of verifier pairwise calls of ``select``."""
    M1 = max(1, _ceil(rho1 * M))
    M2 = max(1, _ceil(rho2 * M1))
    return (_ceil(kappa * M1) if M1 >= 2 else 0) + M2 * (M2 - 1) // 2
