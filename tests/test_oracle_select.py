"""Pins of the selection oracle (Sec. 4.2 Stage 2, Eq. 9-12).

* Elo expected score and update: the textbook tournament example (a 1613 player meets 1609, 1477,
  1388, 1586 and 1720, scores 2.5; expected 2.867; K = 32 gives 1601), worked by hand below.
* A four-candidate run worked by hand, stage by stage.
* Invariants: ratings are zero-sum, so their total stays 1500 M + 100 sum(s - 5); the number of
  verifier calls equals its closed form, about 1.5 M at the paper's defaults versus M (M - 1) / 2 for
  exhaustive pairwise ranking; a verifier that always prefers the better candidate, with scores that
  order the candidates strictly, selects the best one.
* Degenerate pools (M = 1, 2) and kappa = 0.
"""
import math

import numpy as np
import pytest

from oracle import select as osel
from paper_2607_04461_amd import synth


def test_elo_textbook_tournament():
    opponents = [1609, 1477, 1388, 1586, 1720]
    expected = [osel.expected_score(1613, r) for r in opponents]
    # 10^(-4/400) = 0.97724 -> 0.5058; 10^(-136/400) = 0.45709 -> 0.6863; 10^(-225/400) = 0.27384
    # -> 0.7850; 10^(-27/400) = 0.85602 -> 0.5388; 10^(107/400) = 1.85139 -> 0.3507
    np.testing.assert_allclose(expected, [0.5058, 0.6863, 0.7850, 0.5388, 0.3507], atol=1e-4)
    assert sum(expected) == pytest.approx(2.867, abs=1e-3)
    assert round(1613 + 32 * (2.5 - sum(expected))) == 1601
    assert osel.expected_score(1500, 1500) == 0.5
    assert osel.expected_score(1900, 1500) == pytest.approx(10 / 11)     # 400 points: odds 10 : 1


def test_hand_worked_four_candidates():
    # scores 6 6 5 5 -> ratings 1600 1600 1500 1500; top ceil(0.5 * 4) = 2 -> {0, 1} (tie: index);
    # ceil(1.5 * 2) = 3 matches of the only neighbour pair, candidate 1 always wins, high confidence
    # (K c = 38.4):
    #   [0, 1]: E_0 = 0.5, delta = 38.4 (0 - 0.5) = -19.2               -> r0 1580.8, r1 1619.2
    #   [1, 0]: E_1 = 1 / (1 + 10^(-38.4 / 400)) = 0.555041, delta = 17.0864 -> 1636.2864, 1563.7136
    #   [1, 0]: E_1 = 1 / (1 + 10^(-72.5728 / 400)) = 0.602905, delta = 15.2484 -> 1651.5348, 1548.4652
    # top ceil(0.5 * 2) = 1 -> {1}; no dense matches; winner 1.
    calls = []

    def judge(a, b):
        calls.append((a, b))
        return 1, 0

    w, r, st = osel.select([6, 6, 5, 5], judge)
    assert w == 1 and st["S1"] == [0, 1] and st["S2"] == [1]
    assert calls == [(0, 1), (1, 0), (1, 0)]
    np.testing.assert_allclose(r, [1548.4652, 1651.5348, 1500.0, 1500.0], atol=2e-3)


@pytest.mark.parametrize("m", [1, 2, 3, 7, 16, 32, 64])
@pytest.mark.parametrize("params", [(0.5, 0.5, 1.5), (0.25, 0.5, 1.0), (1.0, 1.0, 0.0), (0.3, 0.7, 2.5)])
def test_zero_sum_and_call_count(m, params):
    v = synth.SyntheticVerifier(m, seed=m)
    w, r, st = osel.select(v.scores, v.judge, *params)
    assert sum(r) == pytest.approx(1500 * m + 100 * int(np.sum(v.scores - 5)), abs=1e-6)
    assert v.calls == len(st["matches"]) == osel.pairwise_calls(m, *params)
    assert w in st["S2"] and set(st["S2"]) <= set(st["S1"])


def test_call_count_about_one_and_a_half_m():
    for m in (16, 32):
        calls = osel.pairwise_calls(m)
        assert 1.0 * m <= calls <= 2.0 * m
        assert calls < m * (m - 1) / 2
    assert osel.pairwise_calls(32) == math.ceil(1.5 * 16) + 8 * 7 // 2   # 24 + 28 = 52 ~ 1.6 M


def test_exact_products_are_not_rounded_up():
    assert osel.pairwise_calls(10, 0.3, 1.0, 0.0) == 3 * 2 // 2          # M1 = 3 (0.3 x 10), M2 = 3


def test_perfect_verifier_selects_the_best():
    rng = np.random.default_rng(5)
    for _ in range(20):
        m = int(rng.integers(2, 11))
        quality = rng.permutation(m)
        scores = 1 + quality                                            # strictly ordered, 1..m <= 10
        judge = lambda a, b: ((a if quality[a] > quality[b] else b), 0)
        w, _, _ = osel.select(scores, judge)
        assert w == int(np.argmax(quality))


def test_degenerate_pools():
    never = lambda a, b: pytest.fail("no match expected")
    assert osel.select([3], never)[0] == 0
    assert osel.select([4, 7], never)[0] == 1                            # M1 = 1: pointwise argmax
    assert osel.select([7, 7], never)[0] == 0                            # tie: smaller index
    w, r, st = osel.select([5, 9, 9, 1], never, 1.0, 0.25, 0.0)          # kappa = 0, M2 = 1
    assert w == 1 and r == [1500.0, 1900.0, 1900.0, 1100.0] and st["matches"] == []
