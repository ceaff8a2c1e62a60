"""Pins of the search oracle (Algorithm 1 with the fitness of Eq. 3) against
things other than itself: the published first outputs of SplitMix64, offspring
worked out by hand from scripted draws, closed-form budgets, and invariants
(feasibility, range, elitism, the refine stage's stopping condition).  CPU only."""
import math

import numpy as np
import pytest

from oracle import search as ors


def test_splitmix64_published_outputs():
    # first three outputs of SplitMix64 started from state 0
    r = ors.CounterRng(0)
    assert [r.draw() for _ in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_below_is_in_range_and_roughly_uniform():
    r = ors.CounterRng(12345)
    counts = np.zeros(7, int)
    for _ in range(7000):
        v = r.below(7)
        assert 0 <= v < 7
        counts[v] += 1
    assert counts.min() > 850 and counts.max() < 1150


class Scripted:
    """Stand-in generator that returns scripted indices and checks the range asked for."""

    def __init__(self, script):
        self.script = list(script)

    def below(self, n):
        want_n, v = self.script.pop(0)
        assert n == want_n, f"asked for an index below {n}, script says {want_n}"
        return v


def small_problem(target):
    # latency = N0 + 2 N1 + 3 N2 (gamma = 1, b = 0); accuracy = N0 + N1 + N2
    lut = [[float(n) for n in range(1, 9)], [2.0 * n for n in range(1, 9)], [3.0 * n for n in range(1, 9)]]
    return ors.Problem(lut, [1.0, 1.0, 1.0], 0.0, target, lambda y: float(sum(y)))


def test_offspring_by_hand_overshoot_then_repair():
    P = small_problem(20.0)
    # overshoot K=2: U=[0,1,2], pick index 2 -> layer 2 (U becomes [2,1,0]), then 1 + 0 -> layer 1:
    #   [2,3,3] -> [2,4,4], latency 22 > 20
    # repair: V=[0,1,2], pick index 1 -> layer 1: [2,3,4], latency 20 <= 20
    # refine: every densification exceeds 20 (21, 22, 23): stop
    rng = Scripted([(3, 2), (2, 0), (3, 1)])
    assert ors.make_offspring(P, [2, 3, 3], 2, rng) == [2, 3, 4]
    assert rng.script == []


def test_offspring_by_hand_refine():
    P = small_problem(11.0)
    # overshoot K=1: pick layer 0: [1,1,1] -> [2,1,1], latency 7 (feasible, no repair)
    # refine: base 4; all three densifications fit (8, 9, 10): D=[0,1,2], pick index 2 -> [2,1,2] (10)
    #         base 5; only layer 0 fits (11): D=[0], pick it -> [3,1,2] (11)
    #         nothing fits any more (12, 13, 14): stop
    rng = Scripted([(3, 0), (3, 2), (1, 0)])
    assert ors.make_offspring(P, [1, 1, 1], 1, rng) == [3, 1, 2]
    assert rng.script == []


def test_refine_rejects_a_fitness_drop():
    lut = [[float(n) for n in range(1, 9)]] * 2
    # accuracy falls when layer 1 densifies past 2
    P = ors.Problem(lut, [1.0, 1.0], 0.0, 100.0, lambda y: y[0] - (5 if y[1] > 2 else 0))
    rng = Scripted([(2, 0)] + [(1, 0)] * 6)
    # overshoot layer 0 -> [2,2]; refine: D=[0] each round (layer 1 would lower the fitness) up to N0 = 8
    assert ors.make_offspring(P, [1, 2], 1, rng) == [8, 2]


def test_repair_gives_up_when_everything_is_sparsest():
    P = small_problem(5.0)             # even [1,1,1] costs 6
    y = ors.repair(P, [1, 1, 1], Scripted([]))
    assert y == [1, 1, 1] and P.fitness(y) == -math.inf
    assert ors.search(P.lut, P.gamma, 0.0, 5.0, P.accuracy, 3, 2, 1, seed=1) is None


def random_problem(seed, L=24):
    rng = np.random.default_rng(seed)
    base = rng.uniform(10, 100, L)
    lut = [[float(base[l] * (0.3 + 0.7 * n / 8) + rng.uniform(0, 2)) for n in range(1, 9)] for l in range(L)]
    gamma = rng.uniform(0.8, 1.2, L).tolist()
    b = float(rng.uniform(0, 20))
    sens = rng.uniform(0.1, 1.0, L)
    acc = lambda y: float(sum(sens[l] * math.log(y[l]) for l in range(L)))
    lo = sum(g * t[0] for g, t in zip(gamma, lut)) + b
    hi = sum(g * t[7] for g, t in zip(gamma, lut)) + b
    return lut, gamma, b, lo, hi, acc


@pytest.mark.parametrize("seed", range(4))
def test_search_invariants(seed):
    lut, gamma, b, lo, hi, acc = random_problem(seed)
    target = lo + (hi - lo) * (0.3 + 0.1 * seed)
    x, fx, trace = ors.search(lut, gamma, b, target, acc, generations=6, offspring=4, k_overshoot=3, seed=seed)
    P = ors.Problem(lut, gamma, b, target, acc)
    assert all(1 <= v <= 8 for v in x)
    assert P.latency(x) <= target and fx == P.acc(x)
    assert len(trace) == 7 and all(a <= c for a, c in zip(trace, trace[1:]))   # elitism
    # every offspring either failed repair or stops where refine stops
    rng = ors.CounterRng(99 + seed)
    for _ in range(5):
        y = ors.make_offspring(P, x, 3, rng)
        assert P.feasible(y)
        base = P.acc(y)
        for l in range(len(y)):
            if y[l] < 8:
                z = list(y)
                z[l] += 1
                assert not (P.feasible(z) and P.acc(z) >= base)


def test_closed_form_budgets():
    lut, gamma, b, lo, hi, acc = random_problem(7, L=10)
    x, fx, _ = ors.search(lut, gamma, b, hi + 1.0, acc, 3, 3, 2, seed=3)
    assert x == [8] * 10                                   # everything dense fits
    x, fx, _ = ors.search(lut, gamma, b, lo, acc, 3, 3, 2, seed=3)
    assert x == [1] * 10                                   # only the sparsest fits (the table grows with N)
    # no generation: the initial move leaves no single densification that fits
    mid = (lo + hi) / 2
    x, fx, trace = ors.search(lut, gamma, b, mid, acc, 0, 3, 2, seed=5)
    P = ors.Problem(lut, gamma, b, mid, acc)
    assert P.feasible(x) and trace == [fx]
    for l in range(10):
        if x[l] < 8:
            z = list(x)
            z[l] += 1
            assert not P.feasible(z)
