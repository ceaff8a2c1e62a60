"""Oracle of the layer-wise N:M search (paper Sec. 5.2, Algorithm 1 and the
fitness of Eq. 3) -- test infrastructure only (tests, smoke check and
benchmark baseline use it; the product library never does).

The steps are taken in the paper's order: initialisation (fittest uniform
configuration within the budget, then a random move towards the budget), and
per generation lambda offspring made by overshoot, repair and refine, followed
by selection.  Readings where the paper is silent (the same as the library's):

* search space N:8, N in 1..8 per layer (8 = dense);
* the uniform candidates are the eight all-N configurations; the fittest
  feasible one is taken (first in N order on ties);
* the random move towards the budget makes passes over the layers, each in a
  fresh random order, densifying each visited layer by one level when the
  budget still holds, until a pass changes nothing;
* overshoot densifies `overshoot` distinct random non-dense layers (all of
  them if fewer);
* repair gives up (the offspring stays infeasible, fitness -inf) when every
  layer is already 1:8;
* refine accepts a densification when it keeps the budget and does not lower
  the fitness (Delta fitness >= 0 with -inf for infeasible configurations);
* selection is (1 + lambda): the fittest offspring (first on ties) replaces
  the parent unless it is less fit.

Random draws come from SplitMix64 (Steele, Lea and Flood, 2014) used as a
counter-based generator: draw i of seed s is mix64(s + (i + 1) * golden), and
an index below n is floor(draw * n / 2^64).  Draws are consumed in this order:
the layer order of each initial pass (Fisher-Yates), then per offspring the overshoot
subset (partial Fisher-Yates), one draw per repair step and one per refine
step.
"""
import math

GOLDEN = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1
LEVELS = 8


def mix64(z):
    """SplitMix64's output function."""
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


class CounterRng:
    def __init__(self, seed):
        self.seed = seed & MASK64
        self.count = 0

    def draw(self):
        z = (self.seed + (self.count + 1) * GOLDEN) & MASK64
        self.count += 1
        return mix64(z)

    def below(self, n):
        return (self.draw() * n) >> 64


class Problem:
    """lut[l][N-1] = t_l(N:8); T_pred by Eq. 1; fitness by Eq. 3."""

    def __init__(self, lut, gamma, b, target, accuracy):
        self.lut, self.gamma, self.b, self.target, self.accuracy = lut, gamma, b, target, accuracy
        self.L = len(lut)

    def latency(self, y):
        total = 0.0
        for l in range(self.L):
            total += self.gamma[l] * self.lut[l][y[l] - 1]
        return total + self.b

    def feasible(self, y):
        return self.latency(y) <= self.target

    def acc(self, y):
        v = self.accuracy(list(y))
        return -math.inf if math.isnan(v) else v

    def fitness(self, y):
        return self.acc(y) if self.feasible(y) else -math.inf


def uniform_candidate(P):
    best, best_f = None, None
    for n in range(1, LEVELS + 1):
        y = [n] * P.L
        if not P.feasible(y):
            continue
        f = P.acc(y)
        if best is None or f > best_f:
            best, best_f = y, f
    return best


def towards_target(P, y, rng):
    while True:
        order = list(range(P.L))
        for j in range(P.L - 1):
            r = j + rng.below(P.L - j)
            order[j], order[r] = order[r], order[j]
        changed = False
        for l in order:
            if y[l] < LEVELS:
                y[l] += 1
                if P.feasible(y):
                    changed = True
                else:
                    y[l] -= 1
        if not changed:
            return y


def overshoot(P, y, k, rng):
    U = [l for l in range(P.L) if y[l] < LEVELS]
    K = min(k, len(U))
    for j in range(K):
        r = j + rng.below(len(U) - j)
        U[j], U[r] = U[r], U[j]
        y[U[j]] += 1
    return y


def repair(P, y, rng):
    while not P.feasible(y):
        V = [l for l in range(P.L) if y[l] > 1]
        if not V:
            return y
        y[V[rng.below(len(V))]] -= 1
    return y


def refine(P, y, rng):
    if not P.feasible(y):
        return y
    while True:
        base = P.acc(y)
        D = []
        for l in range(P.L):
            if y[l] >= LEVELS:
                continue
            y[l] += 1
            if P.feasible(y) and P.acc(y) >= base:
                D.append(l)
            y[l] -= 1
        if not D:
            return y
        y[D[rng.below(len(D))]] += 1


def make_offspring(P, x, k, rng):
    y = list(x)
    y = overshoot(P, y, k, rng)
    y = repair(P, y, rng)
    return refine(P, y, rng)


def search(lut, gamma, b, target, accuracy, generations, offspring, k_overshoot, seed, rng=None):
    """Returns (best configuration, its fitness, trace of the parent's fitness
    before each generation and at the end); None when no uniform
    configuration meets the budget."""
    P = Problem(lut, gamma, b, target, accuracy)
    rng = rng or CounterRng(seed)
    x = uniform_candidate(P)
    if x is None:
        return None
    x = towards_target(P, list(x), rng)
    fx = P.fitness(x)
    trace = []
    for _ in range(generations):
        trace.append(fx)
        champion, fc = None, -math.inf
        for _ in range(offspring):
            y = make_offspring(P, x, k_overshoot, rng)
            fy = P.fitness(y)
            if champion is None or fy > fc:
                champion, fc = y, fy
        if fc >= fx:
            x, fx = champion, fc
    trace.append(fx)
    return x, fx, trace
