"""Pins of the GABRA oracle (oracle/gabra.py) against what the paper and the
mathematics fix: the generator's published outputs, the exact optimum of
eqs. 7-10 by enumeration (itself pinned on a hand-solved instance), each
operator of Algorithms 1-3 on worked examples, the roulette wheel's
probabilities, and the rejection of duplicate and infeasible offspring."""
import numpy as np
import pytest

from oracle import gabra as G


def test_splitmix64_published_outputs():
    """The first three outputs of SplitMix64 from state 0, as printed by its
    reference implementation."""
    assert [G.splitmix64(0, k) for k in range(3)] == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_uniform_and_below_ranges():
    r = G.Rng(7)
    u = [r.uniform() for _ in range(20000)]
    assert min(u) >= 0.0 and max(u) < 1.0 and abs(np.mean(u) - 0.5) < 0.01
    b = [r.below(5) for _ in range(20000)]
    assert set(b) == set(range(5))
    assert np.allclose(np.bincount(b) / len(b), 0.2, atol=0.01)


def test_profits_eq3():
    c = G.profits([2.0, 6.0], [4.0, 3.0])
    assert c == [[0.5, 2.0 / 3.0], [1.5, 2.0]]


def test_feasibility_eq8_and_every_gpu():
    p, d = [2.0, 3.0, 1.0], [5.0, 1.0]
    assert G.feasible([0, 0, 1], p, d)            # loads 5 <= 5 and 1 <= 1: capacity may be met
    assert not G.feasible([0, 1, 0], p, d)        # 3 > 1 on GPU 1
    assert not G.feasible([0, 0, 0], p, d)        # 6 > 5
    assert not G.feasible([0, 0, 0], [1.0, 1.0, 1.0], [5.0, 1.0], every_gpu=True)
    assert G.feasible([0, 0, 1], p, d, every_gpu=True)


def test_brute_force_hand_solved():
    """Two unit partitions, GPUs of capacity 1 and 2: both on GPU 1 exceed it,
    both on GPU 2 earn 1/2 + 1/2 = 1, one each earns 1/1 + 1/2 = 1.5."""
    best, f = G.brute_force([1.0, 1.0], [1.0, 2.0])
    assert f == 1.5 and best == [0, 1]
    assert G.brute_force([3.0], [1.0, 2.0]) == (None, None)
    best, f = G.brute_force([1.0, 1.0], [3.0, 3.0], every_gpu=True)
    assert f == pytest.approx(2.0 / 3.0) and sorted(best) == [0, 1]


def test_midpoint_crossover_algorithm3():
    y1, y2 = [1, 1, 1, 1, 1, 1], [2, 2, 2, 2, 2, 2]
    assert G.midpoint_crossover(y1, y2) == ([1, 1, 1, 2, 2, 2], [2, 2, 2, 1, 1, 1])
    a, b = G.midpoint_crossover([0, 1, 2, 3, 4, 5, 6], [9, 8, 7, 6, 5, 4, 3])
    assert a == [0, 1, 2, 6, 5, 4, 3] and b == [9, 8, 7, 3, 4, 5, 6]   # cut after floor(7/2)


def test_inversion_mutation():
    assert G.inversion([1, 2, 3, 4, 5], 1, 3) == [1, 4, 3, 2, 5]
    assert G.inversion([1, 2, 3, 4, 5], 0, 4) == [5, 4, 3, 2, 1]
    assert G.inversion([7, 8], 0, 1) == [8, 7]


def test_roulette_probabilities():
    """Selection probability = fitness / total fitness."""
    r = G.Rng(3)
    fits = [1.0, 2.0, 3.0, 4.0]
    k = np.bincount([G.roulette(r, fits) for _ in range(200000)], minlength=4)
    assert np.allclose(k / k.sum(), [0.1, 0.2, 0.3, 0.4], atol=0.004)


def _instance(seed, n, m, slack):
    rng = np.random.default_rng(seed)
    p = rng.uniform(1.0, 10.0, n).round(3)
    d = rng.uniform(0.5, 1.5, m)
    d = (d / d.sum() * p.sum() * slack).round(3)
    d = np.maximum(d, p.max())  # every partition fits somewhere
    return list(map(float, p)), list(map(float, d))


INSTANCES = [
    (1, 5, 2, 1.3, False), (2, 6, 3, 1.4, False), (3, 7, 3, 1.25, False), (4, 8, 4, 1.5, False),
    (5, 8, 2, 1.2, False), (6, 4, 4, 2.0, False), (7, 8, 3, 1.35, True), (8, 6, 4, 1.6, True),
    (9, 8, 4, 1.3, False), (10, 3, 1, 1.1, False),
]


def test_ga_reaches_brute_force_optimum():
    """The GA is a heuristic: a single run can settle on a local optimum.  On
    each seeded instance (n <= 8 partitions, m <= 4 GPUs) the best of three
    seeded runs equals the exact optimum of eqs. 7-10, every run returns a
    feasible allocation whose profit is its fitness, and at least 24 of the
    30 runs reach the optimum on their own."""
    hits = 0
    for seed, n, m, slack, every in INSTANCES:
        p, d = _instance(seed, n, m, slack)
        best, fb = G.brute_force(p, d, every)
        assert best is not None
        found = []
        for s in range(3):
            z, fz, st = G.gabra(p, d, population=30, generations=1500, seed=1000 * s + seed,
                                every_gpu=every)
            assert G.feasible(z, p, d, every)
            assert fz == G.fitness(z, G.profits(p, d))
            assert fz <= fb * (1 + 1e-12)
            found.append(abs(fz - fb) <= 1e-12 * fb)
        assert any(found), (seed, fb)
        hits += sum(found)
    assert hits >= 24, hits


def test_duplicates_rejected():
    """With one GPU every chromosome is the same allocation: every offspring
    equals a population member and is dropped, so no generation completes and
    the run stops at the attempt bound with the initial best."""
    z, fz, st = G.gabra([1.0, 2.0, 3.0], [10.0], population=5, generations=10, max_attempts=40)
    assert z == [0, 0, 0] and fz == pytest.approx(0.6)
    assert st == dict(generations=0, duplicates=40, infeasible=0, attempts=40)


def test_infeasible_offspring_rejected():
    p, d = _instance(11, 8, 3, 1.05)
    z, fz, st = G.gabra(p, d, population=20, generations=300, seed=5)
    assert st["infeasible"] > 0 and G.feasible(z, p, d)


def test_no_feasible_population_raises():
    with pytest.raises(ValueError):
        G.gabra([5.0, 5.0], [4.0, 4.0], population=4, generations=10, init_tries=50)


def test_initial_population_algorithm2():
    """Each partition goes to a GPU drawn uniformly among those with room
    left: with loads (4, 1) and capacities (4, 1) the only feasible allocation
    is forced; with one unit load and three equal GPUs each GPU is drawn a
    third of the time."""
    r = G.Rng(11)
    for _ in range(50):
        assert G.initial_chromosome(r, [4.0, 1.0], [4.0, 1.0], False, 10) == [0, 1]
    k = np.bincount([G.initial_chromosome(r, [1.0], [5.0, 5.0, 5.0], False, 1)[0]
                     for _ in range(30000)], minlength=3)
    assert np.allclose(k / k.sum(), 1.0 / 3.0, atol=0.01)
    assert G.initial_chromosome(r, [2.0, 2.0], [3.0], False, 5) is None
