"""Pins of the oracle's control plane (oracle.control): ODA (Alg. 1) against worked
examples derived by hand from the algorithm's steps, the PASM's flow invariants, and
the optimality claim of Sec. 4.3 checked by brute force: for super-linear degradation
in the speed gap, Eq. 2 at ODA's PASM equals the minimum over all transport plans
(a linear program solved by scipy). Also the scheduler's draw and Eq. 3."""

import numpy as np
import pytest
from scipy.optimize import linprog

from oracle import control as C


def test_oda_worked_examples():
    # all demand at the fast end, supply at the slow end: excess moves left step by step
    # v3: 0.5 > 0.2 -> 0.3 (60 %) to v2; v2: 0.6 > 0.3 -> 0.3 (50 %) to v1; v1: 0.5 = 0.5
    T = C.oda([0.2, 0.3, 0.5], [0.5, 0.3, 0.2])
    assert np.allclose(T, [[1, 0, 0], [0.5, 0.5, 0], [0.3, 0.3, 0.4]], atol=1e-15)
    # shortfalls at the fast end pull from the nearest slower level first
    # v3: 0 < 0.5 -> all of v2 (0.5); v2: 0 < 0.5 -> all of v1; v1: 0 = 0
    T = C.oda([0.5, 0.5, 0.0], [0.0, 0.5, 0.5])
    assert np.allclose(T, [[0, 1, 0], [0, 0, 1], [0, 0, 1]], atol=1e-15)
    # a shortfall that needs two levels: v3 takes 0.1 from v2 (all of it) and 0.3 of v1
    T = C.oda([0.6, 0.1, 0.3], [0.2, 0.1, 0.7])
    # v3: 0.3 < 0.7 -> 0.1 from v2 (P = 1), 0.3 from v1 (P = 0.5); v2: 0 < 0.1 -> 0.1 from v1
    assert np.allclose(T, [[2 / 6, 1 / 6, 3 / 6], [0, 0, 1], [0, 0, 1]], atol=1e-15)
    # equal histograms: the identity
    assert np.allclose(C.oda([0.25, 0.25, 0.5], [0.25, 0.25, 0.5]), np.eye(3))


def _random_instance(rng, n):
    H = rng.dirichlet(np.ones(n) * 0.7)
    F = rng.dirichlet(np.ones(n) * 0.7)
    H[rng.random(n) < 0.2] = 0.0
    if H.sum() == 0:
        H[rng.integers(n)] = 1.0
    H /= H.sum()
    return H, F


def test_oda_flow_invariants():
    rng = np.random.default_rng(5)
    for n in range(1, 9):
        for _ in range(50):
            H, F = _random_instance(rng, n)
            T = C.oda(H, F)
            assert np.all(T >= -1e-15)
            assert np.allclose(T.sum(axis=1), 1.0, atol=1e-12)
            assert np.allclose(H @ T, F, atol=1e-12)     # the served load is the solver's split


def _lp_min(H, F, D):
    """min sum_{i<j} M[i][j] D[j][i] over M >= 0 with row sums H and column sums F
    (shifts to slower levels, j < i, are free: no quality loss)."""
    n = H.size
    cost = np.array([D[j, i] if j > i else 0.0 for i in range(n) for j in range(n)])
    A, b = [], []
    for i in range(n):
        row = np.zeros(n * n)
        row[i * n:(i + 1) * n] = 1
        A.append(row)
        b.append(H[i])
    for j in range(n - 1):  # the last column sum follows from the totals
        col = np.zeros(n * n)
        col[j::n] = 1
        A.append(col)
        b.append(F[j])
    r = linprog(cost, A_eq=np.array(A), b_eq=np.array(b), bounds=(0, None), method="highs")
    assert r.status == 0
    return r.fun


@pytest.mark.parametrize("power", [1.5, 2.0, 3.0])
def test_oda_attains_the_minimum_of_eq2(power):
    """Sec. 4.3: with degradation growing super-linearly in the throughput gap, ODA's
    PASM minimises Eq. 2 over every redistribution that serves the split F."""
    rng = np.random.default_rng(int(power * 10))
    for n in range(2, 7):
        for _ in range(40):
            H, F = _random_instance(rng, n)
            P = np.cumsum(rng.uniform(0.5, 2.0, n))           # throughput rises with the level
            D = np.array([[max(P[j] - P[i], 0.0) ** power for i in range(n)] for j in range(n)])
            T = C.oda(H, F)
            got = C.degradation(T, H, D)
            best = _lp_min(H, F, D)
            assert got <= best + 1e-9 * max(1.0, best), (H, F, got, best)


def test_oda_rejects_bad_histograms():
    with pytest.raises(ValueError):
        C.oda([0.5, 0.5], [0.5, 0.6])
    with pytest.raises(ValueError):
        C.oda([0.5, 0.5], [1.0])
    with pytest.raises(ValueError):
        C.oda([-0.1, 1.1], [0.5, 0.5])


def test_route_cumulative_draw():
    T = np.array([[1, 0, 0], [0.5, 0.5, 0], [0.3, 0.3, 0.4]])
    assert [C.route(T, 2, u) for u in (0.0, 0.2999, 0.3, 0.5999, 0.6, 0.99999)] == [0, 0, 1, 1, 2, 2]
    assert C.route(T, 0, 0.7) == 0
    # rounding that leaves the row's sum below u falls on the last level with mass
    assert C.route(np.array([[0.25, 0.7499999, 0.0]]), 0, 0.99999999) == 1


def test_select_worker_eq3():
    q = [3, 0, 2, 5, 1]
    t = [1.0, 2.0, 1.0, 0.1, 4.0]
    lv = [1, 0, 1, 1, 1]
    assert C.select_worker(q, t, lv, 1) == 3        # 0.5 beats 3, 2 and 4
    assert C.select_worker(q, t, lv, 0) == 1
    assert C.select_worker(q, t, lv, 2) == -1
    assert C.select_worker([2, 1, 2], [1.0, 2.0, 1.0], [0, 0, 0], 0) == 0   # tie -> lowest index
