"""The library's routing control plane (argus_oda, argus_route, argus_select_worker:
host code, no GPU) against the oracle (oracle.control) on the same seeded inputs:
PASM within 1e-12 (fp64, different summation order), routing and worker choice
identical; argument errors rejected."""

import numpy as np
import pytest

from oracle import control as OC
from paper_2511_06724_amd import dn


def _instance(rng, n):
    H = rng.dirichlet(np.ones(n) * 0.7)
    F = rng.dirichlet(np.ones(n) * 0.7)
    H[rng.random(n) < 0.2] = 0.0
    if H.sum() == 0:
        H[rng.integers(n)] = 1.0
    H /= H.sum()
    F *= H.sum() / F.sum()
    return H, F


def test_oda_matches_oracle():
    rng = np.random.default_rng(17)
    for n in list(range(1, 11)) + [6] * 20 + [64]:
        for _ in range(20):
            H, F = _instance(rng, n)
            T = dn.oda(H, F)
            R = OC.oda(H, F)
            assert np.allclose(T, R, rtol=0, atol=1e-12), n
            assert np.allclose(H @ T, F, atol=1e-12)


def test_oda_six_k_levels_example():
    """Six approximate-caching levels K = 0, 5, ..., 25: demand skewed to small K,
    the solver's split (high load) skewed to large K; every prompt moves to a faster
    level at most as far as needed, and the served split is F."""
    H = np.array([0.30, 0.25, 0.20, 0.10, 0.10, 0.05])
    F = np.array([0.05, 0.10, 0.15, 0.20, 0.25, 0.25])
    T = dn.oda(H, F)
    assert np.allclose(T, OC.oda(H, F), atol=1e-12)
    assert np.allclose(H @ T, F, atol=1e-12)
    assert np.allclose(np.tril(T, -1), 0.0)          # under this load nothing moves to a slower level


def test_route_and_select_match_oracle():
    rng = np.random.default_rng(23)
    for _ in range(200):
        n = int(rng.integers(1, 9))
        H, F = _instance(rng, n)
        T = OC.oda(H, F)
        lvl = int(rng.integers(0, n))
        for u in rng.random(8):
            assert dn.route(T, lvl, float(u)) == OC.route(T, lvl, float(u))
        nw = int(rng.integers(1, 12))
        q = rng.integers(0, 6, nw)
        t = rng.choice([0.5, 1.0, 2.0], nw)
        wl = rng.integers(0, n, nw)
        for level in range(n + 1):
            assert dn.select_worker(q, t, wl, level) == OC.select_worker(q, t, wl, level)


def test_control_argument_errors():
    with pytest.raises(dn.DnError):
        dn.oda([0.5, 0.5], [0.5, 0.6])           # different totals
    with pytest.raises(dn.DnError):
        dn.oda([0.0, 0.0], [0.0, 0.0])           # empty demand
    with pytest.raises(dn.DnError):
        dn.oda([-0.1, 1.1], [0.5, 0.5])
    with pytest.raises(dn.DnError):
        dn.oda(np.full(65, 1 / 65), np.full(65, 1 / 65))
    T = np.eye(3)
    for lvl, u in ((3, 0.5), (-1, 0.5), (0, 1.0), (0, -0.1)):
        with pytest.raises(dn.DnError):
            dn.route(T, lvl, u)
    with pytest.raises(dn.DnError):
        dn.select_worker([1, -1], [1.0, 1.0], [0, 0], 0)
