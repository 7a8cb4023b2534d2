"""Pins of the oracle's similarity-driven approximation level (lookup.select_k):
brute force over the boundary cosines of a threshold table, monotonicity, and the
degenerate cases (no thresholds, nothing retrieved)."""

import numpy as np
import pytest

from oracle import lookup

THR = [0.80, 0.85, 0.90, 0.93, 0.96]
LEV = [0, 5, 10, 15, 20, 25]


def test_select_k_at_and_around_every_threshold():
    """A score equal to a threshold takes that threshold's level; the next fp32 value
    below it stays one level down; the next above stays at the level."""
    for i, t in enumerate(THR):
        t32 = np.float32(t)
        below = np.nextafter(t32, np.float32(-1))
        above = np.nextafter(t32, np.float32(2))
        got = lookup.select_k(np.array([below, t32, above], np.float32), THR, LEV)
        assert list(got) == [LEV[i], LEV[i + 1], LEV[i + 1]], (t, got)


def test_select_k_brute_force_and_monotone():
    rng = np.random.default_rng(3)
    s = np.concatenate([rng.uniform(-1, 1, 2000), rng.uniform(0.78, 0.98, 2000)]).astype(np.float32)
    got = lookup.select_k(s, THR, LEV)
    # brute force: the largest level whose threshold the score reaches
    t32 = np.asarray(THR, np.float32)
    ref = np.array([LEV[int(np.sum(v >= t32))] for v in s], np.int32)
    assert np.array_equal(got, ref)
    order = np.argsort(s, kind="stable")
    assert np.all(np.diff(got[order]) >= 0)          # more similar never gets a smaller K
    assert got[s < t32[0]].max() == 0 and got[s >= t32[-1]].min() == 25


def test_select_k_degenerate_tables_and_missing_rows():
    s = np.array([np.nan, -1.0, 0.5, 1.0], np.float32)
    assert list(lookup.select_k(s, [], [7])) == [0, 7, 7, 7]     # no thresholds: one level
    assert list(lookup.select_k(s, THR, LEV)) == [0, 0, 0, 25]   # nothing retrieved -> K = 0
    with pytest.raises(ValueError):
        lookup.select_k(s, THR, LEV[:-1])
