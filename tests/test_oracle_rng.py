"""Pins of the oracle's counter-based generator (Philox4x32-10, Salmon et al. SC'11)."""
import os

import numpy as np
import pytest
from scipy import stats

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLD):
        if line.startswith("#") or not line.strip():
            continue
        w = [int(x, 16) for x in line.split()]
        rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,want", _kat())
def test_philox_known_answers(ctr, key, want):
    assert [int(x) for x in oracle.philox4x32_10(ctr, key)] == want


def test_uniform_counter_contract():
    # key = (lo32(seed), hi32(seed)); counter = (idx >> 2, row, req_id, tag); word idx & 3
    seed = 0x0123456789ABCDEF
    for (req, tag, row, idx) in [(0, 1, 0, 0), (7, 2, 3, 5), (123456, 2, 16, 128255), (5, 1, 9, 2)]:
        w = oracle.philox4x32_10([idx >> 2, row, req, tag], [seed & 0xFFFFFFFF, seed >> 32])[idx & 3]
        want = (2 * (int(w) >> 9) + 1) / 2.0 ** 24
        assert oracle.uniform(seed, req, tag, row, idx) == np.float32(want)


def test_uniform_grid_and_uniformity():
    n = 1 << 20
    u = oracle.uniform_array(99, 3, 2, 7, n)
    assert u.min() > 0.0 and u.max() < 1.0
    odd = u.astype(np.float64) * 2.0 ** 24          # exact odd integers: the 2^23-cell midpoint grid
    assert np.all(odd == np.round(odd)) and np.all(np.round(odd) % 2 == 1)
    counts = np.bincount((u * 256).astype(np.int64), minlength=256)
    chi2 = ((counts - n / 256) ** 2 / (n / 256)).sum()
    assert stats.chi2.sf(chi2, 255) > 1e-4
    # consecutive words are not trivially correlated
    r = np.corrcoef(u[:-1], u[1:])[0, 1]
    assert abs(r) < 5e-3
