"""Pins for the oracle's random numbers: Philox4x32-10 known-answer vectors
(SC'11 reference implementation) and the 24-bit uniform mapping."""
import os

import numpy as np
import pytest
from scipy import stats

import oracle


def _kat(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = [int(t, 16) for t in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox_known_answers(golden_dir):
    rows = _kat(golden_dir)
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = oracle.philox4x32_10(ctr, key)
        assert [int(v) for v in got] == want


def test_gibbs_uniform_is_word_of_block():
    # replica r of column g uses word r&3 of the block at counter
    # {g, node, r>>2, sweep}; U24 = (w>>8) * 2^-24
    seed = 0x0123456789ABCDEF
    for g in [0, 1, 2, 3, 4, 7, 1 << 20, (1 << 32) - 1]:
        for r in [0, 1, 2, 3, 4, 7, 9, 37]:
            blk = oracle.philox4x32_10([g, 9, (r >> 2) | (0 << 24), 17],
                                       [seed & 0xFFFFFFFF, seed >> 32])
            u = oracle.gibbs_uniform(seed, 9, r, g, 17)
            assert u == (int(blk[r & 3]) >> 8) / 2.0 ** 24
            assert 0.0 <= u < 1.0


def test_gibbs_uniforms_distinct_across_replicas_and_columns():
    # every (replica, column) pair of a node and sweep gets its own word
    seed = 99
    us = {(r, g): oracle.gibbs_uniform(seed, 4, r, g, 2) for r in range(12) for g in range(50)}
    assert len(set(us.values())) == len(us)


def test_uniform_chi_square():
    seed = 151106416
    us = np.array([oracle.gibbs_uniform(seed, 1, 0, g, 0) for g in range(40000)])
    hist, _ = np.histogram(us, bins=40, range=(0.0, 1.0))
    _, p = stats.chisquare(hist)
    assert p > 1e-4
    # U24 values are exact multiples of 2^-24
    assert np.all(us * 2 ** 24 == np.floor(us * 2 ** 24))


@pytest.mark.parametrize("field", ["node", "replica", "sweep", "seed"])
def test_streams_differ(field):
    base = dict(seed=7, node=2, replica=1, gcol=100, sweep_id=4)
    a = oracle.gibbs_uniform(**base)
    alt = dict(base)
    alt[{"node": "node", "replica": "replica", "sweep": "sweep_id", "seed": "seed"}[field]] += 1
    b = oracle.gibbs_uniform(**alt)
    assert a != b
