"""Pins of the oracle's Philox4x32-10 stream (no GPU).

* known-answer vectors published with Random123 (Salmon et al., SC'11);
* uniform and normal outputs pass distribution tests;
* different tags / slots / rounds give uncorrelated streams.
"""
import os

import numpy as np
import pytest
from scipy import stats

from oracle import philox


def _kat_rows(golden_dir):
    rows = []
    with open(os.path.join(golden_dir, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_known_answer_vectors(golden_dir):
    rows = _kat_rows(golden_dir)
    assert len(rows) == 3
    for ctr, key, expect in rows:
        got = philox.philox4x32_10(np.array(ctr), np.array(key))
        assert [int(x) for x in got] == expect


def test_uniform_range_and_distribution():
    w = philox.words(7, np.arange(25000), 3, 11, philox.TAG_COIN, 0).reshape(-1)
    u = philox.word_to_uniform(w)
    assert u.min() > 0.0 and u.max() < 1.0
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    # extreme words map strictly inside (0, 1)
    assert philox.word_to_uniform(np.array([0], np.uint64))[0] == 0.5 * 2.0 ** -24
    assert philox.word_to_uniform(np.array([0xFFFFFFFF], np.uint64))[0] == 1.0 - 2.0 ** -25


def test_normals_distribution():
    z = philox.normal_vector(123, 5, 2, philox.TAG_DRAFT, 3, 100003)
    assert z.shape == (100003,)
    assert abs(z.mean()) < 4.0 / np.sqrt(z.size)
    assert abs(z.var() - 1.0) < 4.0 * np.sqrt(2.0 / z.size)
    assert stats.kstest(z, "norm").pvalue > 1e-3


def test_stream_layout_element_to_counter():
    # element e of a normal vector comes from counter c0 = e >> 2, output e & 3
    d = 10
    z = philox.normal_vector(9, 1, 2, philox.TAG_RESID, 0, d)
    for e in range(d):
        w = philox.words(9, e >> 2, 1, 2, philox.TAG_RESID, 0)
        assert z[e] == philox.words_to_normals(w)[e & 3]


@pytest.mark.parametrize("other", [
    dict(tag=philox.TAG_TARGET, slot=0, rnd=4),
    dict(tag=philox.TAG_DRAFT, slot=2, rnd=4),
    dict(tag=philox.TAG_DRAFT, slot=1, rnd=5),
])
def test_streams_independent(other):
    a = philox.normal_vector(1, 0, 4, philox.TAG_DRAFT, 1, 40000)
    b = philox.normal_vector(1, 0, other["rnd"], other["tag"], other["slot"], 40000)
    assert abs(np.corrcoef(a, b)[0, 1]) < 4.0 / np.sqrt(40000)
