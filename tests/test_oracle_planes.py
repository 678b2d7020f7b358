"""Pins of the oracle's seeded hash planes (Section 3.2.2 draws the hash's
hyperplanes at random; a caller that passes no planes gets them from a seed).

The counter-based generator is checked word for word against numpy's own
Philox4x64-10, an independent implementation of the same published
generator; the normal deviates against the polar identities of the
Box-Muller transform, evaluated on numpy's words, and against the standard
normal distribution.  CPU only.
"""
import math

import numpy as np
import pytest
from scipy import stats

import oracle

MASK = (1 << 64) - 1


def _words(x, count):
    return [(x >> (64 * i)) & MASK for i in range(count)]


@pytest.mark.parametrize("key,counter", [
    (0, 0),
    ((1 << 64) + 5, (3 << 64) + 7),
    (0x0123456789ABCDEF, 0xFEDCBA9876543210),
    (MASK, MASK),  # the counter's first word carries into the second
])
def test_generator_matches_numpy_philox(key, counter):
    # numpy advances its 256-bit counter before it draws each block
    raw = np.random.Philox(key=key, counter=counter).random_raw(12)
    for blk in range(3):
        c = (counter + 1 + blk) % (1 << 256)
        got = oracle.philox4x64_10(_words(c, 4), _words(key, 2))
        assert [int(x) for x in got] == [int(x) for x in raw[4 * blk: 4 * blk + 4]]


def test_planes_are_box_muller_pairs_of_the_generator_words():
    seed, heads, n_bits, d = 0x2007048250, 2, 5, 32
    planes = oracle.planes_from_seed(seed, heads, n_bits, d).reshape(-1)
    # blocks for counters 0, 1, ...: numpy starts one below the first counter
    raw = np.random.Philox(key=seed, counter=(1 << 256) - 1).random_raw(planes.size)
    for i in range(0, planes.size, 2):
        # entries i, i + 1 (i even) are the pair made from words i, i + 1
        u1 = ((int(raw[i]) >> 11) + 1) * 2.0 ** -53
        u2 = (int(raw[i + 1]) >> 11) * 2.0 ** -53
        z0, z1 = planes[i], planes[i + 1]
        r2 = -2.0 * math.log(u1)
        assert abs(z0 * z0 + z1 * z1 - r2) <= 1e-6 * r2 + 1e-12, i
        if r2 > 1e-6:
            diff = (math.atan2(z1, z0) - 2.0 * math.pi * u2) % (2.0 * math.pi)
            assert min(diff, 2.0 * math.pi - diff) < 1e-6, i


def test_planes_are_standard_normal_fp32_values():
    heads, n_bits, d = 8, 64, 64
    for seed in (1, 7, 0xFFFFFFFFFFFFFFFF):
        x = oracle.planes_from_seed(seed, heads, n_bits, d).reshape(-1)
        m = x.size
        assert np.array_equal(x, x.astype(np.float32).astype(np.float64))
        assert abs(x.mean()) < 5.0 / math.sqrt(m)
        assert abs(x.var() - 1.0) < 5.0 * math.sqrt(2.0 / m)
        assert stats.kstest(x, "norm").pvalue > 1e-4
        # the heads are drawn from disjoint counters: no two share a plane
        per_head = x.reshape(heads, -1)
        assert np.abs(np.corrcoef(per_head)[np.triu_indices(heads, 1)]).max() < 0.05


def test_planes_depend_on_the_seed_only():
    a = oracle.planes_from_seed(42, 3, 63, 32)
    b = oracle.planes_from_seed(42, 3, 63, 32)
    c = oracle.planes_from_seed(43, 3, 63, 32)
    assert np.array_equal(a, b)
    assert np.mean(a == c) < 0.01
    # a prefix of the flat order does not depend on the shape asked for
    small = oracle.planes_from_seed(42, 1, 7, 32).reshape(-1)
    assert np.array_equal(small, a.reshape(-1)[:small.size])
