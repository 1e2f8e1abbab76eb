"""Pins of the oracle's noise stream against published values and mathematics."""

import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle.philox import box_muller, philox4x32_10, ring_noise, uniform_angle, uniform_radius

GOLD = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        w = [int(x, 16) for x in line.split()]
        rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox_known_answer_vectors():
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = philox4x32_10(np.array(ctr), np.array(key))
        assert [int(x) for x in got] == want


def test_philox_vectorised_matches_scalar_calls():
    rng = np.random.default_rng(1)
    ctr = rng.integers(0, 2 ** 32, size=(64, 4), dtype=np.uint64)
    key = rng.integers(0, 2 ** 32, size=(2,), dtype=np.uint64)
    batch = philox4x32_10(ctr, key)
    for i in range(64):
        assert np.array_equal(batch[i], philox4x32_10(ctr[i], key))


def test_uniforms_are_exact_and_in_range():
    x = np.array([0, 255, 256, 0xFFFFFFFF], dtype=np.uint32)
    ua = uniform_radius(x)
    ub = uniform_angle(x)
    assert ua.tolist() == [2.0 ** -24, 2.0 ** -24, 2 * 2.0 ** -24, 1.0]
    assert ub.tolist() == [0.0, 0.0, 2.0 ** -24, 1.0 - 2.0 ** -24]
    # representable in float32 without rounding
    assert np.array_equal(ua.astype(np.float32).astype(np.float64), ua)


def test_box_muller_against_math_module():
    rng = np.random.default_rng(2)
    w = rng.integers(0, 2 ** 32, size=(200, 2), dtype=np.uint64).astype(np.uint32)
    c, s = box_muller(w[:, 0], w[:, 1])
    for i in range(200):
        ua = ((int(w[i, 0]) >> 8) + 1) / 16777216.0
        ub = (int(w[i, 1]) >> 8) / 16777216.0
        r = math.sqrt(-2.0 * math.log(ua))
        assert c[i] == pytest.approx(r * math.cos(2 * math.pi * ub), rel=1e-14, abs=1e-14)
        assert s[i] == pytest.approx(r * math.sin(2 * math.pi * ub), rel=1e-14, abs=1e-14)


def test_ring_noise_is_standard_normal():
    z = np.concatenate([ring_noise(7, e, r, 32) for e in range(4) for r in range(500)])
    assert z.dtype == np.float32
    assert abs(z.mean()) < 0.02
    assert abs(z.std() - 1.0) < 0.02
    assert stats.kstest(z.astype(np.float64), "norm").pvalue > 1e-3


def test_ring_noise_counter_layout():
    # element j uses counter (j // 4, env, r_lo, r_hi); elements of one group share a call
    seed, env, r = 0x1234_5678_9ABC, 3, (1 << 32) + 17
    z = ring_noise(seed, env, r, 7)
    words = philox4x32_10(np.array([1, env, 17, 1]), np.array([0x56789ABC, 0x1234]))
    rad = math.sqrt(-2.0 * math.log(((int(words[0]) >> 8) + 1) / 16777216.0))
    ang = 2 * math.pi * ((int(words[1]) >> 8) / 16777216.0)
    assert z[4] == np.float32(rad * math.cos(ang))
    assert z[5] == np.float32(rad * math.sin(ang))
    # streams differ by env, by r and by seed
    assert not np.array_equal(ring_noise(0, 0, 5, 8), ring_noise(0, 1, 5, 8))
    assert not np.array_equal(ring_noise(0, 0, 5, 8), ring_noise(0, 0, 6, 8))
    assert not np.array_equal(ring_noise(0, 0, 5, 8), ring_noise(1, 0, 5, 8))
    # a prefix of a longer draw equals a shorter draw
    assert np.array_equal(ring_noise(0, 2, 9, 32)[:7], ring_noise(0, 2, 9, 7))
