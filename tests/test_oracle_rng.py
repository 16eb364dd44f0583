"""Pins of the oracle's initial-factor generator.

SplitMix64 is checked against the published output sequence of its reference
implementation (state 1234567); Box-Muller against the normal distribution.
"""

import math

import numpy as np
import pytest
from scipy import stats

from oracle import rng


def test_splitmix64_published_sequence():
    assert rng.splitmix64_stream(1234567, 5) == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]


def test_vectorised_mix_matches_scalar():
    xs = [0, 1, 2, 1234567, (1 << 64) - 1, 0x9E3779B97F4A7C15]
    v = rng._mix_vec(np.array(xs, dtype=np.uint64))
    assert [int(a) for a in v] == [rng.mix(x) for x in xs]


def test_uniform_ranges_and_independence_of_keys():
    u1, u2 = rng.uniforms(0, 3, 1, 100000)
    assert u1.min() > 0 and u1.max() <= 1
    assert u2.min() >= 0 and u2.max() < 1
    # element i of the stream is a pure function of (seed, tensor, factor, i)
    a = rng.normals(7, 5, 0, 64)
    b = rng.normals(7, 5, 0, 1000)[:64]
    assert np.array_equal(a, b)
    assert not np.array_equal(rng.normals(7, 5, 0, 64), rng.normals(7, 5, 1, 64))
    assert not np.array_equal(rng.normals(7, 5, 0, 64), rng.normals(7, 6, 0, 64))
    assert not np.array_equal(rng.normals(7, 5, 0, 64), rng.normals(8, 5, 0, 64))


def test_box_muller_by_hand():
    u1, u2 = rng.uniforms(0, 0, 1, 3)
    z = rng.normals(0, 0, 1, 3)
    for k in range(3):
        ref = np.float32(math.sqrt(-2.0 * math.log(u1[k])) * math.cos(2.0 * math.pi * u2[k]))
        assert z[k] == ref


def test_normality():
    z = rng.normals(0, 11, 1, 200000).astype(np.float64)
    assert abs(z.mean()) < 5 / math.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * math.sqrt(2 / z.size)
    assert stats.kstest(z, "norm").pvalue > 1e-4


def test_init_factor_shape():
    q = rng.init_factor(0, 0, "Q", 576, 4)
    assert q.shape == (576, 4) and q.dtype == np.float32
    assert np.array_equal(q.reshape(-1), rng.normals(0, 0, 1, 576 * 4))


def test_step_keyed_stream_extends_the_initial_draw():
    """Step 0 of the step-keyed stream is the initial factor itself (the key's high half is
    zero); later steps give other, standard-normal streams, each a pure function of the step."""
    q0 = rng.init_factor(3, 7, "Q", 100, 8)
    assert np.array_equal(rng.fresh_factor(3, 7, "Q", 100, 8, 0), q0)
    assert rng.stream_key(3, 7, 1, 0) == rng.mix(3 ^ rng.mix(2 * 7 + 1))
    assert rng.stream_key(3, 7, 1, 5) == rng.mix(3 ^ rng.mix((5 << 32) + 2 * 7 + 1))
    f1 = rng.fresh_factor(3, 7, "Q", 100, 8, 1)
    f2 = rng.fresh_factor(3, 7, "Q", 100, 8, 2)
    assert not np.array_equal(f1, q0) and not np.array_equal(f1, f2)
    assert np.array_equal(f1, rng.fresh_factor(3, 7, "Q", 100, 8, 1))
    # (tensor, factor) pairs and steps never share a key: the low half holds 2 * tensor + f
    keys = {rng.stream_key(0, k, f, t) for k in range(4) for f in (0, 1) for t in range(4)}
    assert len(keys) == 32
    z = rng.normals(0, 11, 1, 200000, step=9).astype(np.float64)
    assert abs(z.mean()) < 5 / math.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * math.sqrt(2 / z.size)
    assert stats.kstest(z, "norm").pvalue > 1e-4
