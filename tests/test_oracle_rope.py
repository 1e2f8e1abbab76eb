"""Optional rotary position embedding of the buffer tokens (the paper uses none, its
slots are told apart by their flow time): pins of the oracle's rotation and of its
place in the self-attention."""

import numpy as np

import synth
from oracle import expert as ex

W_ = synth.workloads


def shape(**kw):
    base = dict(layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8, mlp_dim=48, horizon=6, action_dim=5,
                prefix_len=7, n_fop=3, fop_obs_dim=9, dtype=W_.F32, rope_base=100.0, name="rope")
    base.update(kw)
    return synth.RavelShape(**base)


def _weights(s, seed=0):
    return {k: v.astype(np.float64) for k, v in synth.draw_weights(s, seed=seed, stress=True).items()}


def _inputs(s, seed):
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((s.horizon, s.action_dim))
    k = rng.standard_normal((s.layers, s.prefix_len, s.n_kv_heads, s.head_dim))
    v = rng.standard_normal((s.layers, s.prefix_len, s.n_kv_heads, s.head_dim))
    z = rng.standard_normal((s.n_fop, s.width))
    return a, k, v, z


def test_rotation_is_a_complex_phase_per_pair():
    """Pair d of a head, read as the complex number x_d + i x_{d+hd/2}, is multiplied
    by exp(i pos base^(-2d/hd)): position 0 is the identity, norms are kept and two
    rotations compose by adding positions."""
    rng = np.random.default_rng(1)
    hd, nh, base = 16, 3, 500.0
    x = rng.standard_normal((5, nh * hd))
    pos = np.array([0, 1, 7, 40, 913])
    got = ex.rope_rotate(x, pos, nh, hd, base)
    half = hd // 2
    for j in range(nh):
        z = x[:, j * hd:j * hd + half] + 1j * x[:, j * hd + half:(j + 1) * hd]
        zr = z * np.exp(1j * pos[:, None] * base ** (-np.arange(half) * 2.0 / hd))
        np.testing.assert_allclose(got[:, j * hd:j * hd + half], zr.real, rtol=0, atol=1e-12)
        np.testing.assert_allclose(got[:, j * hd + half:(j + 1) * hd], zr.imag, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(got[0], x[0])
    np.testing.assert_allclose(np.linalg.norm(got.reshape(5, nh, hd), axis=2),
                               np.linalg.norm(x.reshape(5, nh, hd), axis=2), rtol=1e-12)
    twice = ex.rope_rotate(ex.rope_rotate(x, pos, nh, hd, base), pos + 3, nh, hd, base)
    np.testing.assert_allclose(twice, ex.rope_rotate(x, 2 * pos + 3, nh, hd, base), rtol=0, atol=1e-10)


def test_scores_depend_only_on_relative_positions():
    """Without a prefix the buffer attends only to itself: moving every slot by the same
    number of positions leaves the velocity unchanged (rotating queries and keys alike),
    while a model with the rotation differs from one without it."""
    s = shape(prefix_len=0)
    W = _weights(s)
    a, _, _, z = _inputs(s, 2)
    e = ex.Expert(s, W)
    v0 = e.velocity(a, None, None, 0.3, z, pos0=0)
    np.testing.assert_allclose(e.velocity(a, None, None, 0.3, z, pos0=11), v0, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(e.velocity(a, None, None, 0.3, z, pos0=123), v0, rtol=1e-10, atol=1e-12)
    plain = ex.Expert(s.replace(rope_base=0.0), W).velocity(a, None, None, 0.3, z)
    assert np.abs(plain - v0).max() / np.abs(v0).max() > 1e-2


def test_prefix_keys_are_used_as_given_and_slots_follow_the_prefix():
    """With a prefix, the buffer sits at positions P .. P + H - 1 after it: the default
    equals an explicit pos0 = P, and other placements change the output (the prefix
    keys are not rotated, so absolute positions matter)."""
    s = shape()
    W = _weights(s)
    a, k, v, z = _inputs(s, 3)
    e = ex.Expert(s, W)
    v_def = e.velocity(a, k, v, 0.4, z)
    np.testing.assert_array_equal(e.velocity(a, k, v, 0.4, z, pos0=s.prefix_len), v_def)
    assert np.abs(e.velocity(a, k, v, 0.4, z, pos0=0) - v_def).max() / np.abs(v_def).max() > 1e-3


def test_one_slot_without_prefix_ignores_the_rotation():
    """A single slot and no prefix: its query meets only its own key at relative position
    0, so every rotation base gives the unrotated model's velocity."""
    s = shape(prefix_len=0, horizon=1)
    W = _weights(s)
    a, _, _, z = _inputs(s, 4)
    ref = ex.Expert(s.replace(rope_base=0.0), W).velocity(a, None, None, 0.5, z)
    for base in (10.0, 10000.0):
        got = ex.Expert(s.replace(rope_base=base), W).velocity(a, None, None, 0.5, z, pos0=37)
        np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)
