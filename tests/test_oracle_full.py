"""Pins of the full-horizon synchronous baseline (Sec. 4.1, App. B.1): all slots
share one flow time and S Euler steps move the chunk from noise to clean.

* linear field v = lambda x: the chunk is scaled by (1 - lambda/S) per step, so
  it ends at (1 - lambda/S)^S eps (pins the step count and dt = 1/S);
* conditional-OT field v = (x - a*)/tau: after k steps the chunk sits at
  a* + (eps - a*)(S - k)/S on the straight path and lands exactly on a* (pins
  tau_s = (S - s)/S);
* one step on a one-slot chunk is one rolling update of a one-slot buffer
  (both evaluate the expert at tau = 1 and move by dt = 1);
* with one shared flow time and no positional encoding the slots are
  exchangeable: permuting the noise rows permutes the output rows.
"""

import numpy as np
import pytest

import oracle.full as full
import synth
from oracle.expert import Expert, flow_times
from oracle.rolling import OracleRavel


@pytest.mark.parametrize("S", [1, 3, 10, 50])
def test_linear_field_closed_form(S):
    lam = 0.9
    eps = np.random.default_rng(S).standard_normal((7, 5))
    got = full.full_denoise(lambda a, tau: lam * a, eps, S)
    np.testing.assert_allclose(got, (1.0 - lam / S) ** S * eps, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("S", [1, 4, 10])
def test_ot_field_follows_the_straight_path_and_lands_on_the_target(S):
    rng = np.random.default_rng(7)
    eps, target = rng.standard_normal((6, 4)), rng.standard_normal(4)
    seen = []

    def v(a, tau):
        seen.append(a.copy())
        return (a - target[None, :]) / tau

    got = full.full_denoise(v, eps, S)
    np.testing.assert_allclose(got, np.broadcast_to(target, got.shape), rtol=0, atol=1e-12)
    for k, a in enumerate(seen):
        np.testing.assert_allclose(a, target + (eps - target) * (S - k) / S, rtol=0, atol=1e-12)


def test_planted_mistakes_fail_the_closed_forms(monkeypatch):
    rng = np.random.default_rng(3)
    eps, target = rng.standard_normal((3, 2)), rng.standard_normal(2)
    S = 5
    # flow times shifted by one step: the OT field no longer lands on the target
    monkeypatch.setattr(full, "step_flow_times", lambda n: (n - np.arange(n, dtype=np.float64) + 1.0) / (n + 1.0))
    got = full.full_denoise(lambda a, tau: (a - target) / tau, eps, S)
    assert np.abs(got - target).max() > 1e-2


def test_explicit_flow_times_reproduce_the_rolling_profile():
    s = synth.get_config("tiny_fp32")
    w = synth.draw_weights(s, seed=1, stress=True)
    ex = Expert(s, w)
    k, v = synth.draw_context(s, 0, 0, 0)
    z = synth.draw_fop_tokens(s, 0, 0)[0]
    a = np.random.default_rng(2).standard_normal((s.horizon, s.action_dim))
    ref = ex.velocity(a, k, v, 0.25, z)
    got = ex.velocity(a, k, v, 0.25, z, taus=flow_times(s.horizon))
    np.testing.assert_array_equal(got, ref)


def test_one_step_on_one_slot_is_one_rolling_update():
    s = synth.get_config("tiny_fp32").replace(horizon=1)
    w = synth.draw_weights(s, seed=4, stress=True)
    k, v = synth.draw_context(s, 0, 0, 0)
    z = synth.draw_fop_tokens(s, 0, 0)
    o = OracleRavel(s, w, batch=1, seed=9)
    o.set_context(0, k, v, 0)
    noise = o.logical_state()[0]
    act = o.step(z)
    ex = Expert(s, w)
    got = full.full_denoise(full.expert_velocity(ex, k, v, z[0], delta=0.0 / s.horizon + s.delta_bias), noise, 1)
    np.testing.assert_allclose(got[0], act[0], rtol=1e-13, atol=1e-13)


def test_shared_flow_time_makes_slots_exchangeable():
    s = synth.get_config("tiny_fp32")
    w = synth.draw_weights(s, seed=5, stress=True)
    ex = Expert(s, w)
    k, v = synth.draw_context(s, 0, 0, 0)
    z = synth.draw_fop_tokens(s, 0, 0)[0]
    noise = np.random.default_rng(6).standard_normal((s.horizon, s.action_dim))
    perm = np.random.default_rng(8).permutation(s.horizon)
    vel = full.expert_velocity(ex, k, v, z)
    a = full.full_denoise(vel, noise, 4)
    b = full.full_denoise(vel, noise[perm], 4)
    np.testing.assert_allclose(b, a[perm], rtol=1e-10, atol=1e-12)
    # and the rolling profile (distinct flow times) does not have this symmetry
    r1 = ex.velocity(noise, k, v, 0.0, z)
    r2 = ex.velocity(noise[perm], k, v, 0.0, z)
    assert np.abs(r2 - r1[perm]).max() > 1e-6
