"""Pins of the streaming-aligned training objective (Sec. 3.3, Eq. 5 and 6).

* the conditional-OT field aimed at the sample's own target, v = (x - a_hat)/tau,
  is exactly the flow-matching target eps - a_hat on every slot of the training
  buffer, so its loss is 0 (pins the buffer's mixing weights and the target);
* a linear field gives the closed form mean_i ||lambda a_i - (eps_i - a_hat_i)||^2;
* the paper's own convention (tau_k = 1 - k/K, buffer (1 - tau_k) eps + tau_k a_hat,
  target a_hat - eps, velocity of the opposite sign) gives the same loss;
* the buffer of slot H-1 is pure noise and the expert sees delta = p / K.
"""

import numpy as np
import pytest

import oracle.training as tr
import synth
from oracle.expert import Expert


def sample(H=10, D=4, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((H, D)), rng.standard_normal((H, D))


@pytest.mark.parametrize("H", [1, 3, 10, 50])
def test_ot_field_towards_the_target_has_zero_loss(H):
    target, noise = sample(H, 5, H)
    tau = (np.arange(H) + 1.0) / H
    loss, v = tr.training_loss(lambda a: (a - target) / tau[:, None], target, noise)
    np.testing.assert_allclose(v, noise - target, rtol=0, atol=1e-12)
    assert loss < 1e-24


def test_linear_field_closed_form():
    lam = 0.6
    target, noise = sample(7, 3, 1)
    tau = (np.arange(7) + 1.0) / 7
    a = tau[:, None] * noise + (1 - tau[:, None]) * target
    want = np.mean(np.sum((lam * a - (noise - target)) ** 2, axis=1))
    loss, _ = tr.training_loss(lambda x: lam * x, target, noise)
    assert abs(loss - want) <= 1e-14 * max(1.0, want)


def test_paper_convention_gives_the_same_loss():
    H = 10
    target, noise = sample(H, 4, 2)
    rng = np.random.default_rng(3)
    M = rng.standard_normal((4, 4))
    field = lambda a: a @ M  # any velocity field of this repository's convention
    loss, _ = tr.training_loss(field, target, noise)
    k = np.arange(1, H + 1)
    tau_p = 1.0 - k / H  # the paper's profile
    a_p = (1.0 - tau_p)[:, None] * noise + tau_p[:, None] * target
    v_p = -field(a_p)  # the paper's velocity points from noise to data
    loss_p = np.mean(np.sum((v_p - (target - noise)) ** 2, axis=1))
    assert abs(loss - loss_p) <= 1e-12 * loss_p
    # and its buffer is this repository's buffer slot for slot
    np.testing.assert_allclose(a_p, tr.training_buffer(target, noise), rtol=0, atol=1e-15)


def test_last_slot_is_pure_noise_and_first_is_nearly_clean():
    target, noise = sample(8, 3, 4)
    a = tr.training_buffer(target, noise)
    np.testing.assert_array_equal(a[-1], noise[-1])
    np.testing.assert_allclose(a[0], (noise[0] + 7 * target[0]) / 8, rtol=1e-15)


def test_offset_conditioning_is_p_over_K_without_the_lead_bias():
    s = synth.get_config("tiny_fp32").replace(delta_bias=0.3)
    w = synth.draw_weights(s, seed=1, stress=True)
    ex = Expert(s, w)
    k, v = synth.draw_context(s, 0, 0, 0)
    z = synth.draw_fop_tokens(s, 0, 0)[0]
    target, noise = sample(s.horizon, s.action_dim, 5)
    a = tr.training_buffer(target, noise)
    got = tr.expert_velocity(ex, k, v, 3, z)(a)
    np.testing.assert_array_equal(got, ex.velocity(a, k, v, 3 / s.horizon, z))
    assert np.abs(got - ex.velocity(a, k, v, 3 / s.horizon + 0.3, z)).max() > 1e-6
