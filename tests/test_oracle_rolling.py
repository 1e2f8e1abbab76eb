"""Pins of the oracle's rolling buffer (Sec. 3.1 Eq. 3 and the release/append
rule after it; cold start of App. A.1; context reuse of Sec. 3.2).

Analytic velocity fields give closed forms for whole rolls:
* linear field v = lambda x: an action released at step r has been scaled by
  (1 - lambda/H) once per update, i.e. exactly min(r+1, H) times (App. A.1:
  one update for the first action, K in steady state);
* conditional-OT field v = (x - a*)/tau: a slot that starts as noise eps at
  tau = 1 and receives H updates lands exactly on a* (the straight path of
  flow matching, Sec. 3.3 Eq. 5 written in this repository's time direction).
"""

import numpy as np
import pytest

import synth
from oracle.philox import ring_noise
from oracle.rolling import OracleRavel


def analytic_shape(kind, H=8, D=7, B=2):
    return synth.RavelShape(layers=0, width=0, n_q_heads=1, n_kv_heads=1, head_dim=1, mlp_dim=0,
                            horizon=H, action_dim=D, prefix_len=0, n_fop=0, fop_obs_dim=0,
                            dtype=synth.workloads.F32, model_kind=kind, batch=B, name="analytic")


@pytest.mark.parametrize("H", [1, 5, 8, 16])
def test_linear_field_closed_form_counts_updates(H):
    lam = 0.7
    s = analytic_shape(synth.workloads.ANALYTIC_LINEAR, H=H, B=3)
    o = OracleRavel(s, {"analytic.lambda": np.array([lam])}, batch=3, seed=11)
    for r in range(3 * H + 5):
        act = o.step()
        n_upd = min(r + 1, H)
        for e in range(3):
            want = (1.0 - lam / H) ** n_upd * ring_noise(11, e, r, s.action_dim).astype(np.float64)
            np.testing.assert_allclose(act[e], want, rtol=1e-12, atol=1e-14)


def test_ot_field_releases_the_target_in_steady_state():
    H = 10
    s = analytic_shape(synth.workloads.ANALYTIC_OT, H=H, D=5, B=2)
    tgt = np.array([0.5, -1.0, 2.0, 0.0, 3.25])
    o = OracleRavel(s, {"analytic.target": tgt}, batch=2, seed=3)
    for r in range(4 * H):
        act = o.step()
        if r >= H:
            np.testing.assert_allclose(act, np.tile(tgt, (2, 1)), atol=1e-12)
        else:
            # cold start: action r starts as pure noise although its slot has
            # tau = (r+1)/H, then gets r+1 updates at tau = (r+1-m)/H; the last
            # cold-start action (r = H-1) starts at tau = 1 and lands on a*.
            eps = np.stack([ring_noise(3, e, r, 5) for e in range(2)]).astype(np.float64)
            x = eps.copy()
            for m in range(r + 1):
                tau = (r + 1 - m) / H
                x = x - (1.0 / H) * (x - tgt) / tau
            np.testing.assert_allclose(act, x, rtol=1e-12, atol=1e-12)
            if r == H - 1:
                np.testing.assert_allclose(act, np.tile(tgt, (2, 1)), atol=1e-12)


def test_ot_field_intermediate_slots_follow_the_straight_path():
    H = 6
    s = analytic_shape(synth.workloads.ANALYTIC_OT, H=H, D=3, B=1)
    tgt = np.array([1.0, 2.0, -1.0])
    o = OracleRavel(s, {"analytic.target": tgt}, batch=1, seed=0)
    for _ in range(2 * H):
        o.step()
    # at step t, logical slot i holds action r = t + i appended at step r - H with
    # m = H - 1 - i updates so far: x = a* + (eps - a*) (1 - m/H) = a* + (eps - a*) tau_i
    X = o.logical_state()[0]
    for i in range(H):
        r = o.t + i
        eps = ring_noise(0, 0, r, 3).astype(np.float64)
        tau = (i + 1) / H
        np.testing.assert_allclose(X[i], tgt + (eps - tgt) * tau, atol=1e-12)


def test_release_index_invariants():
    H, steps = 7, 40
    s = analytic_shape(synth.workloads.ANALYTIC_LINEAR, H=H, D=4, B=1)
    o = OracleRavel(s, {"analytic.lambda": np.array([0.0])}, batch=1, seed=5)
    # lambda = 0: actions are never changed, so every release is exactly the noise
    # drawn for action index r, which must come out at step r from slot r mod H
    for r in range(steps):
        slot = o.t % H
        before = o.X[0, slot].copy()
        act = o.step()
        assert np.array_equal(act[0], before)
        assert np.array_equal(act[0], ring_noise(5, 0, r, 4).astype(np.float64))
        assert np.array_equal(o.X[0, slot], ring_noise(5, 0, r + H, 4).astype(np.float64))


def test_float32_mode_is_float32_throughout():
    s = analytic_shape(synth.workloads.ANALYTIC_OT, H=8, D=7, B=1)
    o = OracleRavel(s, {"analytic.target": np.ones(7)}, batch=1, seed=0, dtype=np.float32)
    act = o.step()
    assert act.dtype == np.float32 and o.X.dtype == np.float32


def _tiny_transformer():
    s = synth.RavelShape(layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8, mlp_dim=48,
                         horizon=6, action_dim=5, prefix_len=7, n_fop=3, fop_obs_dim=9,
                         dtype=synth.workloads.F32, batch=2, name="pin")
    return s, synth.draw_weights(s, seed=1, stress=True)


def test_context_age_grows_until_a_new_context_is_published():
    s, W = _tiny_transformer()
    o = OracleRavel(s, W, batch=2, seed=0)
    k0, v0 = synth.draw_context(s, 0, 0, 0)
    for e in range(2):
        o.set_context(e, k0, v0, 0)
    deltas = []
    for t in range(5):
        o.step()
        deltas.append(o.offset(0))  # offset the next step would use
    assert deltas == pytest.approx([(t + 1) / 6 for t in range(5)])
    k1, v1 = synth.draw_context(s, 0, 0, 1)
    o.set_context(0, k1, v1, 3)  # computed from the observation at step 3
    o.step()  # applied at t = 5
    assert o.log[-1] == (0, 5, 3)
    assert o.offset(0) == pytest.approx((6 - 3) / 6)
    assert o.offset(1) == pytest.approx(6 / 6)
    with pytest.raises(ValueError):
        o.set_context(0, k1, v1, 2)


def test_no_context_is_an_error_for_the_transformer():
    s, W = _tiny_transformer()
    o = OracleRavel(s, W, batch=2, seed=0)
    with pytest.raises(RuntimeError):
        o.step()


def test_envs_are_independent():
    s, W = _tiny_transformer()
    rolls = []
    for batch in (2, 1):
        o = OracleRavel(s, W, batch=batch, seed=4)
        for e in range(batch):
            k, v = synth.draw_context(s, 0, e, 0)
            o.set_context(e, k, v, 0)
        outs = []
        for t in range(8):
            z = synth.draw_fop_tokens(s, 0, t, batch=2)[:batch]
            outs.append(o.step(z))
        rolls.append(np.stack(outs))
    np.testing.assert_array_equal(rolls[0][:, 0], rolls[1][:, 0])


def test_planted_mistakes_are_caught_by_the_closed_forms(monkeypatch):
    """A wrong Euler sign, a wrong dt or an off-by-one release breaks a pin."""
    import oracle.rolling as rl

    def run_linear():
        s = analytic_shape(synth.workloads.ANALYTIC_LINEAR, H=5, B=1)
        o = rl.OracleRavel(s, {"analytic.lambda": np.array([0.7])}, batch=1, seed=2)
        ok = True
        for r in range(12):
            act = o.step()
            want = (1 - 0.7 / 5) ** min(r + 1, 5) * ring_noise(2, 0, r, 7).astype(np.float64)
            ok &= np.allclose(act[0], want, rtol=1e-12)
        return ok

    assert run_linear()
    orig = rl.OracleRavel.velocity
    monkeypatch.setattr(rl.OracleRavel, "velocity", lambda self, *a, **k: -orig(self, *a, **k))
    assert not run_linear()
    monkeypatch.setattr(rl.OracleRavel, "velocity", orig)
    orig_noise = rl.ring_noise
    monkeypatch.setattr(rl, "ring_noise", lambda seed, e, r, d: orig_noise(seed, e, r + 1, d))
    assert not run_linear()
