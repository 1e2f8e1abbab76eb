"""Pins of the relative-action buffer (App. B.1 / B.3: clean targets kept absolute,
converted relative to the latest state around each expert pass, noise in model
coordinates).

* with a constant state nothing is re-expressed: the roll is the ordinary roll and
  every released action is the ordinary one plus the state on the relative dimensions;
* an OT field aimed at a fixed absolute target (relative to the current state on the
  relative dimensions) releases exactly that target in steady state while the state
  wanders, and every slot stays on the straight path tau eps + (1 - tau)(a* - s) in
  the current state's coordinates -- the conversion preserves the intended targets
  (the paper's stated purpose); switching the conversion off (planted mistake)
  leaves the slots' clean parts relative to stale states;
* dimensions outside the mask never see the state.
"""

import numpy as np
import pytest

import synth
from oracle.philox import ring_noise
from oracle.rolling import OracleRavel


def shape(kind, H=8, D=5, B=2):
    return synth.RavelShape(layers=0, width=0, n_q_heads=1, n_kv_heads=1, head_dim=1, mlp_dim=0,
                            horizon=H, action_dim=D, prefix_len=0, n_fop=0, fop_obs_dim=0,
                            dtype=synth.workloads.F32, model_kind=kind, batch=B, name="analytic")


MASK = np.array([1, 1, 0, 1, 0], dtype=np.float64)


def states(steps, B=2, D=5, seed=0):
    rng = np.random.default_rng(seed)
    return np.cumsum(rng.standard_normal((steps, B, D)) * 0.3, axis=0)


def test_constant_state_is_the_ordinary_roll_plus_the_state():
    s = shape(synth.workloads.ANALYTIC_LINEAR)
    w = {"analytic.lambda": np.array([0.6])}
    ordinary, rel = OracleRavel(s, w, 2, seed=4), OracleRavel(s, w, 2, seed=4)
    rel.set_relative_dims(MASK)
    st = np.random.default_rng(1).standard_normal((2, 5))
    for _ in range(20):
        a = ordinary.step()
        b = rel.step(state=st)
        np.testing.assert_array_equal(b, a + MASK * st)
    np.testing.assert_array_equal(rel.X, ordinary.X)


@pytest.mark.parametrize("H", [1, 4, 10])
def test_conversion_keeps_absolute_targets_under_a_moving_state(H):
    s = shape(synth.workloads.ANALYTIC_OT, H=H)
    target = np.array([0.5, -1.0, 2.0, 0.25, -0.75])
    o = OracleRavel(s, {"analytic.target": target}, 2, seed=9)
    o.set_relative_dims(MASK)
    S = states(3 * H + 6)
    for t in range(3 * H + 6):
        act = o.step(state=S[t])
        if t >= H:
            np.testing.assert_allclose(act, np.broadcast_to(target, act.shape), rtol=0, atol=1e-12)


def _straight_path_error(o, target, state, seed):
    """Largest distance of the buffer from tau_i eps_r + (1 - tau_i)(a* - s) over
    slots appended after the start (logical slot i holds action r = t + i)."""
    H, D = o.H, o.s.action_dim
    tau = (np.arange(H) + 1.0) / H
    X = o.logical_state()
    worst = 0.0
    for e in range(o.B):
        rel_target = target - MASK * state[e]
        for i in range(H):
            eps = ring_noise(seed, e, o.t + i, D).astype(np.float64)
            want = tau[i] * eps + (1 - tau[i]) * rel_target
            worst = max(worst, np.abs(X[e, i] - want).max())
    return worst


@pytest.mark.parametrize("planted", [False, True])
def test_buffer_stays_on_the_straight_path_to_the_absolute_target(planted):
    H = 6
    s = shape(synth.workloads.ANALYTIC_OT, H=H)
    target = np.array([0.5, -1.0, 2.0, 0.25, -0.75])
    o = OracleRavel(s, {"analytic.target": target}, 2, seed=9)
    o.set_relative_dims(MASK)
    S = states(4 * H)
    worst = 0.0
    for t in range(4 * H):
        if planted:
            o.has_prev[:] = False  # planted mistake: never re-express the buffer
        o.step(state=S[t])
        if t >= 2 * H:
            worst = max(worst, _straight_path_error(o, target, S[t], 9))
    if planted:
        assert worst > 1e-2
    else:
        assert worst < 1e-12


def test_absolute_dimensions_never_see_the_state():
    s = shape(synth.workloads.ANALYTIC_LINEAR)
    w = {"analytic.lambda": np.array([0.9])}
    a, b = OracleRavel(s, w, 2, seed=2), OracleRavel(s, w, 2, seed=2)
    a.set_relative_dims(MASK)
    b.set_relative_dims(MASK)
    S1, S2 = states(15, seed=1), states(15, seed=2)
    S2[..., MASK == 1] = S1[..., MASK == 1]  # states differ on absolute dimensions only
    for t in range(15):
        np.testing.assert_array_equal(a.step(state=S1[t]), b.step(state=S2[t]))
