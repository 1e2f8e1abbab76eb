"""GPU parity of the relative-action buffer (ravel_set_relative_dims + ravel_step_state)
against the CPU oracle (App. B.1 / B.3: clean targets absolute, re-expressed against the
latest robot state around each pass; noise in model coordinates).

Bars: bit-exact for the analytic fields; 1e-4 (fp32) and 2e-2 (bf16) normwise relative
error on every released action and on the ring state for the transformer.
"""

import numpy as np
import pytest

import synth
from oracle.rolling import OracleRavel
from tests.harness import TOL_BF16, TOL_F32, GpuRoll, have_gpu, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads
MASK = np.array([1, 1, 0, 1, 0, 1, 1], dtype=np.int32)


def analytic(kind, H, D, B):
    return synth.RavelShape(layers=0, width=0, n_q_heads=1, n_kv_heads=1, head_dim=32, mlp_dim=0,
                            horizon=H, action_dim=D, prefix_len=0, n_fop=0, fop_obs_dim=0,
                            dtype=W.F32, model_kind=kind, batch=B, name="analytic")


def walk(steps, B, D, seed):
    rng = np.random.default_rng(seed)
    return np.cumsum(rng.standard_normal((steps, B, D)) * 0.2, axis=0).astype(np.float32)


def gstep(g, state, fop=None):
    st = g.torch.from_numpy(np.ascontiguousarray(state, dtype=np.float32)).to(g.dev)
    if fop is not None:
        g.fop.copy_(g.to_dev(fop))
    g.buf.step_state(g.fop, st, g.action)
    return g.action.cpu().numpy().copy()


def test_analytic_ot_roll_is_bit_exact_and_keeps_the_absolute_target():
    H, D, B = 8, 7, 2
    s = analytic(W.ANALYTIC_OT, H, D, B)
    target = np.random.default_rng(0).standard_normal(D).astype(np.float32)
    w = {"analytic.target": target}
    g = GpuRoll(s, w, B, 5)
    g.buf.set_relative_dims(MASK)
    o = OracleRavel(s, w, B, seed=5, dtype=np.float32)
    o.set_relative_dims(MASK)
    S = walk(4 * H, B, D, 1)
    for t in range(4 * H):
        a = gstep(g, S[t])
        b = o.step(state=S[t])
        assert np.array_equal(a, b), t
        if t >= H:
            np.testing.assert_allclose(a, np.broadcast_to(target, a.shape), atol=2e-5)
    X, tt, _ = g.state()
    assert np.array_equal(X, o.X)


def test_constant_state_is_the_ordinary_roll_plus_the_state():
    H, D, B = 6, 7, 2
    s = analytic(W.ANALYTIC_LINEAR, H, D, B)
    w = {"analytic.lambda": np.array([0.6], np.float32)}
    rel, ordinary = GpuRoll(s, w, B, 3), GpuRoll(s, w, B, 3)
    rel.buf.set_relative_dims(MASK)
    st = np.random.default_rng(2).standard_normal((B, D)).astype(np.float32)
    for _ in range(3 * H):
        a = gstep(rel, st)
        b = ordinary.step()
        assert np.array_equal(a, b + MASK.astype(np.float32) * st)  # fp32 sum, as released


def _transformer(name, B, steps, oracle_dtype, persistent=None, **replace):
    s = synth.get_config(name).replace(**replace) if replace else synth.get_config(name)
    mask = (np.arange(s.action_dim) % 3 != 2).astype(np.int32)
    wts = synth.draw_weights(s, seed=7, stress=True)
    g = GpuRoll(s, wts, B, 11)
    if persistent is not None:
        g.buf.set_option(g.rv.OPT_PERSISTENT, 1 if persistent else 0)
    g.buf.set_relative_dims(mask)
    o = OracleRavel(s, wts, B, seed=11, dtype=oracle_dtype)
    o.set_relative_dims(mask)
    for e in range(B):
        k, v = synth.draw_context(s, 0, e, 0)
        g.set_context(e, k, v, 0)
        o.set_context(e, k, v, 0)
    S = walk(steps, B, s.action_dim, 3)
    tol = TOL_F32 if s.dtype == W.F32 else TOL_BF16
    worst = 0.0
    for t in range(steps):
        z = synth.draw_fop_tokens(s, 0, t, batch=B) if s.n_fop > 0 else None
        a = gstep(g, S[t], z)
        b = o.step(z, state=S[t])
        err = rel_err(a, b)
        worst = max(worst, err)
        assert err <= tol, f"step {t}: action error {err:.3e}"
    X, _, _ = g.state()
    assert rel_err(X, o.X) <= tol
    return worst


def test_tiny_fp32_relative_roll_matches_oracle():
    print("tiny_fp32", _transformer("tiny_fp32", 1, 40, np.float64))


@pytest.mark.parametrize("persistent", [False, True])
def test_small_bf16_relative_roll_matches_oracle(persistent):
    print("small_bf16", persistent, _transformer("small_bf16", 2, 24, np.float64, persistent=persistent, layers=2))


def test_save_load_resumes_bit_exact_with_relative_state():
    H, D, B = 6, 7, 2
    s = analytic(W.ANALYTIC_OT, H, D, B)
    w = {"analytic.target": np.linspace(-1, 1, D).astype(np.float32)}
    a, b = GpuRoll(s, w, B, 8), GpuRoll(s, w, B, 8)
    a.buf.set_relative_dims(MASK)
    b.buf.set_relative_dims(MASK)
    S = walk(20, B, D, 4)
    for t in range(10):
        gstep(a, S[t])
    blob = a.buf.save()
    b.buf.load(blob)
    for t in range(10, 20):
        assert np.array_equal(gstep(a, S[t]), gstep(b, S[t])), t


def test_relative_mode_errors():
    H, D, B = 4, 7, 1
    s = analytic(W.ANALYTIC_LINEAR, H, D, B)
    w = {"analytic.lambda": np.array([0.5], np.float32)}
    g = GpuRoll(s, w, B, 0)
    st = np.zeros((B, D), np.float32)
    with pytest.raises(g.rv.RavelError) as ei:
        gstep(g, st)  # no relative dimensions set
    assert ei.value.status == -5
    g.buf.set_relative_dims(MASK)
    with pytest.raises(g.rv.RavelError) as ei:
        g.step()  # relative actions need the state
    assert ei.value.status == -5
    gstep(g, st)
    with pytest.raises(g.rv.RavelError) as ei:
        g.buf.set_relative_dims(MASK)  # after the first step
    assert ei.value.status == -5
