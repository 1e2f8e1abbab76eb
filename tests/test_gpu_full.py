"""GPU parity of the full-horizon synchronous baseline (ravel_full_denoise) against
the CPU oracle (oracle/full.py): every slot of a fresh chunk shares one flow time and
S Euler steps bring the chunk from noise to clean (Sec. 4.1, App. B.1).

Bars as for the rolling step: bit-exact for the analytic fields (same fp32 operations
in the same order), max normwise relative error 1e-4 for the fp32 model and 2e-2 for
bf16 models.  The call must leave the rolling state untouched.
"""

import numpy as np
import pytest

import synth
from oracle.expert import Expert
from oracle.full import expert_velocity, full_denoise
from tests.harness import TOL_BF16, TOL_F32, GpuRoll, have_gpu, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def analytic(kind, H, D, B):
    return synth.RavelShape(layers=0, width=0, n_q_heads=1, n_kv_heads=1, head_dim=32, mlp_dim=0,
                            horizon=H, action_dim=D, prefix_len=0, n_fop=0, fop_obs_dim=0,
                            dtype=W.F32, model_kind=kind, batch=B, name="analytic")


def gpu_full(g, steps, noise, fop=None):
    torch = g.torch
    nz = torch.from_numpy(np.ascontiguousarray(noise, dtype=np.float32)).to(g.dev)
    out = torch.empty_like(nz)
    f = None
    if fop is not None:
        g.fop.copy_(g.to_dev(fop))
        f = g.fop
    g.buf.full_denoise(steps, f, nz, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("S", [1, 5, 50])
def test_linear_field_chunk_is_bit_exact(S):
    lam = np.float32(0.8)
    s = analytic(W.ANALYTIC_LINEAR, 8, 7, 2)
    g = GpuRoll(s, {"analytic.lambda": np.array([lam], np.float32)}, 2, 0)
    noise = np.random.default_rng(S).standard_normal((2, 8, 7)).astype(np.float32)
    got = gpu_full(g, S, noise)
    for e in range(2):
        ref = full_denoise(lambda a, tau: lam * a, noise[e], S)
        assert np.array_equal(got[e], ref), e
        np.testing.assert_allclose(got[e], (1.0 - float(lam) / S) ** S * noise[e].astype(np.float64), rtol=1e-4)


@pytest.mark.parametrize("S", [1, 4, 10])
def test_ot_field_chunk_is_bit_exact_and_lands_on_the_target(S):
    s = analytic(W.ANALYTIC_OT, 6, 5, 3)
    target = np.random.default_rng(1).standard_normal(5).astype(np.float32)
    g = GpuRoll(s, {"analytic.target": target}, 3, 0)
    noise = np.random.default_rng(S + 10).standard_normal((3, 6, 5)).astype(np.float32)
    got = gpu_full(g, S, noise)
    for e in range(3):
        ref = full_denoise(lambda a, tau: (a - target[None, :]) / np.float32(tau), noise[e], S)
        assert np.array_equal(got[e], ref), e
        np.testing.assert_allclose(got[e], np.broadcast_to(target, (6, 5)), atol=1e-5)


def _transformer_case(name, batch, S, oracle_dtype, persistent=None, **replace):
    s = synth.get_config(name).replace(**replace) if replace else synth.get_config(name)
    wts = synth.draw_weights(s, seed=2, stress=name != "pi_b1")
    g = GpuRoll(s, wts, batch, 0)
    if persistent is not None:
        g.buf.set_option(g.rv.OPT_PERSISTENT, 1 if persistent else 0)
    ctx = [synth.draw_context(s, 0, e, 0) for e in range(batch)]
    for e, (k, v) in enumerate(ctx):
        g.set_context(e, k, v, 0)
    z = synth.draw_fop_tokens(s, 0, 0, batch=batch) if s.n_fop > 0 else None
    noise = np.random.default_rng(3).standard_normal((batch, s.horizon, s.action_dim)).astype(np.float32)
    got = gpu_full(g, S, noise, z)
    ex = Expert(s, wts, oracle_dtype)
    tol = TOL_F32 if s.dtype == W.F32 else TOL_BF16
    worst = 0.0
    for e in range(batch):
        k, v = ctx[e]
        ref = full_denoise(expert_velocity(ex, k, v, None if z is None else z[e]), noise[e].astype(oracle_dtype), S)
        err = rel_err(got[e], ref)
        worst = max(worst, err)
        assert err <= tol, f"env {e}: chunk error {err:.3e} > {tol:.1e}"
    return worst


@pytest.mark.parametrize("S", [1, 4, 8])
def test_tiny_fp32_chunk_matches_oracle(S):
    print("tiny_fp32 S", S, _transformer_case("tiny_fp32", 1, S, np.float64))


@pytest.mark.parametrize("persistent", [False, True])
def test_small_bf16_chunk_matches_oracle_on_both_paths(persistent):
    print("small_bf16", persistent, _transformer_case("small_bf16", 2, 5, np.float64, persistent=persistent,
                                                      layers=2))


def test_pi_b1_chunk_matches_oracle_at_ten_steps():
    print("pi_b1 S=10", _transformer_case("pi_b1", 1, 10, np.float32))


def test_rolling_state_is_untouched():
    s = synth.get_config("small_bf16").replace(layers=2)
    wts = synth.draw_weights(s, seed=5, stress=True)
    a, b = GpuRoll(s, wts, 1, 7), GpuRoll(s, wts, 1, 7)
    k, v = synth.draw_context(s, 0, 0, 0)
    for g in (a, b):
        g.set_context(0, k, v, 0)
    z = synth.draw_fop_tokens(s, 0, 0, batch=1)
    a.step(z)
    b.step(z)
    X0, t0, o0 = a.state()
    log0 = a.buf.publish_log()
    noise = np.random.default_rng(0).standard_normal((1, s.horizon, s.action_dim)).astype(np.float32)
    gpu_full(a, 6, noise, z)
    X1, t1, o1 = a.state()
    assert np.array_equal(X0, X1) and t0 == t1 and np.array_equal(o0, o1)
    assert a.buf.publish_log() == log0
    # the next rolling step is the same as on a buffer that never ran the baseline
    assert np.array_equal(a.step(z), b.step(z))


def test_argument_errors():
    s = analytic(W.ANALYTIC_LINEAR, 4, 3, 1)
    g = GpuRoll(s, {"analytic.lambda": np.array([0.5], np.float32)}, 1, 0)
    noise = np.zeros((1, 4, 3), np.float32)
    for bad in (0, 1025):
        with pytest.raises(g.rv.RavelError) as ei:
            gpu_full(g, bad, noise)
        assert ei.value.status == -4
    with pytest.raises(g.rv.RavelError) as ei:
        g.buf.full_denoise(2, None, None, None)
    assert ei.value.status == -1
