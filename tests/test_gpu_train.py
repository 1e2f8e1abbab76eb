"""GPU parity of the streaming-aligned training objective (ravel_train_loss) against
the CPU oracle (oracle/training.py, Sec. 3.3 Eq. 5 and 6): training buffer at the
rolling flow-time profile, offset p / K, flow-matching loss per sample.

Bars: bit-exact velocities for the analytic fields (same fp32 operations), the
conditional-OT field aimed at the target gives loss 0; transformer velocities within
the rolling step's tolerances (1e-4 fp32, 2e-2 bf16) and losses within the same
relative bound.
"""

import numpy as np
import pytest

import synth
from oracle.expert import Expert
from oracle.training import expert_velocity, training_loss
from tests.harness import TOL_BF16, TOL_F32, GpuRoll, have_gpu, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def analytic(kind, H, D, B):
    return synth.RavelShape(layers=0, width=0, n_q_heads=1, n_kv_heads=1, head_dim=32, mlp_dim=0,
                            horizon=H, action_dim=D, prefix_len=0, n_fop=0, fop_obs_dim=0,
                            dtype=W.F32, model_kind=kind, batch=B, name="analytic")


def gpu_train(g, target, noise, ages, fop=None):
    torch = g.torch
    dev = g.dev
    t = torch.from_numpy(np.ascontiguousarray(target, dtype=np.float32)).to(dev)
    n = torch.from_numpy(np.ascontiguousarray(noise, dtype=np.float32)).to(dev)
    a = torch.from_numpy(np.asarray(ages, dtype=np.int64)).to(dev)
    loss = torch.empty(len(ages), dtype=torch.float32, device=dev)
    v = torch.empty_like(t)
    f = None
    if fop is not None:
        g.fop.copy_(g.to_dev(fop))
        f = g.fop
    g.buf.train_loss(t, n, a, f, loss, v)
    torch.cuda.synchronize()
    return loss.cpu().numpy(), v.cpu().numpy()


def test_ot_field_towards_the_target_has_zero_loss_and_exact_velocities():
    H, D, B = 10, 6, 3
    s = analytic(W.ANALYTIC_OT, H, D, B)
    target_vec = np.random.default_rng(0).standard_normal(D).astype(np.float32)
    g = GpuRoll(s, {"analytic.target": target_vec}, B, 0)
    target = np.broadcast_to(target_vec, (B, H, D)).copy()
    noise = np.random.default_rng(1).standard_normal((B, H, D)).astype(np.float32)
    loss, v = gpu_train(g, target, noise, [0, 3, 7])
    tau = ((np.arange(H) + 1) / H).astype(np.float32)[:, None]
    for e in range(B):
        ref_loss, ref_v = training_loss(lambda a: (a - target_vec) / tau, target[e], noise[e])
        assert np.array_equal(v[e], ref_v), e
        assert loss[e] < 1e-10 and ref_loss < 1e-10


def test_linear_field_velocities_are_bit_exact():
    lam = np.float32(0.7)
    H, D, B = 8, 5, 2
    s = analytic(W.ANALYTIC_LINEAR, H, D, B)
    g = GpuRoll(s, {"analytic.lambda": np.array([lam], np.float32)}, B, 0)
    rng = np.random.default_rng(2)
    target = rng.standard_normal((B, H, D)).astype(np.float32)
    noise = rng.standard_normal((B, H, D)).astype(np.float32)
    loss, v = gpu_train(g, target, noise, [1, 2])
    for e in range(B):
        ref_loss, ref_v = training_loss(lambda a: lam * a, target[e], noise[e])
        assert np.array_equal(v[e], ref_v), e
        assert abs(loss[e] - ref_loss) <= 1e-6 * ref_loss


def _case(name, batch, ages, oracle_dtype, sample=None, persistent=None, **replace):
    s = synth.get_config(name).replace(**replace) if replace else synth.get_config(name)
    wts = synth.draw_weights(s, seed=3, stress=name not in ("pi_b1", "pi_b64"))
    g = GpuRoll(s, wts, batch, 0)
    if persistent is not None:
        g.buf.set_option(g.rv.OPT_PERSISTENT, 1 if persistent else 0)
    envs = list(range(batch)) if sample is None else sample
    ctx = {}
    for e in range(batch):
        k, v = synth.draw_context(s, 0, e, 0)
        g.set_context(e, k, v, 0)
        if e in envs:
            ctx[e] = (k, v)
    z = synth.draw_fop_tokens(s, 0, 1, batch=batch) if s.n_fop > 0 else None
    rng = np.random.default_rng(4)
    target = rng.standard_normal((batch, s.horizon, s.action_dim)).astype(np.float32)
    noise = rng.standard_normal((batch, s.horizon, s.action_dim)).astype(np.float32)
    loss, v = gpu_train(g, target, noise, ages, z)
    ex = Expert(s, wts, oracle_dtype)
    tol = TOL_F32 if s.dtype == W.F32 else TOL_BF16
    worst = 0.0
    for e in envs:
        k, vv = ctx[e]
        ref_loss, ref_v = training_loss(expert_velocity(ex, k, vv, ages[e], None if z is None else z[e]),
                                        target[e].astype(oracle_dtype), noise[e].astype(oracle_dtype))
        ev = rel_err(v[e], ref_v)
        el = abs(float(loss[e]) - ref_loss) / ref_loss
        worst = max(worst, ev, el)
        assert ev <= tol, f"sample {e}: velocity error {ev:.3e}"
        assert el <= tol, f"sample {e}: loss error {el:.3e}"
    return worst


def test_tiny_fp32_matches_oracle():
    print("tiny_fp32", _case("tiny_fp32", 3, [0, 2, 9], np.float64))


@pytest.mark.parametrize("persistent", [False, True])
def test_small_bf16_matches_oracle_on_both_paths(persistent):
    print("small_bf16", persistent, _case("small_bf16", 3, [0, 5, 5], np.float64, persistent=persistent, layers=2))


def test_pi_b64_sampled_samples_match_oracle():
    ages = [int(a) for a in np.random.default_rng(5).integers(0, 10, 64)]
    print("pi_b64", _case("pi_b64", 64, ages, np.float32, sample=[0, 31, 63]))


def test_rolling_state_is_untouched():
    s = synth.get_config("small_bf16").replace(layers=2)
    wts = synth.draw_weights(s, seed=6, stress=True)
    a, b = GpuRoll(s, wts, 1, 3), GpuRoll(s, wts, 1, 3)
    k, v = synth.draw_context(s, 0, 0, 0)
    for g in (a, b):
        g.set_context(0, k, v, 0)
    z = synth.draw_fop_tokens(s, 0, 0, batch=1)
    a.step(z)
    b.step(z)
    X0, t0, _ = a.state()
    rng = np.random.default_rng(7)
    tgt = rng.standard_normal((1, s.horizon, s.action_dim)).astype(np.float32)
    gpu_train(a, tgt, rng.standard_normal(tgt.shape).astype(np.float32), [4], z)
    X1, t1, _ = a.state()
    assert np.array_equal(X0, X1) and t0 == t1
    assert np.array_equal(a.step(z), b.step(z))
