"""The pi0.5 way of feeding the context-age offset (App. A.1: an MLP of delta added to
the flow-time embedding; all slots share delta and keep their own flow time).  Pins of
the oracle's conditioning rows cond_i = silu(c_tau(i) + d) with
d = W_d2 silu(W_d1 delta + b_d1) + b_d2, and of the offset delta = p / K + delta_0
(Sec. 3.1 after Eq. 2; Sec. 4.4 for the lead bias).

The flow-time embedding is forced to a known vector c (W_t2 = 0, b_t2 = c), so the
conditioning is written out below element by element from its definition, with no
call into the oracle's arithmetic; planted variants of the oracle (inner silu
dropped, d added after the final silu, the sign of d flipped, d scaled) must fail the
same check."""

import math

import numpy as np
import pytest

import synth
from oracle import expert as ex
from oracle.rolling import OracleRavel

W_ = synth.workloads


def shape(**kw):
    base = dict(layers=2, width=16, n_q_heads=2, n_kv_heads=1, head_dim=8, mlp_dim=32, horizon=5, action_dim=3,
                prefix_len=4, n_fop=2, fop_obs_dim=6, dtype=W_.F32, name="mlp")
    base.update(kw)
    return synth.RavelShape(**base)


def _weights(s, c, seed=0):
    W = {k: v.astype(np.float64) for k, v in synth.draw_weights(s, seed=seed, stress=True).items()}
    W["time.w2"][:] = 0.0
    W["time.b2"][:] = c
    return W


def _scalar_silu(x):
    return x / (1.0 + math.exp(-x))


def conditioning_by_definition(W, c, delta):
    """cond_j = silu(c_j + sum_k W_d2[j, k] silu(W_d1[k, 0] delta + b_d1[k]) + b_d2[j]), scalar loops."""
    w = len(c)
    hid = [_scalar_silu(float(W["delta.w1"][k, 0]) * delta + float(W["delta.b1"][k])) for k in range(w)]
    out = []
    for j in range(w):
        d = float(W["delta.b2"][j])
        for k in range(w):
            d += float(W["delta.w2"][j, k]) * hid[k]
        out.append(_scalar_silu(float(c[j]) + d))
    return np.array(out)


class NoInnerSilu(ex.Expert):
    def delta_conditioning(self, delta):
        W = self.W
        return W["delta.w2"] @ (W["delta.w1"][:, 0] * delta + W["delta.b1"]) + W["delta.b2"]


class OffsetAfterSilu(ex.Expert):
    def conditioning(self, delta, taus=None):
        return ex.silu(self.tau_conditioning(taus)) + self.delta_conditioning(delta)[None, :]


class OffsetSignFlipped(ex.Expert):
    def conditioning(self, delta, taus=None):
        return ex.silu(self.tau_conditioning(taus) - self.delta_conditioning(delta)[None, :])


class OffsetHalved(ex.Expert):
    def delta_conditioning(self, delta):
        return 0.5 * super().delta_conditioning(delta)


DELTAS = [0.0, 0.3, 1.7, -2.5, 12.0]


def _max_dev(cls, s, W, c):
    e = cls(s, W)
    dev = 0.0
    for delta in DELTAS:
        got = e.conditioning(delta)
        ref = conditioning_by_definition(W, c, delta)
        assert got.shape == (s.horizon, s.width)
        dev = max(dev, float(np.abs(got - ref[None, :]).max()))
    return dev


def _c(s, seed=5):
    return np.random.default_rng(seed).standard_normal(s.width) * 1.5


def test_conditioning_rows_follow_the_definition():
    s = shape()
    c = _c(s)
    W = _weights(s, c)
    assert _max_dev(ex.Expert, s, W, c) < 1e-12


@pytest.mark.parametrize("cls", [NoInnerSilu, OffsetAfterSilu, OffsetSignFlipped, OffsetHalved])
def test_planted_offset_mistakes_fail_the_definition(cls):
    s = shape()
    c = _c(s)
    W = _weights(s, c)
    assert _max_dev(cls, s, W, c) > 1e-2, cls.__name__


def offset_embedding_by_definition(W, delta):
    """d_j = sum_k W_d2[j, k] silu(W_d1[k, 0] delta + b_d1[k]) + b_d2[j], scalar loops."""
    w = W["delta.b2"].shape[0]
    hid = [_scalar_silu(float(W["delta.w1"][k, 0]) * delta + float(W["delta.b1"][k])) for k in range(w)]
    return np.array([float(W["delta.b2"][j]) + sum(float(W["delta.w2"][j, k]) * hid[k] for k in range(w))
                     for j in range(w)])


def test_every_slot_gets_the_same_offset_embedding():
    """All slots share delta and keep their own flow time (App. A.1): with the flow-time
    embedding left free, row i is silu(c_tau(i) + d) with one d for every slot."""
    s = shape()
    W = {k: v.astype(np.float64) for k, v in synth.draw_weights(s, seed=1, stress=True).items()}
    e = ex.Expert(s, W)
    ct = e.tau_conditioning()
    assert np.abs(ct - ct[0]).max() > 1e-3  # the slots' flow-time rows differ
    for delta in (0.2, 0.9):
        d = offset_embedding_by_definition(W, delta)
        ref = np.array([[_scalar_silu(x) for x in row] for row in (ct + d[None, :])])
        np.testing.assert_allclose(e.conditioning(delta), ref, rtol=1e-12, atol=1e-13)


def test_identity_layers_velocity_carries_the_offset_through_the_final_norm():
    """Zero gates make every layer the identity, so the velocity is the output head of
    the encoded actions under the final modulation of cond -- written out here with the
    conditioning from its scalar definition."""
    s = shape()
    c = _c(s, 7)
    W = _weights(s, c, seed=3)
    w = s.width
    for l in range(s.layers):
        for lo, hi in ((2 * w, 3 * w), (5 * w, 6 * w)):
            W[f"layers.{l}.mod.w"][lo:hi] = 0
            W[f"layers.{l}.mod.b"][lo:hi] = 0
        if f"layers.{l}.fop.alpha" in W:
            W[f"layers.{l}.fop.alpha"][:] = 0
    rng = np.random.default_rng(4)
    a = rng.standard_normal((s.horizon, s.action_dim))
    k = rng.standard_normal((s.layers, s.prefix_len, s.n_kv_heads, s.head_dim))
    v = rng.standard_normal((s.layers, s.prefix_len, s.n_kv_heads, s.head_dim))
    z = rng.standard_normal((s.n_fop, w))
    for delta in (0.1, 2.3):
        cond = conditioning_by_definition(W, c, delta)
        fm = W["final.mod.w"] @ cond + W["final.mod.b"]
        h = a @ W["in.w"].T + W["in.b"]
        hn = h / np.sqrt((h * h).mean(1, keepdims=True) + s.rms_eps)
        ref = (hn * (1 + fm[:w]) + fm[w:2 * w]) @ W["out.w"].T + W["out.b"]
        got = ex.Expert(s, W).velocity(a, k, v, delta, z)
        np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_rolling_offset_is_age_over_slots_plus_lead_bias():
    """The offset handed to the expert at step t is (t - t_obs) / H + delta_0 (Sec. 3.1:
    delta_p = p / K; Sec. 4.4: the lead bias), recorded from the expert's own call."""
    H, d0 = 5, 0.25
    s = shape(horizon=H, delta_bias=d0)
    W = synth.draw_weights(s, seed=0, stress=True)
    o = OracleRavel(s, W, batch=2, seed=0)
    seen = []
    real = o.expert.velocity

    def spy(a, ck, cv, delta, *args, **kw):
        seen.append(delta)
        return real(a, ck, cv, delta, *args, **kw)

    o.expert.velocity = spy
    rng = np.random.default_rng(0)
    ctx = lambda: (rng.standard_normal((s.layers, s.prefix_len, 1, s.head_dim)),  # noqa: E731
                   rng.standard_normal((s.layers, s.prefix_len, 1, s.head_dim)))
    o.set_context(0, *ctx(), 0)
    o.set_context(1, *ctx(), 0)
    z = rng.standard_normal((2, s.n_fop, s.width))
    want = []
    t_obs = [0, 0]
    for t in range(9):
        if t == 4:
            o.set_context(1, *ctx(), 2)
            t_obs[1] = 2
        o.step(z)
        want += [(t - t_obs[0]) / H + d0, (t - t_obs[1]) / H + d0]
    assert seen == want
