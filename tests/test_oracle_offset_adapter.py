"""The DynamicVLA way of feeding the context-age offset (App. A.1): delta concatenated
with the action and flow-time embeddings before the action-time MLP, and its
sinusoidal embedding conditioning a gated residual adapter on the resulting action
tokens.  Pins of the oracle's form: where delta may and may not enter, the gate's
tanh law, the per-slot flow time, and the reduction of the layers to the identity."""

import numpy as np

import synth
from oracle import expert as ex

W_ = synth.workloads


def shape(**kw):
    base = dict(layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8, mlp_dim=48, horizon=6, action_dim=5,
                prefix_len=7, n_fop=3, fop_obs_dim=9, dtype=W_.F32, offset_mode=W_.OFFSET_ADAPTER, name="ada")
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


def test_weights_have_the_action_time_mlp_and_adapter_and_no_offset_mlp():
    s = shape()
    W = synth.draw_weights(s)
    w, r = s.width, s.width // 4
    assert W["in.w"].shape == (w, s.action_dim)
    assert W["at.w1"].shape == (w, 2 * w + 1) and W["at.w2"].shape == (w, w)
    assert W["ta.w1"].shape == (r, 2 * w) and W["ta.w2"].shape == (w, r) and W["ta.alpha"].shape == (1,)
    assert not any(n.startswith("delta.") for n in W)


def test_offset_enters_only_through_its_mlp_column_and_the_adapter():
    s = shape()
    W = _weights(s)
    a, k, v, z = _inputs(s, 2)
    e = ex.Expert(s, W)
    v1, v2 = e.velocity(a, k, v, 0.1, z), e.velocity(a, k, v, 0.9, z)
    # the offset moves the output well above the bf16 tolerance ...
    assert np.abs(v1 - v2).max() / np.abs(v1).max() > 0.2
    # ... and nowhere else than the action-time MLP's last input column and the adapter
    W0 = dict(W)
    W0["at.w1"] = W["at.w1"].copy()
    W0["at.w1"][:, 2 * s.width] = 0
    W0["ta.alpha"] = np.zeros(1)
    e0 = ex.Expert(s, W0)
    np.testing.assert_array_equal(e0.velocity(a, k, v, 0.1, z), e0.velocity(a, k, v, 0.9, z))
    # each of the two alone carries it
    for key in ("mlp", "adapter"):
        W1 = dict(W0)
        if key == "mlp":
            W1["at.w1"] = W["at.w1"]
        else:
            W1["ta.alpha"] = W["ta.alpha"]
        e1 = ex.Expert(s, W1)
        d = e1.velocity(a, k, v, 0.1, z) - e1.velocity(a, k, v, 0.9, z)
        assert np.abs(d).max() > 1e-3, key


def test_offset_column_is_a_shift_of_the_mlp_bias():
    """Before the MLP's nonlinearity delta only adds delta * W_a1[:, 2w]: with the
    adapter switched off, encoding at delta equals encoding at 0 with b_a1 moved by
    that vector (a dropped term, a wrong column or delta applied after the
    nonlinearity all break this)."""
    s = shape()
    W = _weights(s)
    W["ta.alpha"] = np.zeros(1)
    a, _, _, _ = _inputs(s, 3)
    d = 0.37
    got = ex.Expert(s, W).encode_actions(a, d)
    Wb = dict(W)
    Wb["at.b1"] = W["at.b1"] + d * W["at.w1"][:, 2 * s.width]
    ref = ex.Expert(s, Wb).encode_actions(a, 0.0)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_adapter_scales_with_the_tanh_of_its_gate():
    """The adapter's contribution is tanh(beta) times one fixed vector per slot."""
    s = shape()
    W = _weights(s)
    a, _, _, _ = _inputs(s, 4)

    def enc(beta):
        Wb = dict(W)
        Wb["ta.alpha"] = np.array([beta])
        return ex.Expert(s, Wb).encode_actions(a, 0.55)

    base = enc(0.0)
    u1 = (enc(0.3) - base) / np.tanh(0.3)
    u2 = (enc(-1.7) - base) / np.tanh(-1.7)
    np.testing.assert_allclose(u1, u2, rtol=1e-10, atol=1e-12)
    assert np.abs(u1).max() > 1e-2


def test_adapter_sees_the_sinusoid_of_delta_on_every_slot():
    """The adapter's condition is the flow-time sinusoid evaluated at delta, the same
    on every slot: zeroing the adapter's condition half removes delta from it, and
    putting delta = tau_j reproduces the sinusoid the flow time uses at slot j."""
    s = shape()
    W = _weights(s)
    W["at.w1"][:, 2 * s.width] = 0  # delta only in the adapter
    a, _, _, _ = _inputs(s, 5)
    e = ex.Expert(s, W)
    assert np.abs(e.encode_actions(a, 0.2) - e.encode_actions(a, 0.8)).max() > 1e-3
    Wn = dict(W)
    Wn["ta.w1"] = W["ta.w1"].copy()
    Wn["ta.w1"][:, s.width:] = 0
    en = ex.Expert(s, Wn)
    np.testing.assert_array_equal(en.encode_actions(a, 0.2), en.encode_actions(a, 0.8))
    # the adapter condition at delta = tau_j against the flow time's own table row j
    w, half = s.width, s.width // 2
    tau = (np.arange(s.horizon) + 1.0) / s.horizon
    j = 2
    om = 10000.0 ** (-np.arange(half) / half)
    row = np.concatenate([np.sin(1000.0 * tau[j] * om), np.cos(1000.0 * tau[j] * om)])
    np.testing.assert_allclose(ex.time_embedding([tau[j]], w)[0], row, rtol=0, atol=1e-12)


def test_each_slot_uses_its_own_flow_time():
    """Equal actions in every slot: the tokens then differ only through tau_i, so
    giving every slot the flow time of slot j (a full-horizon pass) reproduces row j
    of the rolling pass on every row."""
    s = shape()
    W = _weights(s)
    rng = np.random.default_rng(6)
    a = np.repeat(rng.standard_normal((1, s.action_dim)), s.horizon, axis=0)
    e = ex.Expert(s, W)
    roll = e.encode_actions(a, 0.4)
    tau = (np.arange(s.horizon) + 1.0) / s.horizon
    assert np.abs(roll[0] - roll[-1]).max() > 1e-3
    for j in (0, 3, s.horizon - 1):
        full = e.encode_actions(a, 0.4, taus=np.full(s.horizon, tau[j]))
        np.testing.assert_allclose(full, np.broadcast_to(roll[j], full.shape), rtol=1e-12, atol=1e-13)


def test_identity_layers_reduce_to_the_output_head_of_the_tokens():
    """Zero residual and adapter gates make every layer the identity: the velocity is
    the output head of the encoder's tokens, conditioned by the flow time alone."""
    s = shape()
    W = _weights(s)
    w = s.width
    for l in range(s.layers):
        for lo, hi in ((2 * w, 3 * w), (5 * w, 6 * w)):
            W[f"layers.{l}.mod.w"][lo:hi] = 0
            W[f"layers.{l}.mod.b"][lo:hi] = 0
        if f"layers.{l}.fop.alpha" in W:
            W[f"layers.{l}.fop.alpha"][:] = 0
    a, k, v, z = _inputs(s, 1)
    delta = 0.7
    e = ex.Expert(s, W)
    got = e.velocity(a, k, v, delta, z)
    h = e.encode_actions(a, delta)
    sig = lambda x: x / (1.0 + np.exp(-x))
    cond = sig(e.tau_conditioning())
    fm = cond @ W["final.mod.w"].T + W["final.mod.b"]
    hn = h / np.sqrt((h * h).mean(1, keepdims=True) + s.rms_eps)
    ref = (hn * (1 + fm[:, :w]) + fm[:, w:2 * w]) @ W["out.w"].T + W["out.b"]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    # and the context never reaches the output
    np.testing.assert_allclose(e.velocity(a, k * 3.0, v - 1.0, delta, z), got, rtol=1e-12, atol=1e-12)
