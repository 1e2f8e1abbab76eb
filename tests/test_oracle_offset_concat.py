"""The X-VLA way of feeding the context-age offset (App. A.1): delta concatenated to
every slot's noisy action at the action encoder instead of an MLP of delta added to
the flow-time embedding.  Pins of the oracle's concatenated form."""

import numpy as np

import synth
from oracle import expert as ex

W_ = synth.workloads


def shape(**kw):
    base = dict(layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8, mlp_dim=48, horizon=6, action_dim=5,
                prefix_len=7, n_fop=3, fop_obs_dim=9, dtype=W_.F32, offset_mode=W_.OFFSET_CONCAT, name="cat")
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


def test_weights_have_an_offset_column_and_no_offset_mlp():
    s = shape()
    W = synth.draw_weights(s)
    assert W["in.w"].shape == (s.width, s.action_dim + 1)
    assert not any(n.startswith("delta.") for n in W)


def test_identity_layers_closed_form():
    """Zero residual gates and adapter gates make every layer the identity; the velocity
    is then the output head applied to the action encoder of [a_i ; delta], conditioned
    by the flow time alone: written out here from the time MLP's definition."""
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
    got = ex.Expert(s, W).velocity(a, k, v, delta, z)

    tau = (np.arange(s.horizon) + 1.0) / s.horizon
    half = w // 2
    om = 10000.0 ** (-np.arange(half) / half)
    emb = np.concatenate([np.sin(1000.0 * tau[:, None] * om), np.cos(1000.0 * tau[:, None] * om)], axis=1)
    sig = lambda x: x / (1.0 + np.exp(-x))
    ctau = sig(emb @ W["time.w1"].T + W["time.b1"]) @ W["time.w2"].T + W["time.b2"]
    cond = sig(ctau)
    h = a @ W["in.w"][:, :s.action_dim].T + delta * W["in.w"][:, s.action_dim] + W["in.b"]
    fm = cond @ W["final.mod.w"].T + W["final.mod.b"]
    hn = h / np.sqrt((h * h).mean(1, keepdims=True) + s.rms_eps)
    ref = (hn * (1 + fm[:, :w]) + fm[:, w:2 * w]) @ W["out.w"].T + W["out.b"]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_offset_enters_only_through_its_input_column():
    s = shape()
    W = _weights(s)
    a, k, v, z = _inputs(s, 2)
    e = ex.Expert(s, W)
    v1, v2 = e.velocity(a, k, v, 0.1, z), e.velocity(a, k, v, 0.9, z)
    # the offset moves the output well above the bf16 tolerance ...
    assert np.abs(v1 - v2).max() / np.abs(v1).max() > 0.2
    # ... and only through the last column of the action encoder
    W0 = dict(W)
    W0["in.w"] = W["in.w"].copy()
    W0["in.w"][:, s.action_dim] = 0
    e0 = ex.Expert(s, W0)
    np.testing.assert_array_equal(e0.velocity(a, k, v, 0.1, z), e0.velocity(a, k, v, 0.9, z))


def test_every_slot_sees_the_same_offset():
    """All slots share one offset (App. A.1): the encoder's response to delta is the same
    vector delta * W_in[:, D_a] on every slot, whatever the slot's action."""
    s = shape()
    W = _weights(s)
    a, _, _, _ = _inputs(s, 3)
    e = ex.Expert(s, W)
    dh = e.encode_actions(a, 0.45) - e.encode_actions(a, 0.0)
    np.testing.assert_allclose(dh, np.broadcast_to(0.45 * W["in.w"][:, s.action_dim], dh.shape), rtol=1e-12,
                               atol=1e-14)


def test_zero_offset_paths_agree_with_the_mlp_form():
    """With its offset column zero, the concatenated form equals the MLP form whose offset
    embedding is zero (W_d2 = 0, b_d2 = 0): both reduce to cond = silu(c_tau)."""
    sc = shape()
    sm = shape(offset_mode=W_.OFFSET_MLP)
    Wc = _weights(sc)
    Wc["in.w"][:, sc.action_dim] = 0
    Wm = {k: v.copy() for k, v in _weights(sm).items()}
    for k in Wm:
        if not k.startswith("delta.") and k != "in.w":
            Wm[k] = Wc[k].copy()
    Wm["in.w"] = Wc["in.w"][:, :sm.action_dim].copy()
    Wm["delta.w2"][:] = 0
    Wm["delta.b2"][:] = 0
    a, k, v, z = _inputs(sc, 4)
    np.testing.assert_allclose(ex.Expert(sc, Wc).velocity(a, k, v, 0.6, z), ex.Expert(sm, Wm).velocity(a, k, v, 0.6, z),
                               rtol=1e-12, atol=1e-12)
