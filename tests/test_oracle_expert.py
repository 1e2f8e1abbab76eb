"""Pins of the oracle's action expert.

Independent references used here: torch CPU library routines (scaled dot
product attention with grouped-query heads, rms_norm, gelu 'tanh', silu),
closed forms (uniform attention, identity layers) and the parameter count the
paper reports for its pi0.5 action expert.
"""

import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import expert as ex

GOLD = os.path.join(os.path.dirname(__file__), "golden", "paper_pins.txt")


def _pins():
    out = {}
    for line in open(GOLD):
        line = line.split("#")[0].strip()
        if line:
            k, v = line.split("=")
            out[k.strip()] = float(v)
    return out


def tiny_shape(**kw):
    base = dict(layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8, mlp_dim=48,
                horizon=6, action_dim=5, prefix_len=7, n_fop=3, fop_obs_dim=9,
                dtype=synth.workloads.F32, name="pin")
    base.update(kw)
    return synth.RavelShape(**base)


# --- parameter count ---------------------------------------------------------------

def test_pi_expert_parameter_count_matches_paper():
    pins = _pins()
    n = synth.param_count(synth.get_config("pi_b1"), with_fop=False)
    assert n == 431_150_112
    assert round(n / 1e6, 2) == pins["pi_expert_params_millions"]


# --- primitives against torch library routines -------------------------------------

@pytest.mark.parametrize("nq,nkv", [(4, 4), (4, 2), (8, 1)])
def test_attention_matches_torch_sdpa(nq, nkv):
    rng = np.random.default_rng(0)
    hd, tq, tk = 16, 9, 13
    q = rng.standard_normal((tq, nq * hd))
    k = rng.standard_normal((tk, nkv * hd))
    v = rng.standard_normal((tk, nkv * hd))
    got = ex.attention(q, k, v, nq, nkv, hd)
    tq_ = torch.from_numpy(q).view(tq, nq, hd).transpose(0, 1)[None]
    tk_ = torch.from_numpy(k).view(tk, nkv, hd).transpose(0, 1)[None].contiguous()
    tv_ = torch.from_numpy(v).view(tk, nkv, hd).transpose(0, 1)[None].contiguous()
    ref = F.scaled_dot_product_attention(tq_, tk_, tv_, enable_gqa=(nq != nkv))
    ref = ref[0].transpose(0, 1).reshape(tq, nq * hd).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_attention_identical_keys_is_mean_of_values():
    rng = np.random.default_rng(1)
    k = np.tile(rng.standard_normal((1, 8)), (5, 1))
    v = rng.standard_normal((5, 8))
    q = rng.standard_normal((3, 16))
    out = ex.attention(q, k, v, 2, 1, 8)
    np.testing.assert_allclose(out, np.tile(v.mean(0), (3, 2)), rtol=1e-12)


def test_attention_dominant_key_selects_its_value():
    hd = 4
    k = np.zeros((3, hd)); k[1, 0] = 100.0
    v = np.arange(12, dtype=np.float64).reshape(3, hd)
    q = np.zeros((1, hd)); q[0, 0] = 10.0
    np.testing.assert_allclose(ex.attention(q, k, v, 1, 1, hd)[0], v[1], atol=1e-12)


def test_norm_and_activations_match_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((6, 24)) * 3
    np.testing.assert_allclose(ex.rms_normalize(x, 1e-6),
                               F.rms_norm(torch.from_numpy(x), (24,), eps=1e-6).numpy(), rtol=1e-12)
    np.testing.assert_allclose(ex.gelu_tanh(x), F.gelu(torch.from_numpy(x), approximate="tanh").numpy(),
                               rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(ex.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-12, atol=1e-14)


def test_time_embedding_closed_forms():
    e = ex.time_embedding(np.array([0.0, 0.5]), 8)
    np.testing.assert_array_equal(e[0], [0, 0, 0, 0, 1, 1, 1, 1])
    # frequencies 10000^(-j/4): j = 0 -> 1, j = 2 -> 1/100
    assert e[1, 0] == pytest.approx(np.sin(500.0))
    assert e[1, 2] == pytest.approx(np.sin(5.0))
    assert e[1, 6] == pytest.approx(np.cos(5.0))


def test_flow_times_mirror_the_paper_profile():
    # paper: tau'_k = 1 - k/K for k = 1..K (1 = clean); here tau_i = 1 - tau'_{i+1}
    K = 10
    paper = 1.0 - np.arange(1, K + 1) / K
    np.testing.assert_allclose(ex.flow_times(K), 1.0 - paper, atol=1e-15)
    assert ex.flow_times(K)[-1] == 1.0 and ex.flow_times(K)[0] == pytest.approx(0.1)


# --- whole-expert special cases -------------------------------------------------------

def _weights(shape, seed=0, stress=True):
    return synth.draw_weights(shape, seed=seed, stress=stress)


def _ctx(shape, rng):
    k = rng.standard_normal((shape.layers, shape.prefix_len, shape.n_kv_heads, shape.head_dim))
    v = rng.standard_normal(k.shape)
    return k, v


def test_zero_gates_make_every_layer_the_identity():
    s = tiny_shape()
    W = _weights(s)
    w = s.width
    for l in range(s.layers):
        W[f"layers.{l}.mod.w"][2 * w:3 * w] = 0
        W[f"layers.{l}.mod.b"][2 * w:3 * w] = 0
        W[f"layers.{l}.mod.w"][5 * w:6 * w] = 0
        W[f"layers.{l}.mod.b"][5 * w:6 * w] = 0
        if f"layers.{l}.fop.alpha" in W:
            W[f"layers.{l}.fop.alpha"][:] = 0
    rng = np.random.default_rng(3)
    a = rng.standard_normal((s.horizon, s.action_dim))
    k, v = _ctx(s, rng)
    z = rng.standard_normal((s.n_fop, w))
    e = ex.Expert(s, W)
    got = e.velocity(a, k, v, 0.2, z)
    # closed form with identity layers: output head applied to the input projection
    h = a @ W["in.w"].T + W["in.b"]
    cond = e.conditioning(0.2)
    fm = cond @ W["final.mod.w"].T + W["final.mod.b"]
    hn = h / np.sqrt((h * h).mean(1, keepdims=True) + s.rms_eps)
    ref = (hn * (1 + fm[:, :w]) + fm[:, w:2 * w]) @ W["out.w"].T + W["out.b"]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    # and the context and FOP tokens then cannot matter
    got2 = e.velocity(a, k * 3 + 1, v - 2, 0.2, z * 5)
    np.testing.assert_allclose(got, got2, rtol=1e-12, atol=1e-12)


def test_final_modulation_gate_chunk_is_unused():
    s = tiny_shape()
    W = _weights(s)
    rng = np.random.default_rng(4)
    a = rng.standard_normal((s.horizon, s.action_dim))
    k, v = _ctx(s, rng)
    e1 = ex.Expert(s, W).velocity(a, k, v, 0.1)
    W2 = dict(W)
    W2["final.mod.w"] = W["final.mod.w"].copy(); W2["final.mod.w"][2 * s.width:] = 7.0
    e2 = ex.Expert(s, W2).velocity(a, k, v, 0.1)
    np.testing.assert_array_equal(e1, e2)


def test_offset_bias_equals_three_steps_at_ten_slots():
    # App. B.4: with K = 10, delta_0 = 0.3 corresponds to three control steps.
    pins = _pins()
    K = int(pins["buffer_slots"])
    assert 3 / K == pytest.approx(pins["delta_bias"])
    s = tiny_shape(horizon=K)
    from oracle.rolling import OracleRavel
    W = _weights(s)
    rng = np.random.default_rng(5)
    k, v = _ctx(s, rng)
    a = OracleRavel(s.replace(delta_bias=0.0), W, 1, 0)
    b = OracleRavel(s.replace(delta_bias=pins["delta_bias"]), W, 1, 0)
    a.set_context(0, k, v, 0)
    b.set_context(0, k, v, 0)
    a._apply_pending(); b._apply_pending()
    a.t = 3  # context age p = 3, no bias
    b.t = 0  # fresh context, bias 0.3
    assert a.offset(0) == pytest.approx(b.offset(0))
    x = rng.standard_normal((K, s.action_dim))
    np.testing.assert_allclose(a.velocity(0, x), b.velocity(0, x), rtol=1e-12)


def test_mha_is_the_special_case_nkv_equal_nq():
    # n_kv = n_q: every query head has its own KV head (j -> j)
    rng = np.random.default_rng(6)
    q = rng.standard_normal((4, 24)); k = rng.standard_normal((6, 24)); v = rng.standard_normal((6, 24))
    out = ex.attention(q, k, v, 3, 3, 8)
    for j in range(3):
        sl = slice(8 * j, 8 * j + 8)
        np.testing.assert_allclose(out[:, sl], ex.attention(q[:, sl], k[:, sl], v[:, sl], 1, 1, 8))


def test_no_prefix_is_pure_self_attention():
    s = tiny_shape(prefix_len=0)
    W = _weights(s)
    rng = np.random.default_rng(7)
    a = rng.standard_normal((s.horizon, s.action_dim))
    kk = np.zeros((s.layers, 0, s.n_kv_heads, s.head_dim))
    out = ex.Expert(s, W).velocity(a, kk, kk, 0.0)
    assert out.shape == (s.horizon, s.action_dim) and np.isfinite(out).all()


def test_buffer_attention_is_permutation_equivariant_over_slots():
    # No positional encoding of buffer tokens: permuting slots together with
    # their flow times permutes the velocities the same way.
    s = tiny_shape()
    W = _weights(s)
    rng = np.random.default_rng(8)
    a = rng.standard_normal((s.horizon, s.action_dim))
    k, v = _ctx(s, rng)
    z = rng.standard_normal((s.n_fop, s.width))
    e = ex.Expert(s, W)
    base = e.velocity(a, k, v, 0.3, z)
    perm = rng.permutation(s.horizon)
    e2 = ex.Expert(s, W)
    e2._ctau = e.tau_conditioning()[perm]
    np.testing.assert_allclose(e2.velocity(a[perm], k, v, 0.3, z), base[perm], rtol=1e-11, atol=1e-12)


def test_fop_encoder_shape_and_closed_form():
    s = tiny_shape()
    W = _weights(s)
    rng = np.random.default_rng(9)
    obs = rng.standard_normal((2, s.fop_obs_dim))
    z = ex.fop_encode(s, W, obs)
    assert z.shape == (2, s.n_fop, s.width)
    # zero first-layer weights and bias: z = W_f2 gelu(0) + b_f2 = b_f2
    W0 = dict(W); W0["fop.w1"] = np.zeros_like(W["fop.w1"]); W0["fop.b1"] = np.zeros_like(W["fop.b1"])
    np.testing.assert_allclose(ex.fop_encode(s, W0, obs)[1].reshape(-1), W["fop.b2"], rtol=1e-12)


@pytest.mark.parametrize("cfg", ["tiny_fp32", "small_bf16"])
def test_every_sub_block_moves_the_output_above_tolerance(cfg):
    # Parity is only meaningful if each sub-block changes v by far more than the
    # tolerance; checked on the stress weights used by the GPU parity tests.
    s = synth.get_config(cfg)
    W = synth.draw_weights(s, seed=0, stress=True)
    k, v = synth.draw_context(s, 0, 0, 0)
    z = synth.draw_fop_tokens(s, 0, 0, scale=1.0)[0]
    rng = np.random.default_rng(10)
    a = rng.standard_normal((s.horizon, s.action_dim))
    e = ex.Expert(s, W)
    full = e.velocity(a, k, v, 0.5, z)
    tol = 1e-4 if s.dtype == synth.workloads.F32 else 2e-2
    for block in ["attn", "adapter", "mlp", "delta"]:
        cut = e.velocity(a, k, v, 0.5, z, hooks={block})
        rel = np.abs(full - cut).max() / np.abs(full).max()
        assert rel > 10 * tol, (block, rel)
