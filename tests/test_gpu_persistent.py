"""The persistent few-row path (one kernel for all layers) against
the per-kernel path and the oracle."""

import numpy as np
import pytest

import synth
from oracle.rolling import OracleRavel
from tests.harness import GpuRoll, have_gpu, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def _roll(shape, wts, batch, steps, persistent, seed=3):
    from paper_2609_34170_amd import ravel
    g = GpuRoll(shape, wts, batch, seed=seed)
    g.buf.set_option(ravel.OPT_PERSISTENT, 1 if persistent else 0)
    for e in range(batch):
        k, v = synth.draw_context(shape, 0, e, 0)
        g.set_context(e, k, v, 0)
    outs = []
    for st in range(steps):
        outs.append(g.step(synth.draw_fop_tokens(shape, 0, st, batch=batch)))
    g.buf.sync()
    X, t, _ = g.state()
    return np.stack(outs), X


@pytest.mark.parametrize("shape_kw,batch", [
    (dict(layers=2, width=256, n_q_heads=4, n_kv_heads=2, head_dim=64, mlp_dim=512, horizon=12,
          action_dim=7, prefix_len=40, n_fop=3, fop_obs_dim=16), 2),
    (dict(layers=3, width=512, n_q_heads=2, n_kv_heads=1, head_dim=256, mlp_dim=1024, horizon=50,
          action_dim=32, prefix_len=300, n_fop=4, fop_obs_dim=16), 1),
])
def test_persistent_matches_per_kernel_path_and_oracle(shape_kw, batch):
    s = synth.RavelShape(dtype=W.BF16, batch=batch, name="pers", **shape_kw)
    wts = synth.draw_weights(s, seed=5, stress=True)
    steps = 6
    a_p, X_p = _roll(s, wts, batch, steps, True)
    a_k, X_k = _roll(s, wts, batch, steps, False)
    o = OracleRavel(s, wts, batch=batch, seed=3)
    for e in range(batch):
        k, v = synth.draw_context(s, 0, e, 0)
        o.set_context(e, k, v, 0)
    a_o = np.stack([o.step(synth.draw_fop_tokens(s, 0, st, batch=batch)) for st in range(steps)])
    print(f"persistent vs kernels {rel_err(a_p, a_k):.2e}, vs oracle {rel_err(a_p, a_o):.2e}")
    assert rel_err(a_p, a_o) < 2e-2
    assert rel_err(X_p, o.X) < 2e-2
    assert rel_err(a_p, a_k) < 2e-2


def test_persistent_is_deterministic():
    s = synth.RavelShape(layers=2, width=256, n_q_heads=4, n_kv_heads=2, head_dim=64, mlp_dim=512, horizon=12,
                         action_dim=7, prefix_len=40, n_fop=3, fop_obs_dim=16, dtype=W.BF16, batch=2, name="pd")
    wts = synth.draw_weights(s, seed=6, stress=True)
    a1, _ = _roll(s, wts, 2, 10, True)
    a2, _ = _roll(s, wts, 2, 10, True)
    assert np.array_equal(a1, a2)


def _phase_classes(shape, wts):
    """Phase classes of the persistent kernel's list for one env (from the profile records)."""
    from tests.harness import GpuRoll
    g = GpuRoll(shape, wts, 1, seed=3)
    k, v = synth.draw_context(shape, 0, 0, 0)
    g.set_context(0, k, v, 0)
    g.fop.copy_(g.to_dev(synth.draw_fop_tokens(shape, 0, 0, batch=1)))
    recs = g.buf.profile_step(g.fop, g.action)
    return {r[0].split("/", 1)[1] for r in recs if r[0].startswith("persistent/")}


@pytest.mark.parametrize("n_fop", [16, 5])
def test_fused_cross_attention_matches_the_attention_phase_and_oracle(n_fop, monkeypatch):
    """One env with 256-dim heads: the adapter output projection computes its head's
    cross-attention itself (no attention phase); against the separate attention
    phase and the oracle, with every FOP slot used and with a ragged key count."""
    s = synth.RavelShape(layers=2, width=512, n_q_heads=4, n_kv_heads=1, head_dim=256, mlp_dim=1024, horizon=20,
                         action_dim=9, prefix_len=70, n_fop=n_fop, fop_obs_dim=16, dtype=W.BF16, batch=1,
                         name="xattn")
    wts = synth.draw_weights(s, seed=7, stress=True)
    steps = 6
    assert "cross_attn" not in _phase_classes(s, wts)
    a_f, X_f = _roll(s, wts, 1, steps, True)
    monkeypatch.setenv("RAVEL_NO_FUSED_XATTN", "1")
    assert "cross_attn" in _phase_classes(s, wts)
    a_u, X_u = _roll(s, wts, 1, steps, True)
    o = OracleRavel(s, wts, batch=1, seed=3)
    k, v = synth.draw_context(s, 0, 0, 0)
    o.set_context(0, k, v, 0)
    a_o = np.stack([o.step(synth.draw_fop_tokens(s, 0, st, batch=1)) for st in range(steps)])
    print(f"fused vs attention phase {rel_err(a_f, a_u):.2e}, fused vs oracle {rel_err(a_f, a_o):.2e}, "
          f"attention phase vs oracle {rel_err(a_u, a_o):.2e}")
    assert rel_err(a_f, a_o) < 2e-2
    assert rel_err(X_f, o.X) < 2e-2
    assert rel_err(a_u, a_o) < 2e-2
    assert rel_err(a_f, a_u) < 2e-2


def _launch_names(shape, wts, batch):
    from tests.harness import GpuRoll
    g = GpuRoll(shape, wts, batch, seed=3)
    for e in range(batch):
        k, v = synth.draw_context(shape, 0, e, 0)
        g.set_context(e, k, v, 0)
    g.fop.copy_(g.to_dev(synth.draw_fop_tokens(shape, 0, 0, batch=batch)))
    return {r[0] for r in g.buf.profile_step(g.fop, g.action) if not r[0].startswith(("persistent/", "phase/"))}


@pytest.mark.parametrize("shape_kw,batch,paired", [
    # 50 rows and 4 FOP tokens: layer 0's modulation and the FOP keys/values share a launch
    (dict(layers=2, width=512, n_q_heads=2, n_kv_heads=1, head_dim=256, mlp_dim=1024, horizon=50,
          action_dim=32, prefix_len=300, n_fop=4, fop_obs_dim=16), 1, True),
    # 24 rows: the modulation launch forms the norm operands alone
    (dict(layers=2, width=256, n_q_heads=4, n_kv_heads=2, head_dim=64, mlp_dim=512, horizon=12,
          action_dim=7, prefix_len=40, n_fop=3, fop_obs_dim=16), 2, False),
    # 64 rows of 4 envs and 16 FOP rows: both GEMMs of the paired launch at their full row fragments
    (dict(layers=2, width=256, n_q_heads=4, n_kv_heads=2, head_dim=64, mlp_dim=512, horizon=16,
          action_dim=5, prefix_len=33, n_fop=4, fop_obs_dim=16), 4, True),
])
def test_fused_prologue_is_bitwise_the_separate_launches(shape_kw, batch, paired, monkeypatch):
    """The persistent step's two-launch prologue (offset conditioning with the input
    projection; layer 0's modulation forming the first norm's p and shift copies) computes
    every value with the same operations as the separate launches: actions and ring agree
    bit for bit over several steps."""
    s = synth.RavelShape(dtype=W.BF16, batch=batch, name="prologue", **shape_kw)
    wts = synth.draw_weights(s, seed=8, stress=True)
    names = _launch_names(s, wts, batch)
    assert "offset_cond_in_proj" in names, names
    assert ("mod_layer0_fop_kv" in names) == paired, names
    a_f, X_f = _roll(s, wts, batch, 6, True)
    monkeypatch.setenv("RAVEL_NO_FUSED_PROLOGUE", "1")
    names_sep = _launch_names(s, wts, batch)
    assert "offset_cond_in_proj" not in names_sep and "in_proj" in names_sep, names_sep
    a_s, X_s = _roll(s, wts, batch, 6, True)
    assert np.array_equal(a_f, a_s)
    assert np.array_equal(X_f, X_s)
