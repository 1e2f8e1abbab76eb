"""The persistent few-row path (one cooperative kernel for all layers) against
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
