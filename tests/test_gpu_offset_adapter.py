"""GPU parity of the DynamicVLA way of feeding the context-age offset (App. A.1: delta
concatenated with the action and flow-time embeddings before the action-time MLP,
and a gated residual adapter conditioned on delta's sinusoidal embedding) against
the CPU oracle, with context refreshes so that the offset changes from step to step.

Bars as for the rolling step: 1e-4 (fp32 model) and 2e-2 (bf16 models) on every
released action and on the ring state; the full-horizon chunk and training losses
within the same bounds."""

import numpy as np
import pytest

import synth
from tests.harness import have_gpu, run_parity

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def test_tiny_fp32_adapter_roll_matches_oracle():
    s = synth.get_config("tiny_fp32").replace(offset_mode=W.OFFSET_ADAPTER, context_period=3, delta_bias=0.2)
    wts = synth.draw_weights(s, seed=21, stress=True)
    ea, ex, n = run_parity(s, wts, batch=1, seed=5, steps=40, oracle_dtype=np.float64, check_every=10)
    print(f"tiny_fp32 adapter: {n} steps, action err {ea:.2e}, state err {ex:.2e}")


@pytest.mark.parametrize("persistent", [True, False])
def test_small_bf16_adapter_roll_matches_oracle_on_both_paths(persistent, monkeypatch):
    if not persistent:
        monkeypatch.setenv("RAVEL_NO_PERSISTENT", "1")
    s = synth.get_config("small_bf16").replace(layers=2, offset_mode=W.OFFSET_ADAPTER, context_period=4)
    wts = synth.draw_weights(s, seed=22, stress=True)
    ea, ex, n = run_parity(s, wts, batch=2, seed=6, steps=24, oracle_dtype=np.float64, check_every=8)
    print(f"small_bf16 adapter persistent={persistent}: action err {ea:.2e}, state err {ex:.2e}")


def test_staggered_refreshes_give_each_env_its_own_offset():
    """Five envs refreshed at staggered steps (so their offsets differ within a step),
    80 rows: the per-kernel path with conditioning groups and tiled GEMMs."""
    s = synth.get_config("small_bf16").replace(layers=2, offset_mode=W.OFFSET_ADAPTER, context_period=3,
                                               stagger=True)
    wts = synth.draw_weights(s, seed=23, stress=True)
    ea, ex, n = run_parity(s, wts, batch=5, seed=7, steps=12, oracle_dtype=np.float64, check_every=6)
    print(f"small_bf16 adapter B=5 staggered: action err {ea:.2e}, state err {ex:.2e}")


def test_pi_width_adapter_roll_on_the_persistent_path():
    """The pi-style widths (w = 1024, 256-dim heads, 50 slots) with two layers: the
    action-time MLP's 2112-wide inputs and the 256-wide adapter bottleneck through the
    few-row GEMMs ahead of the persistent kernel."""
    s = synth.get_config("pi_b1").replace(layers=2, offset_mode=W.OFFSET_ADAPTER, context_period=2)
    wts = synth.draw_weights(s, seed=24, stress=True)
    ea, ex, n = run_parity(s, wts, batch=1, seed=8, steps=6, oracle_dtype=np.float32, check_every=3)
    print(f"pi widths adapter: action err {ea:.2e}, state err {ex:.2e}")


@pytest.mark.parametrize("persistent", [False, True])
def test_full_horizon_chunk_with_the_adapter_form(persistent):
    from tests.test_gpu_full import _transformer_case
    print("full-horizon adapter", persistent,
          _transformer_case("small_bf16", 2, 5, np.float64, persistent=persistent, layers=2,
                            offset_mode=W.OFFSET_ADAPTER, delta_bias=0.3))


def test_tiny_fp32_full_horizon_chunk_with_the_adapter_form():
    from tests.test_gpu_full import _transformer_case
    print("full-horizon adapter fp32",
          _transformer_case("tiny_fp32", 1, 4, np.float64, offset_mode=W.OFFSET_ADAPTER, delta_bias=0.3))


def test_training_loss_with_the_adapter_form():
    from tests.test_gpu_train import _case
    print("tiny_fp32 adapter training", _case("tiny_fp32", 3, [0, 4, 11], np.float64, offset_mode=W.OFFSET_ADAPTER))
    print("small_bf16 adapter training", _case("small_bf16", 4, [0, 2, 5, 9], np.float64, layers=2,
                                               offset_mode=W.OFFSET_ADAPTER))


def test_ragged_shapes_with_the_adapter_form_and_rotary_positions():
    """63 rows (3 envs x 21 slots), 77 prefix tokens, 32-dim heads, width 256 (adapter
    bottleneck 64): the adapter form on the persistent path, then with rotary positions
    on the per-kernel path."""
    base = dict(layers=2, width=256, n_q_heads=4, n_kv_heads=2, head_dim=32, mlp_dim=512, horizon=21,
                action_dim=5, prefix_len=77, n_fop=3, fop_obs_dim=16, dtype=W.BF16, batch=3,
                offset_mode=W.OFFSET_ADAPTER, context_period=3, stagger=True, delta_bias=0.1, name="ragged_ada")
    for rope in (0.0, 1000.0):
        s = synth.RavelShape(rope_base=rope, **base)
        wts = synth.draw_weights(s, seed=25, stress=True)
        ea, ex, n = run_parity(s, wts, batch=3, seed=9, steps=9, oracle_dtype=np.float64, check_every=3)
        print(f"ragged adapter rope={rope}: action err {ea:.2e}, state err {ex:.2e}")


def test_batch64_widths_with_the_adapter_form_sampled_envs():
    """The pi-style widths at batch 64 (3200 rows: the action-time MLP's 2112-wide inputs
    through the tiled MFMA GEMMs, conditioning groups, staggered refreshes) with two
    layers and rotary positions; envs {0, 31, 63} against the oracle."""
    s = synth.get_config("pi_b64").replace(layers=2, offset_mode=W.OFFSET_ADAPTER, rope_base=10000.0)
    wts = synth.draw_weights(s, seed=26, stress=True)
    ea, ex, n = run_parity(s, wts, batch=64, seed=10, steps=6, env_sample=[0, 31, 63], oracle_dtype=np.float32,
                           check_every=3)
    print(f"batch 64 adapter + rope: action err {ea:.2e}, state err {ex:.2e}")
