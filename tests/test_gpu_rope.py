"""GPU parity of the optional rotary position embedding of the buffer tokens (slot i
at position P + i, prefix keys as given) against the CPU oracle.  Bars as for the
rolling step: 1e-4 (fp32 model) and 2e-2 (bf16 models) on every released action and
on the ring state; the full-horizon chunk and training losses within the same bounds."""

import numpy as np
import pytest

import synth
from tests.harness import GpuRoll, have_gpu, run_parity

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def test_tiny_fp32_rope_roll_matches_oracle():
    s = synth.get_config("tiny_fp32").replace(rope_base=10000.0, context_period=3)
    wts = synth.draw_weights(s, seed=31, stress=True)
    ea, ex, n = run_parity(s, wts, batch=1, seed=5, steps=40, oracle_dtype=np.float64, check_every=10)
    print(f"tiny_fp32 rope: {n} steps, action err {ea:.2e}, state err {ex:.2e}")


@pytest.mark.parametrize("persistent", [True, False])
def test_small_bf16_rope_roll_matches_oracle_on_both_paths(persistent, monkeypatch):
    if not persistent:
        monkeypatch.setenv("RAVEL_NO_PERSISTENT", "1")
    s = synth.get_config("small_bf16").replace(layers=2, rope_base=100.0, context_period=4)
    wts = synth.draw_weights(s, seed=32, stress=True)
    ea, ex, n = run_parity(s, wts, batch=2, seed=6, steps=24, oracle_dtype=np.float64, check_every=8)
    print(f"small_bf16 rope persistent={persistent}: action err {ea:.2e}, state err {ex:.2e}")


def test_pi_widths_rope_roll_matches_oracle():
    """256-dim heads, 816 prefix tokens (positions up to 865), one env: the persistent
    kernel with its rotary phase after every QKV projection."""
    s = synth.get_config("pi_b1").replace(layers=2, rope_base=10000.0, context_period=2)
    wts = synth.draw_weights(s, seed=33, stress=True)
    ea, ex, n = run_parity(s, wts, batch=1, seed=8, steps=6, oracle_dtype=np.float32, check_every=3)
    print(f"pi widths rope: action err {ea:.2e}, state err {ex:.2e}")


def test_persistent_kernel_has_a_rotary_phase():
    from tests.test_gpu_persistent import _phase_classes
    s = synth.get_config("small_bf16").replace(layers=3, rope_base=10000.0)
    assert "rope" in _phase_classes(s, synth.draw_weights(s, seed=34))


def test_full_horizon_chunk_with_rope():
    from tests.test_gpu_full import _transformer_case
    print("full-horizon rope fp32", _transformer_case("tiny_fp32", 1, 4, np.float64, rope_base=10000.0))
    print("full-horizon rope bf16", _transformer_case("small_bf16", 2, 5, np.float64, layers=2, rope_base=100.0))


def test_training_loss_with_rope():
    from tests.test_gpu_train import _case
    print("tiny_fp32 rope training", _case("tiny_fp32", 3, [0, 4, 11], np.float64, rope_base=10000.0))
