"""GPU parity of the X-VLA way of feeding the context-age offset (App. A.1: delta
concatenated to every slot's noisy action at the action encoder) against the CPU
oracle, with context refreshes so that the offset changes from step to step.

Bars as for the rolling step: 1e-4 (fp32 model) and 2e-2 (bf16 models) on every
released action and on the ring state; training losses within the same bound."""

import numpy as np
import pytest

import synth
from tests.harness import have_gpu, run_parity

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def test_tiny_fp32_concat_roll_matches_oracle():
    s = synth.get_config("tiny_fp32").replace(offset_mode=W.OFFSET_CONCAT, context_period=3, delta_bias=0.2)
    wts = synth.draw_weights(s, seed=11, stress=True)
    ea, ex, n = run_parity(s, wts, batch=1, seed=5, steps=40, oracle_dtype=np.float64, check_every=10)
    print(f"tiny_fp32 concat: {n} steps, action err {ea:.2e}, state err {ex:.2e}")


@pytest.mark.parametrize("persistent", [True, False])
def test_small_bf16_concat_roll_matches_oracle_on_both_paths(persistent, monkeypatch):
    if not persistent:
        monkeypatch.setenv("RAVEL_NO_PERSISTENT", "1")
    s = synth.get_config("small_bf16").replace(layers=2, offset_mode=W.OFFSET_CONCAT, context_period=4)
    wts = synth.draw_weights(s, seed=12, stress=True)
    ea, ex, n = run_parity(s, wts, batch=2, seed=6, steps=24, oracle_dtype=np.float64, check_every=8)
    print(f"small_bf16 concat persistent={persistent}: action err {ea:.2e}, state err {ex:.2e}")


def test_staggered_refreshes_give_each_env_its_own_offset():
    """Five envs refreshed at staggered steps (so their offsets differ within a step),
    80 rows: the per-kernel path with conditioning groups."""
    s = synth.get_config("small_bf16").replace(layers=2, offset_mode=W.OFFSET_CONCAT, context_period=3,
                                               stagger=True)
    wts = synth.draw_weights(s, seed=13, stress=True)
    ea, ex, n = run_parity(s, wts, batch=5, seed=7, steps=12, oracle_dtype=np.float64, check_every=6)
    print(f"small_bf16 concat B=5 staggered: action err {ea:.2e}, state err {ex:.2e}")


def test_training_loss_with_concatenated_offset():
    from tests.test_gpu_train import _case
    print("tiny_fp32 concat training", _case("tiny_fp32", 3, [0, 4, 11], np.float64, offset_mode=W.OFFSET_CONCAT))
