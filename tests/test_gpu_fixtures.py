"""The two long parity rolls compared with oracle outputs stored by
tests/golden/make_oracle_fixtures.py (oracle only, same seeded inputs): the pi-style
expert at batch 1 rolled 1000 steps (the benchmark spec's roll length for that workload), and
the large expert at all 24 of its layers at batch 16 (envs 0 and 15) across a
context refresh.  Every released action and the ring at the stored checkpoints are
compared at max normwise relative error 2e-2 (bf16 with fp32 accumulation)."""

import importlib.util
import os

import numpy as np
import pytest

import synth
from tests.harness import TOL_BF16, GpuRoll, have_gpu, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

_HERE = os.path.dirname(os.path.abspath(__file__))


def _fixtures():
    spec = importlib.util.spec_from_file_location("make_oracle_fixtures",
                                                  os.path.join(_HERE, "golden", "make_oracle_fixtures.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def roll_against_fixture(name, use_graph=True):
    fx = _fixtures()
    want = fx.load(name)
    wl, batch, envs, steps, every, _ = fx.FIXTURES[name]
    s = synth.get_config(wl)
    wts = synth.draw_weights(s, seed=fx.WEIGHT_SEED)
    g = GpuRoll(s, wts, batch, fx.RING_SEED, use_graph=use_graph)
    sched = synth.context_schedule(s.replace(batch=batch), steps)
    worst_a = worst_x = 0.0
    ck = 0
    for st in range(steps):
        for (s_, e, t_obs, ref) in sched:
            if s_ == st:
                g.set_context(e, *synth.draw_context(s, fx.CTX_SEED, e, ref), t_obs)
        a = g.step(synth.draw_fop_tokens(s, fx.CTX_SEED, st, batch=batch))
        err = rel_err(a[envs], want["actions"][st])
        worst_a = max(worst_a, err)
        assert err <= TOL_BF16, f"{name} step {st}: released-action error {err:.3e}"
        if ck < len(want["ring_steps"]) and want["ring_steps"][ck] == st + 1:
            X, t, _ = g.state()
            assert t == st + 1
            ex = rel_err(X[envs], want["rings"][ck])
            worst_x = max(worst_x, ex)
            print(f"{name} step {st + 1}: action error so far {worst_a:.3e}, ring error {ex:.3e}", flush=True)
            assert ex <= TOL_BF16, f"{name} step {st}: ring error {ex:.3e}"
            ck += 1
    assert ck == len(want["ring_steps"])
    return worst_a, worst_x


def test_pi_b1_roll_1000_steps():
    ea, ex = roll_against_fixture("pi_b1_roll1000")
    print(f"pi_b1 1000 steps: action error {ea:.3e}, ring error {ex:.3e}")


def test_large_b16_all_24_layers():
    ea, ex = roll_against_fixture("large_b16_roll4")
    print(f"large_b16 (24 layers): action error {ea:.3e}, ring error {ex:.3e}")
