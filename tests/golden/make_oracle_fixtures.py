"""Write the oracle's outputs for the long GPU parity rolls as fixtures.

Two rolls are too slow for the CPU oracle to run beside the GPU inside a test:
  * the pi-style expert at batch 1 (18 layers, width 1024, 8q/1kv x 256, 816 prefix
    tokens, 50 slots, 16 FOP tokens) rolled 1000 steps with one context (t_obs = 0);
  * the large expert at batch 16 (24 layers, width 2048, 16q/4kv x 128, 2048 prefix
    tokens, 100 slots, 32 FOP tokens), envs 0 and 15, 4 steps with the context
    refresh at step 3.
This script rolls them with the oracle alone (``oracle/`` plus the seeded input
generators of ``synth/``) and stores every released action and the ring at
checkpoints, float32, in ``tests/golden/<name>.npz`` (no pickled objects).  The GPU
tests replay the same seeded inputs and compare.

Usage: python tests/golden/make_oracle_fixtures.py [pi_b1_roll1000] [large_b16_roll4]
"""

from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle.rolling import OracleRavel  # noqa: E402

# name -> (workload, batch, env sample, steps, ring checkpoint every, oracle dtype)
FIXTURES = {
    "pi_b1_roll1000": ("pi_b1", 1, [0], 1000, 100, np.float32),
    "large_b16_roll4": ("large_b16", 16, [0, 15], 4, 2, np.float32),
}
WEIGHT_SEED = 0
RING_SEED = 0
CTX_SEED = 0


def describe(name: str) -> dict:
    wl, batch, envs, steps, every, dt = FIXTURES[name]
    s = synth.get_config(wl)
    return dict(workload=wl, shape=s.__dict__ if hasattr(s, "__dict__") else str(s), batch=batch, envs=envs,
                steps=steps, every=every, dtype=np.dtype(dt).name, weight_seed=WEIGHT_SEED, ring_seed=RING_SEED,
                ctx_seed=CTX_SEED)


def roll(name: str, log=print) -> dict:
    wl, batch, envs, steps, every, dt = FIXTURES[name]
    s = synth.get_config(wl)
    wts = synth.draw_weights(s, seed=WEIGHT_SEED)
    o = OracleRavel(s, wts, batch=len(envs), seed=RING_SEED, dtype=dt, env_ids=envs)
    o_env = {e: i for i, e in enumerate(envs)}
    sched = synth.context_schedule(s.replace(batch=batch), steps)
    actions = np.zeros((steps, len(envs), s.action_dim), np.float32)
    rings, ring_steps = [], []
    t0 = time.time()
    for st in range(steps):
        for (s_, e, t_obs, ref) in sched:
            if s_ == st and e in o_env:
                k, v = synth.draw_context(s, CTX_SEED, e, ref)
                o.set_context(o_env[e], k, v, t_obs)
        z = synth.draw_fop_tokens(s, CTX_SEED, st, batch=batch)
        actions[st] = o.step(z[envs])
        if (st + 1) % every == 0 or st == steps - 1:
            rings.append(o.X.astype(np.float32).copy())
            ring_steps.append(st + 1)
        if st % 50 == 0:
            log(f"{name}: step {st} ({time.time() - t0:.0f} s)")
    return dict(actions=actions, rings=np.stack(rings), ring_steps=np.array(ring_steps, np.int64),
                meta=np.array(json.dumps(describe(name), sort_keys=True, default=str)))


def path(name: str) -> str:
    return os.path.join(HERE, name + ".npz")


def load(name: str) -> dict:
    """The stored fixture, checked against the current description of its roll."""
    with np.load(path(name), allow_pickle=False) as f:
        d = {k: f[k] for k in f.files}
    want = json.dumps(describe(name), sort_keys=True, default=str)
    if str(d["meta"]) != want:
        raise RuntimeError(f"{name}: fixture is stale (inputs changed); rerun {os.path.basename(__file__)}")
    return d


def main(argv):
    names = argv or list(FIXTURES)
    for n in names:
        d = roll(n)
        np.savez_compressed(path(n), **d)
        print(f"wrote {path(n)}")


if __name__ == "__main__":
    main(sys.argv[1:])
