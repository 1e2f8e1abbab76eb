"""Full-horizon synchronous denoising -- plain CPU definition of the baseline
that rolling inference is compared with.

Sec. 4.1 (synchronous evaluation) and App. B.1: the baseline spends the same
generation budget as rolling inference -- one VLM prefill and ten passes of the
action expert -- on ten full-horizon denoising steps.  Every slot of a fresh
chunk starts as Gaussian noise, all slots share one flow time, the passes move
the whole chunk from noise to clean together, and the chunk is executed after
the last pass.  Rolling inference (oracle/rolling.py) instead advances every
slot by one step per pass and releases one clean slot per pass; the paper's
first-action latency table (Sec. 4.1) compares the two.

Time convention as in oracle/rolling.py (tau = 1 pure noise, tau = 0 clean).
With S steps, step s = 0 .. S-1 evaluates the velocity with every slot at
tau_s = (S - s) / S and applies a <- a - v / S: Eq. 3's Euler update with one
shared flow time instead of the rolling profile.

Reading (the paper is silent on it): the baseline's context is fresh, so the
offset conditioning uses context age 0, delta = delta_0.

This is test infrastructure: only the tests, the smoke check and the bench's
CPU-baseline leg may import it.
"""

from __future__ import annotations

import numpy as np


def step_flow_times(steps: int) -> np.ndarray:
    """tau_s = (S - s) / S for s = 0 .. S-1: the shared flow time of each step."""
    return (steps - np.arange(steps, dtype=np.float64)) / steps


def full_denoise(velocity, noise, steps: int):
    """Integrate a chunk from tau = 1 (noise) to tau = 0 with `steps` Euler steps.

    velocity(a, tau) -> v: the velocity of every slot of chunk a [H, D] when all
    slots are at flow time tau.  Returns the chunk at tau = 0 (same dtype as noise).
    """
    a = np.array(noise, copy=True)
    dt = a.dtype.type(1) / a.dtype.type(steps)
    for tau in step_flow_times(steps):
        a = a - dt * np.asarray(velocity(a, tau), dtype=a.dtype)
    return a


def expert_velocity(expert, ctx_k, ctx_v, z=None, delta=None):
    """The expert's velocity with every slot at the same flow time (context age 0
    unless delta is given)."""
    d = expert.s.delta_bias if delta is None else delta

    def v(a, tau):
        return expert.velocity(a, ctx_k, ctx_v, d, z, taus=np.full(len(a), tau))

    return v
