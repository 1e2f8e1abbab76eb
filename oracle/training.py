"""Streaming-aligned training objective -- plain CPU definition (forward and loss).

Sec. 3.3: an observation step t_o and an offset p are sampled (t_a = t_o + p);
the VLM context comes from t_o, the target is the K-step horizon after t_a, and
the expert receives delta_p = p / K.  The training buffer uses the rolling
buffer's flow-time profile: slot k holds (1 - tau_k) eps_k + tau_k a_hat_k with
tau_k = 1 - k/K (Eq. 5), the target velocity of slot k is a_hat_k - eps_k, and
the loss is the expectation over slots of the squared L2 error (Eq. 6).

Time convention as in oracle/rolling.py (tau = 1 pure noise): slot i = k - 1 has
tau_i = (i+1)/H = 1 - tau_k, so the buffer is tau_i eps_i + (1 - tau_i) a_hat_i and
the velocity this repository's expert predicts is the negated one, eps_i - a_hat_i;
the squared error, and so the loss, is the same number in both conventions.

Readings (the paper is silent on them): the offset is delta = p / K without the
inference-time lead bias delta_0 (Sec. 4.4 adds that bias at inference only); the
loss of one sample is the mean over its H slots of the squared L2 norm over the
action dimension; a batch reports one loss per sample.

This is test infrastructure: only the tests, the smoke check and the bench's
CPU-baseline leg may import it.
"""

from __future__ import annotations

import numpy as np

from .expert import flow_times


def training_buffer(target, noise):
    """[H, D] buffer: slot i = tau_i * eps_i + (1 - tau_i) * a_hat_i, tau_i = (i+1)/H."""
    target = np.asarray(target)
    noise = np.asarray(noise, dtype=target.dtype)
    H = target.shape[0]
    tau = flow_times(H).astype(target.dtype)[:, None]
    return tau * noise + (target.dtype.type(1) - tau) * target


def training_loss(velocity, target, noise):
    """Loss of one sample: mean over slots of ||v_i - (eps_i - a_hat_i)||^2.

    velocity(a) -> v [H, D] for the training buffer a (slot i at tau_i)."""
    a = training_buffer(target, noise)
    v = np.asarray(velocity(a), dtype=a.dtype)
    r = v - (np.asarray(noise, dtype=a.dtype) - np.asarray(target, dtype=a.dtype))
    return float(np.mean(np.sum(r * r, axis=1))), v


def expert_velocity(expert, ctx_k, ctx_v, p: int, z=None):
    """The expert on a training buffer with context age p: delta = p / H."""
    delta = float(p) / expert.s.horizon

    def v(a):
        return expert.velocity(a, ctx_k, ctx_v, delta, z)

    return v
