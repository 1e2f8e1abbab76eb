"""Counter-based Gaussian noise for the rolling buffer's append step (oracle side).

The paper appends a fresh N(0, I) action at the end of the buffer after every
release (Sec. 3.1, text following Eq. 3). Both sides of the parity check must
draw the *same* noise without sharing code, so the noise is defined here from
published algorithms:

* Philox4x32-10: Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy
  as 1, 2, 3" (SC'11), Sec. 4.2 -- a 10-round Feistel-like bijection of a
  128-bit counter keyed by 64 bits, with round multipliers 0xD2511F53 and
  0xCD9E8D57 and Weyl key increments 0x9E3779B9 and 0xBB67AE85.
* Box-Muller (Box & Muller, 1958): two uniforms (u_a in (0,1], u_b in [0,1))
  give two independent normals sqrt(-2 ln u_a) cos(2 pi u_b) and
  sqrt(-2 ln u_a) sin(2 pi u_b).

Noise stream of the rolling buffer (the convention this repository fixes):
  key     = (seed & 0xffffffff, seed >> 32)
  counter = (j // 4, env, r & 0xffffffff, r >> 32) for action index r and
            vector element j; one Philox call yields elements 4c .. 4c+3.
  u_a     = ((x >> 8) + 1) * 2^-24   (radius uniform, never 0)
  u_b     = (x >> 8) * 2^-24          (angle uniform)
  z[4c]   = R(x0) cos(T(x1)),  z[4c+1] = R(x0) sin(T(x1)),
  z[4c+2] = R(x2) cos(T(x3)),  z[4c+3] = R(x2) sin(T(x3)),
computed in float64 and rounded to float32 (round to nearest even).

This is test infrastructure (part of the CPU oracle); product code never
imports it.
"""

from __future__ import annotations

import numpy as np

PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10(counter, key):
    """Philox4x32 with 10 rounds.

    counter: uint array [..., 4]; key: uint array [..., 2] (broadcastable).
    Returns uint32 array [..., 4].
    """
    c = np.asarray(counter, dtype=np.uint64) & np.uint64(MASK32)
    k = np.asarray(key, dtype=np.uint64) & np.uint64(MASK32)
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = k[..., 0].copy(), k[..., 1].copy()
    m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
    mask = np.uint64(MASK32)
    sh = np.uint64(32)
    for rnd in range(10):
        if rnd > 0:  # key schedule: bump before every round but the first
            k0 = (k0 + np.uint64(PHILOX_W0)) & mask
            k1 = (k1 + np.uint64(PHILOX_W1)) & mask
        p0 = m0 * c0  # exact: both factors < 2^32
        p1 = m1 * c2
        hi0, lo0 = p0 >> sh, p0 & mask
        hi1, lo1 = p1 >> sh, p1 & mask
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def uniform_radius(x):
    """u_a = ((x >> 8) + 1) / 2^24 in (0, 1]; exact in float32 and float64."""
    x = np.asarray(x, dtype=np.uint32)
    return ((x >> np.uint32(8)).astype(np.float64) + 1.0) * 2.0 ** -24


def uniform_angle(x):
    """u_b = (x >> 8) / 2^24 in [0, 1)."""
    x = np.asarray(x, dtype=np.uint32)
    return (x >> np.uint32(8)).astype(np.float64) * 2.0 ** -24


TWO_PI = 6.283185307179586  # float64 nearest to 2*pi


def box_muller(x0, x1):
    """Two float64 normals from two Philox words (radius word, angle word)."""
    rad = np.sqrt(-2.0 * np.log(uniform_radius(x0)))
    ang = TWO_PI * uniform_angle(x1)
    return rad * np.cos(ang), rad * np.sin(ang)


def ring_noise(seed: int, env: int, r: int, dim: int) -> np.ndarray:
    """The N(0, I) action appended for action index r of environment env: float32 [dim]."""
    ngroups = (dim + 3) // 4
    ctr = np.zeros((ngroups, 4), dtype=np.uint64)
    ctr[:, 0] = np.arange(ngroups, dtype=np.uint64)
    ctr[:, 1] = env
    ctr[:, 2] = r & MASK32
    ctr[:, 3] = (r >> 32) & MASK32
    key = np.array([seed & MASK32, (seed >> 32) & MASK32], dtype=np.uint64)
    words = philox4x32_10(ctr, key)  # [ngroups, 4]
    z = np.empty((ngroups, 4), dtype=np.float64)
    z[:, 0], z[:, 1] = box_muller(words[:, 0], words[:, 1])
    z[:, 2], z[:, 3] = box_muller(words[:, 2], words[:, 3])
    return z.reshape(-1)[:dim].astype(np.float32)
